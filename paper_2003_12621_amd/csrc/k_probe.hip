// Measurement hooks: the practical ceilings the path's kernels are measured
// against, on the chip they run on.  Neither is part of the method.
//
// matrix_probe_kernel: the contraction's launch (same grid, 256 threads,
// same dynamic LDS, hence the same workgroups per compute unit) with each
// wave issuing the same number of v_mfma_f32_32x32x2f32 operations as a
// contraction wave, from registers, with no memory traffic: the rate the
// fp32 matrix cores sustain for this launch shape, fill and drain included.
//
// stream_probe_kernel: a plain streaming kernel that reads R and writes W
// bytes (the byte mix of the forward or inverse transform), 16 bytes per
// lane per access, many workgroups: the rate HBM sustains for that mix.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

// C independent accumulation chains, `iters` rounds of C operations per
// wave.  The operands change every round so that nothing is loop-invariant;
// the accumulators are summed and written to sink only if the sum equals a
// value it does not take (which keeps the arithmetic from being removed).
template <int C>
__global__ __launch_bounds__(256) void matrix_probe_kernel(float* __restrict__ sink, int iters, float seed) {
    floatx16 acc[C];
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
    float a = seed + float(threadIdx.x) * 1e-3f, b = seed - float(threadIdx.x) * 1e-3f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < C; ++c)
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(c & 1 ? b : a, c & 2 ? a - b : b, acc[c], 0, 0, 0);
        a += 1e-7f;
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    if (s == -1.0f) sink[0] = s;
}

// dst4[i] = src4[i] for i < min(nr4, nw4), 0 for nr4 <= i < nw4; every
// element of src4[0, nr4) is loaded (those past nw4 into an empty asm
// operand, so the loads are not removed).
__global__ __launch_bounds__(256) void stream_probe_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                                           long long nr4, long long nw4) {
    const long long stride = (long long)gridDim.x * blockDim.x;
    const long long n = nr4 > nw4 ? nr4 : nw4;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i < nr4) v = src[i];
        if (i < nw4) dst[i] = v;
        else asm volatile("" ::"v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w));
    }
}

bool probe_aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool probe_overlap(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bn && b0 < a0 + an;
}

}  // namespace fftsplit

using namespace fftsplit;

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_probe_matrix(fftsplit_plan_t plan, float* sink, hipStream_t stream) {
    set_error("");
    if (!plan) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "plan is NULL");
    if (!sink) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "sink is NULL");
    if (plan->device < 0) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "the plan was made for an architecture, not a device");
    if (plan->fuse_cin) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "the plan runs no contraction (channel sum fused into the inverse)");
    const int bm = plan->con_bm, bn = plan->con_bn, kc = plan->con_kc;
    const int wm = bm == 128 && bn == 32 ? 4 : (bm == 256 ? 4 : 2);   // the wave grids launch_contract uses
    const int tm = bm / wm / 32, tn = bn / (4 / wm) / 32;
    const int nstage = (plan->prob.cin + kc - 1) / kc;
    const long long per_wave = (long long)nstage * (kc / 2) * tm * tn * plan->con_products;
    const int pf = plan->con_prefetch;
    const int lds = (pf > 1 ? pf + 1 : 2) * kc * (bm + bn) * 8;
    const long long nb = (long long)(plan->coutp / bm) * (plan->ntp / bn) * plan->bins;
    if (nb < 1 || nb > 0x7fffffffLL) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "grid size out of range");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    const LaunchEvents ev = timing_events();
    hipError_t e;
    if (plan->con_products == 3) {
        e = allow_dynamic_lds(matrix_probe_kernel<3>, lds);
        if (e == hipSuccess)
            e = launch_kernel(matrix_probe_kernel<3>, dim3(unsigned(nb)), dim3(256), unsigned(lds), stream, ev.start,
                              ev.stop, sink, int(per_wave / 3), 1.0f);
    } else {
        e = allow_dynamic_lds(matrix_probe_kernel<4>, lds);
        if (e == hipSuccess)
            e = launch_kernel(matrix_probe_kernel<4>, dim3(unsigned(nb)), dim3(256), unsigned(lds), stream, ev.start,
                              ev.stop, sink, int(per_wave / 4), 1.0f);
    }
    if (e != hipSuccess) return fail(FFTSPLIT_ERROR_DEVICE, std::string("matrix probe launch: ") + hipGetErrorString(e));
    return FFTSPLIT_SUCCESS;
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_probe_stream(const void* src, void* dst, size_t read_bytes,
                                                        size_t write_bytes, hipStream_t stream) {
    set_error("");
    if ((read_bytes && !src) || (write_bytes && !dst))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "NULL buffer with a nonzero size");
    if (read_bytes % 16 || write_bytes % 16 || !probe_aligned16(src) || !probe_aligned16(dst))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "sizes and pointers must be multiples of 16 bytes");
    if (read_bytes && write_bytes && probe_overlap(src, read_bytes, dst, write_bytes))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "src and dst overlap");
    if (!read_bytes && !write_bytes) return FFTSPLIT_SUCCESS;
    const LaunchEvents ev = timing_events();
    const hipError_t e = launch_kernel(stream_probe_kernel, dim3(8192), dim3(256), 0u, stream, ev.start, ev.stop,
                                       static_cast<const float4*>(src), static_cast<float4*>(dst),
                                       (long long)(read_bytes / 16), (long long)(write_bytes / 16));
    if (e != hipSuccess) return fail(FFTSPLIT_ERROR_DEVICE, std::string("stream probe launch: ") + hipGetErrorString(e));
    return FFTSPLIT_SUCCESS;
}
