// Forward patch transform (Section 3.1: split, eq. 4; pad, eqs. 5-6; FFT of
// each padded patch, first factor of eq. 9).
//
// A workgroup owns TG consecutive patches of one input channel.  Work per
// (patch, channel) is L/2 threads:
//   1. cooperative gather of the TG windows into LDS -- overlap-save: the
//      L x L window starting P rows/cols before the tile, zeros outside the
//      image; overlap-add: the T x T tile, zeros to L x L;
//   2. row pass: thread j transforms rows 2j and 2j+1 packed as one complex
//      sequence (real part row 2j, imaginary part row 2j+1) and separates
//      the two half spectra (bins 0..L/2);
//   3. column pass through LDS: thread j >= 1 transforms column k2 = j;
//      thread 0 transforms the two real-valued columns k2 = 0 and k2 = L/2
//      packed as one complex sequence, then separates them;
//   4. each bin is stored to X[f][c][t]; lanes with consecutive patch index
//      write consecutive addresses.
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"

namespace fftsplit {

template <int L, int TG, bool OAA>
__global__ __launch_bounds__(TG * (L / 2)) void forward_kernel(const float* __restrict__ x, float2* __restrict__ xs,
                                                               int cin, int h, int w, int T, int P, int th, int tw,
                                                               int nt, int ntp) {
    constexpr int H2 = L / 2;
    constexpr int NT = TG * H2;
    constexpr int WP = L + 1;                          // window row pitch (floats)
    constexpr int WIN = TG * L * WP;                   // floats
    constexpr int TBF = TG * L * (H2 + 1) * 2;         // floats of the transpose buffer
    constexpr int SMF = WIN > TBF ? WIN : TBF;
    static_assert(NT % L == 0, "thread count must be a multiple of L");
    __shared__ float sm[SMF];
    __shared__ size_t plane_off[TG];
    __shared__ int org_r[TG], org_c[TG], valid[TG];

    const int tid = threadIdx.x;
    const int c = blockIdx.y;
    const int t0 = blockIdx.x * TG;

    if (tid < TG) {
        const int t = t0 + tid;
        int ok = t < nt;
        int r0 = 0, c0 = 0;
        size_t off = 0;
        if (ok) {
            const int b = t % tw;
            const int rest = t / tw;
            const int a = rest % th;
            const int img = rest / th;
            r0 = OAA ? a * T : a * T - P;
            c0 = OAA ? b * T : b * T - P;
            off = (size_t(img) * cin + c) * size_t(h) * size_t(w);
        }
        plane_off[tid] = off;
        org_r[tid] = r0;
        org_c[tid] = c0;
        valid[tid] = ok;
    }
    __syncthreads();

    // 1. gather: element e = (u, m, q) with q fastest; q is fixed per thread.
    {
        const int q = tid % L;
#pragma unroll
        for (int i = 0; i < (TG * L * L) / NT; ++i) {
            const int e = i * NT + tid;
            const int m = (e / L) % L;
            const int u = e / (L * L);
            const int r = org_r[u] + m;
            const int col = org_c[u] + q;
            bool ok = valid[u] && r >= 0 && r < h && col >= 0 && col < w;
            if (OAA) ok = ok && m < T && q < T;
            float v = 0.f;
            if (ok) v = x[plane_off[u] + size_t(r) * w + col];
            sm[(u * L + m) * WP + q] = v;
        }
    }
    __syncthreads();

    const int u = tid % TG;
    const int j = tid / TG;

    // 2. row pass
    float2 z[L];
#pragma unroll
    for (int q = 0; q < L; ++q)
        z[q] = make_float2(sm[(u * L + 2 * j) * WP + q], sm[(u * L + 2 * j + 1) * WP + q]);
    __syncthreads();  // the transpose buffer reuses the window's LDS
    fft<L, false>(z);
    float2* tb = reinterpret_cast<float2*>(sm);  // [TG][L][H2 + 1]
#pragma unroll
    for (int k = 0; k <= H2; ++k) {
        float2 ra, rb;
        split_two_real(z[k], z[(L - k) % L], ra, rb);
        tb[(u * L + 2 * j) * (H2 + 1) + k] = ra;
        tb[(u * L + 2 * j + 1) * (H2 + 1) + k] = rb;
    }
    __syncthreads();

    // 3. column pass
    float2 cz[L];
    if (j == 0) {
#pragma unroll
        for (int m = 0; m < L; ++m)
            cz[m] = make_float2(tb[(u * L + m) * (H2 + 1)].x, tb[(u * L + m) * (H2 + 1) + H2].x);
    } else {
#pragma unroll
        for (int m = 0; m < L; ++m) cz[m] = tb[(u * L + m) * (H2 + 1) + j];
    }
    fft<L, false>(cz);

    // 4. store
    const size_t bs = size_t(cin) * ntp;
    float2* out = xs + size_t(c) * ntp + t0 + u;
    if (j == 0) {
#pragma unroll
        for (int k1 = 0; k1 <= H2; ++k1) {
            float2 a, b;
            split_two_real(cz[k1], cz[(L - k1) % L], a, b);
            out[size_t(bin_col0(L, k1)) * bs] = a;
            out[size_t(bin_colh(L, k1)) * bs] = b;
        }
    } else {
        float2* o = out + size_t(bin_mid(L, 0, j)) * bs;
#pragma unroll
        for (int k1 = 0; k1 < L; ++k1) o[size_t(k1) * bs] = cz[k1];
    }
}

template <int L, int TG>
static hipError_t launch_forward_L(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s) {
    const dim3 grid(p.ntp / TG, p.prob.cin);
    const dim3 block(TG * (L / 2));
    if (p.oaa)
        hipLaunchKernelGGL((forward_kernel<L, TG, true>), grid, block, 0, s, x, xs, p.prob.cin, p.prob.h, p.prob.w,
                           p.T, p.P, p.th, p.tw, p.nt, p.ntp);
    else
        hipLaunchKernelGGL((forward_kernel<L, TG, false>), grid, block, 0, s, x, xs, p.prob.cin, p.prob.h, p.prob.w,
                           p.T, p.P, p.th, p.tw, p.nt, p.ntp);
    return hipGetLastError();
}

hipError_t launch_forward(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s) {
    switch (p.L) {
        case 8: return launch_forward_L<8, 32>(p, x, xs, s);
        case 16: return launch_forward_L<16, 16>(p, x, xs, s);
        case 32: return launch_forward_L<32, 8>(p, x, xs, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
