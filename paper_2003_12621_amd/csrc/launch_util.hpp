// Launch helpers shared by the kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace fftsplit {

// MI355X dispatches consecutive workgroup ids round-robin over its 8
// accelerator dies (XCDs), each with a private L2.  Remapping the hardware
// id so that every XCD receives one contiguous range of logical ids keeps
// workgroups that share inputs (neighbouring patches, the channel blocks of
// one frequency bin) on the same L2.  The map is a bijection on [0, nb).
constexpr int kNumXcd = 8;

__device__ __forceinline__ int xcd_logical_block(int hw_block, int nb) {
    const int q = nb / kNumXcd;
    const int r = nb % kNumXcd;
    const int x = hw_block % kNumXcd;
    const int i = hw_block / kNumXcd;
    return x * q + (x < r ? x : r) + i;
}

// Allows a kernel to use more than the default dynamic LDS once per process.
template <typename K>
inline hipError_t allow_dynamic_lds(K kernel, int bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               bytes);
}

// Workgroups of `kernel` (with `threads` threads and `lds` bytes of dynamic
// LDS) that one compute unit holds at once; at least 1.
template <typename K>
inline int resident_blocks(K kernel, int threads, int lds) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(kernel), threads, lds) !=
            hipSuccess ||
        n < 1)
        n = 1;
    return n;
}

// Items per workgroup for a kernel that walks consecutive work items:
// enough that the grid fits the `slots` workgroups the device holds at once
// (a single wave of workgroups), at least 1.
inline int items_per_workgroup(int nitems, int slots) {
    if (slots < 1) slots = 1;
    const int ipw = (nitems + slots - 1) / slots;
    return ipw < 1 ? 1 : ipw;
}

// Raw buffer access (gfx9 buffer descriptors).  A load whose byte offset
// (VGPR offset; the scalar offset is only used for accesses known to be in
// range) is at or beyond `bytes` returns 0 and a store there is dropped, so
// padding outside an image costs no compare-and-select per element.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
constexpr unsigned kOutOfRange = 0x80000000u;   // offset that is always out of range

__device__ __forceinline__ BufRsrc make_rsrc(const void* base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// A 16-byte load of data read once and not again soon (the filter spectra
// in the contraction): marked non-temporal, so that streaming it through
// does not push the patch and output spectra out of the caches.
__device__ __forceinline__ uint4 load_stream_u4(const uint4* p) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(t.x, t.y, t.z, t.w);
}

// Cache policy of a buffer load or store: kCacheDefault, or kCacheStream
// (the "nt" bit) for data that no later kernel of the same convolution
// reads (an input the stage consumes for good, or the layer's output), so
// that it does not displace data a following kernel still needs.
constexpr int kCacheDefault = 0;
constexpr int kCacheStream = 2;

__device__ __forceinline__ float buf_load_f32(BufRsrc r, unsigned voff, unsigned soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
template <int CP = kCacheDefault>
__device__ __forceinline__ float2 buf_load_f32x2(BufRsrc r, unsigned voff, unsigned soff) {
    typedef int int2v __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, CP));
}
template <int CP = kCacheDefault>
__device__ __forceinline__ float4 buf_load_f32x4(BufRsrc r, unsigned voff, unsigned soff) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, CP));
}
// A store of more than 8 bytes needs one wait state before a VALU
// instruction may overwrite its data registers.  The compiler's hazard model
// assumes the wait is only needed when the scalar offset is not a register,
// but on gfx950 a 16-byte store with a register scalar offset immediately
// followed by such a write was measured to store the new value.  The
// uniform offset is therefore added to the lane offset and the scalar
// offset is the constant 0, for which the compiler inserts the wait.
// (`soff` + an out-of-range `voff` stays out of range: both are below 2^31.)
template <int CP = kCacheDefault>
__device__ __forceinline__ void buf_store_f32x4(float4 v, BufRsrc r, unsigned voff, unsigned soff) {
    typedef int int4v __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(int4v, v), r, voff + soff, 0, CP);
}
template <int CP = kCacheDefault>
__device__ __forceinline__ void buf_store_f32(float v, BufRsrc r, unsigned voff, unsigned soff) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, voff, soff, CP);
}
template <int CP = kCacheDefault>
__device__ __forceinline__ void buf_store_f32x2(float2 v, BufRsrc r, unsigned voff, unsigned soff) {
    typedef int int2v __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(int2v, v), r, voff, soff, CP);
}

// Maximum of two or three floats for ReLU and the max-pool, as IEEE 754-2019
// `maximum` (a NaN operand gives NaN, as numpy's maximum does).  gfx950 has
// it as one instruction (v_maximum3_f32) for up to three operands; fmaxf
// (IEEE maxNum) costs an extra instruction per operand that the compiler
// cannot prove quiet, which is every value read from memory or computed
// in another basic block.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float vmax3(float a, float b, float c) { return vmax(vmax(a, b), c); }

// Optional timing events of one entry-point call: `start` is recorded when
// the call's first kernel begins and `stop` when its last kernel ends
// (hipExtLaunchKernel timestamps, no separate event packets).
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

// The calling thread's timing events (fftsplit_set_timing_events).
LaunchEvents timing_events();

template <typename K, typename... Args>
inline hipError_t launch_kernel(K kernel, dim3 grid, dim3 block, unsigned lds, hipStream_t s, hipEvent_t start,
                                hipEvent_t stop, Args... args) {
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, grid, block, lds, s, start, stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
    return hipGetLastError();
}

}  // namespace fftsplit
