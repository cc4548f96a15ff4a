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

// Optional timing events of one entry-point call: `start` is recorded when
// the call's first kernel begins and `stop` when its last kernel ends
// (hipExtLaunchKernel timestamps, no separate event packets).
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

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
