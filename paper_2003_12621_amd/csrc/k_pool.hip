// 2x2 stride-2 max-pool (floor) between VGG-16 stages; not part of the
// split method.  One thread per output pixel; a wavefront's 64 outputs read
// two rows of 128 consecutive inputs as float2 pairs when the width is even.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

__global__ __launch_bounds__(256) void maxpool_kernel(const float* __restrict__ x, float* __restrict__ y, int h,
                                                      int w, int ho, int wo, size_t total) {
    const size_t idx = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int j = int(idx % wo);
    const size_t r = idx / wo;
    const int i = int(r % ho);
    const size_t plane = r / ho;
    const float* p = x + (plane * h + 2 * i) * w + 2 * j;
    y[idx] = vmax(vmax3(p[0], p[1], p[w]), p[w + 1]);
}

hipError_t launch_maxpool(const float* x, float* y, int n, int c, int h, int w, hipStream_t s, hipEvent_t stop) {
    const int ho = h / 2, wo = w / 2;
    const size_t total = size_t(n) * c * ho * wo;
    const unsigned blocks = unsigned((total + 255) / 256);
    return launch_kernel(maxpool_kernel, dim3(blocks), dim3(256), 0, s, nullptr, stop, x, y, h, w, ho, wo, total);
}

}  // namespace fftsplit
