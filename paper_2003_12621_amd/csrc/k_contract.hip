// Per-frequency-bin channel contraction (Section 3.1, eq. 9, summed over
// input channels): for every stored bin f,
//     Y[f][co][t] = sum_ci W[f][ci][co] * X[f][ci][t]        (complex)
// a batched complex matrix product -- the path's one dense contraction, and
// the only place the fp32 matrix cores (MFMA) are used.
//
// Each complex product is four real MFMA accumulations:
//     Yr += Wr Xr - Wi Xi,   Yi += Wr Xi + Wi Xr.
// v_mfma_f32_32x32x2_f32 operand layout (64 lanes, lane l):
//     A[i][k]: i = l % 32, k = l / 32    (here A = W^T: i = co, k = ci)
//     B[k][j]: k = l / 32, j = l % 32    (here B = X:   j = t)
//     D[i][j], register r: i = 8 (r / 4) + 4 (l / 32) + r % 4, j = l % 32
// so every operand fragment is 32 consecutive complex values of one row,
// and every stored output row is 32 consecutive patches.
#include "fftsplit_internal.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 64;   // output channels per workgroup
constexpr int kBN = 64;   // patches per workgroup
constexpr int kKC = 8;    // input channels per LDS stage

__global__ __launch_bounds__(256) void contract_kernel(const float2* __restrict__ xs, const float2* __restrict__ ws,
                                                       float2* __restrict__ ys, int cin, int coutp, int ntp) {
    __shared__ float2 sW[kKC][kBM];
    __shared__ float2 sX[kKC][kBN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    const int f = blockIdx.z;
    const int co0 = blockIdx.y * kBM;
    const int t0 = blockIdx.x * kBN;

    const float2* xb = xs + size_t(f) * cin * ntp + t0;
    const float2* wb = ws + size_t(f) * cin * coutp + co0;

    floatx16 accR, accI;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        accR[r] = 0.f;
        accI[r] = 0.f;
    }

    for (int k0 = 0; k0 < cin; k0 += kKC) {
#pragma unroll
        for (int it = 0; it < (kKC * 64) / 256; ++it) {
            const int e = it * 256 + tid;
            const int kk = e / 64, jj = e % 64;
            const int ci = k0 + kk;
            float2 wv = make_float2(0.f, 0.f), xv = make_float2(0.f, 0.f);
            if (ci < cin) {
                wv = wb[size_t(ci) * coutp + jj];
                xv = xb[size_t(ci) * ntp + jj];
            }
            sW[kk][jj] = wv;
            sX[kk][jj] = xv;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kKC; kk += 2) {
            const float2 a = sW[kk + (lane >> 5)][wr * 32 + (lane & 31)];
            const float2 b = sX[kk + (lane >> 5)][wc * 32 + (lane & 31)];
            accR = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, b.x, accR, 0, 0, 0);
            accR = __builtin_amdgcn_mfma_f32_32x32x2f32(-a.y, b.y, accR, 0, 0, 0);
            accI = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, b.y, accI, 0, 0, 0);
            accI = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, b.x, accI, 0, 0, 0);
        }
        __syncthreads();
    }

    float2* yb = ys + (size_t(f) * coutp + co0 + wr * 32) * ntp + t0 + wc * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        yb[size_t(i) * ntp] = make_float2(accR[r], accI[r]);
    }
}

hipError_t launch_contract(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                           hipStream_t s) {
    const dim3 grid(p.ntp / kBN, p.coutp / kBM, p.bins);
    hipLaunchKernelGGL(contract_kernel, grid, dim3(256), 0, s, xs, ws, ys, p.prob.cin, p.coutp, p.ntp);
    return hipGetLastError();
}

}  // namespace fftsplit
