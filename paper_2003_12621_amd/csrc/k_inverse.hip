// Inverse patch transform with placement, bias and ReLU (Section 3.1,
// eq. 10 and the concatenation that follows it).
//
// A workgroup owns TG consecutive patches of one output channel; L/2
// threads per (patch, channel):
//   1. column pass: thread j >= 1 inverse-transforms column k2 = j; thread 0
//      rebuilds the full Hermitian columns k2 = 0 and k2 = L/2 from their
//      stored halves, packs them as one complex sequence and inverse-
//      transforms it (both results are real);
//   2. row pass through LDS: thread j rebuilds rows 2j and 2j+1 over all L
//      bins from Hermitian symmetry, packs them as one complex sequence
//      (row 2j real, row 2j+1 imaginary) and inverse-transforms it;
//   3. overlap-save: the top-left T x T block is the output tile (crop), it
//      is written at the tile's place (concatenation) with bias and ReLU.
// The 1/L^2 of the inverse is already in the filter spectra.
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"

namespace fftsplit {

template <int L, int TG>
__global__ __launch_bounds__(TG * (L / 2)) void inverse_os_kernel(const float2* __restrict__ ys,
                                                                  const float* __restrict__ bias,
                                                                  float* __restrict__ y, int cout, int coutp, int h,
                                                                  int w, int T, int th, int tw, int nt, int ntp,
                                                                  int relu) {
    constexpr int H2 = L / 2;
    constexpr int TP = H2 + 1;
    __shared__ float2 tb[TG * L * TP];

    const int tid = threadIdx.x;
    const int co = blockIdx.y;
    const int t0 = blockIdx.x * TG;
    const int u = tid % TG;
    const int j = tid / TG;

    const size_t bs = size_t(coutp) * ntp;
    const float2* in = ys + size_t(co) * ntp + t0 + u;

    // 1. column pass
    float2 cz[L];
    if (j == 0) {
        float2 y0[H2 + 1], yh[H2 + 1];
#pragma unroll
        for (int k1 = 0; k1 <= H2; ++k1) {
            y0[k1] = in[size_t(bin_col0(L, k1)) * bs];
            yh[k1] = in[size_t(bin_colh(L, k1)) * bs];
        }
#pragma unroll
        for (int k1 = 0; k1 < L; ++k1) {
            if (k1 <= H2) {  // U = Y0 + i YH
                cz[k1] = make_float2(y0[k1].x - yh[k1].y, y0[k1].y + yh[k1].x);
            } else {         // Y0[k1] = conj(Y0[L-k1]), likewise YH
                const float2 a = y0[L - k1], b = yh[L - k1];
                cz[k1] = make_float2(a.x + b.y, b.x - a.y);
            }
        }
    } else {
        const float2* src = in + size_t(bin_mid(L, 0, j)) * bs;
#pragma unroll
        for (int k1 = 0; k1 < L; ++k1) cz[k1] = src[size_t(k1) * bs];
    }
    fft<L, true>(cz);
    if (j == 0) {
#pragma unroll
        for (int m = 0; m < L; ++m) {
            tb[(u * L + m) * TP] = make_float2(cz[m].x, 0.f);
            tb[(u * L + m) * TP + H2] = make_float2(cz[m].y, 0.f);
        }
    } else {
#pragma unroll
        for (int m = 0; m < L; ++m) tb[(u * L + m) * TP + j] = cz[m];
    }
    __syncthreads();

    // 2. row pass for rows 2j, 2j+1
    float2 z[L];
    const float2* ra = tb + (u * L + 2 * j) * TP;
    const float2* rb = ra + TP;
#pragma unroll
    for (int k2 = 0; k2 < L; ++k2) {
        if (k2 <= H2) {
            const float2 a = ra[k2], b = rb[k2];
            z[k2] = make_float2(a.x - b.y, a.y + b.x);
        } else {
            const float2 a = ra[L - k2], b = rb[L - k2];
            z[k2] = make_float2(a.x + b.y, b.x - a.y);
        }
    }
    fft<L, true>(z);

    // 3. crop, concatenate, bias, ReLU
    const int t = t0 + u;
    if (t >= nt) return;
    const int b = t % tw;
    const int rest = t / tw;
    const int a = rest % th;
    const int img = rest / th;
    const float bv = bias ? bias[co] : 0.f;
    const int c0 = b * T;
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
        const int m = 2 * j + rr;
        const int r = a * T + m;
        if (m >= T || r >= h) continue;
        float* dst = y + ((size_t(img) * cout + co) * h + r) * size_t(w) + c0;
#pragma unroll
        for (int q = 0; q < L; ++q) {
            if (q < T && c0 + q < w) {
                float v = (rr ? z[q].y : z[q].x) + bv;
                if (relu) v = fmaxf(v, 0.f);
                dst[q] = v;
            }
        }
    }
}

template <int L, int TG>
static hipError_t launch_inverse_L(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                   hipStream_t s) {
    const dim3 grid(p.ntp / TG, p.prob.cout);
    const dim3 block(TG * (L / 2));
    hipLaunchKernelGGL((inverse_os_kernel<L, TG>), grid, block, 0, s, ys, bias, y, p.prob.cout, p.coutp, p.prob.h,
                       p.prob.w, p.T, p.th, p.tw, p.nt, p.ntp, int(p.relu));
    return hipGetLastError();
}

hipError_t launch_inverse(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y, void* aux,
                          hipStream_t s) {
    (void)aux;
    if (p.oaa) return hipErrorNotSupported;
    switch (p.L) {
        case 8: return launch_inverse_L<8, 32>(p, ys, bias, y, s);
        case 16: return launch_inverse_L<16, 16>(p, ys, bias, y, s);
        case 32: return launch_inverse_L<32, 8>(p, ys, bias, y, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
