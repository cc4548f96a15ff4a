// OaAConv: the method the paper compares the split convolution against
// (Section 2 and Fig. 1; its operation counts are eqs. 11-12).  The image is
// cut into patches of the filter's size, T = K; each is zero-padded to
// L = 2K - 1 points per side and transformed, multiplied by the filter
// spectra per bin and summed over input channels (the shared contraction
// kernel), inverse-transformed, and the L x L results of neighbouring
// patches are overlap-added.  Here it is the library's overlap-add pipeline
// run at T = K, with the odd transform sizes L = 5, 9, 13 (K = 3, 5, 7) that
// this file adds.
//
// One thread owns one (channel, patch): at these sizes a patch's whole 2-D
// transform fits in registers, and the lanes of a wave hold consecutive
// patches, so every spectrum slot is written (forward) or read (inverse) as
// one contiguous run across the wave.  The transforms are direct sums with
// compile-time twiddles that use the structure of the data:
//   forward: only K x K of the L x L inputs are nonzero, and the input is
//     real, so only columns k2 in [0, (L-1)/2] are formed
//     (S(k1, L-k2) = conj S(L-k1, k2));
//   inverse: the output is real; column k2 = 0 and the pairs k2, L-k2
//     combine into real parts (y = C_0 + 2 Re sum_{k2=1}^{(L-1)/2} ...).
// The inverse's 1/L^2 is folded into the filter spectra, as for even L.
// Of each L x L result, the one entry whose output pixel no other patch
// reaches (T - 2P = 1 per side) is written to y with bias and ReLU; the
// others go to the patch's slot of the aux buffer, and the seam pass sums
// the 1-4 contributions of every other pixel.
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"
#include "launch_util.hpp"

namespace fftsplit {

// cos and sin of 2 pi k / L for the odd sizes (twiddles.inc), k reduced
// mod L; k is a compile-time constant after unrolling.
template <int L>
__device__ __forceinline__ float odd_cos(int k) {
    k %= L;
    if constexpr (L == 5) return kTw5CosF[k];
    else if constexpr (L == 9) return kTw9CosF[k];
    else return kTw13CosF[k];
}
template <int L>
__device__ __forceinline__ float odd_sin(int k) {
    k %= L;
    if constexpr (L == 5) return kTw5SinF[k];
    else if constexpr (L == 9) return kTw9SinF[k];
    else return kTw13SinF[k];
}

template <int L>
__global__ __launch_bounds__(256) void oaa_forward_kernel(const float* __restrict__ x, float2* __restrict__ xs,
                                                          int cin, int h, int w, int th, int tw, int nt, int ntp) {
    constexpr int K = (L + 1) / 2, T = K, H = L / 2, F = stored_bins(L);
    const int c = blockIdx.y;
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= ntp) return;
    float2* dst = xs + spec_offset(c, 0, t, F, ntp);
    const size_t bstride = size_t(kChanBlock) * ntp;   // between the slots of one channel
    if (t >= nt) {   // padding patches: zero spectra
#pragma unroll
        for (int f = 0; f < F; ++f) dst[f * bstride] = make_float2(0.f, 0.f);
        return;
    }
    const int b = t % tw;
    const int rest = t / tw;
    const int a = rest % th;
    const int img = rest / th;
    const int rows = min(T, h - a * T), cols = min(T, w - b * T);
    const float* src = x + ((size_t(img) * cin + c) * h + a * T) * w + b * T;
    float v[K][K];
#pragma unroll
    for (int m = 0; m < K; ++m)
#pragma unroll
        for (int q = 0; q < K; ++q) v[m][q] = (m < rows && q < cols) ? src[m * w + q] : 0.f;

    // rows: R[m][k2] = sum_q v[m][q] exp(-2 pi i q k2 / L), k2 in [0, H]
    float2 R[K][H + 1];
#pragma unroll
    for (int m = 0; m < K; ++m) {
#pragma unroll
        for (int k2 = 0; k2 <= H; ++k2) {
            float re = 0.f, im = 0.f;
#pragma unroll
            for (int q = 0; q < K; ++q) {
                re = fmaf(v[m][q], odd_cos<L>(q * k2), re);
                im = fmaf(-v[m][q], odd_sin<L>(q * k2), im);
            }
            R[m][k2] = make_float2(re, im);
        }
    }
    // columns: S(k1, k2) = sum_m R[m][k2] exp(-2 pi i m k1 / L)
    auto bin = [&](int k1, int k2) {
        float re = 0.f, im = 0.f;
#pragma unroll
        for (int m = 0; m < K; ++m) {
            const float cs = odd_cos<L>(m * k1), sn = odd_sin<L>(m * k1);
            re = fmaf(R[m][k2].x, cs, fmaf(R[m][k2].y, sn, re));
            im = fmaf(R[m][k2].y, cs, fmaf(-R[m][k2].x, sn, im));
        }
        return make_float2(re, im);
    };
#pragma unroll
    for (int k2 = 1; k2 <= H; ++k2)
#pragma unroll
        for (int k1 = 0; k1 < L; ++k1) dst[bin_mid(L, k1, k2) * bstride] = bin(k1, k2);
#pragma unroll
    for (int k1 = 0; k1 <= H; ++k1) dst[bin_odd_col0(L, k1) * bstride] = bin(k1, 0);
}

template <int L>
__global__ __launch_bounds__(256) void oaa_inverse_kernel(const float2* __restrict__ ys,
                                                          const float* __restrict__ bias, float* __restrict__ y,
                                                          float* __restrict__ aux, int cout, int h, int w, int th,
                                                          int tw, int nt, int ntp, int relu) {
    constexpr int K = (L + 1) / 2, T = K, P = K / 2, H = L / 2, F = stored_bins(L), G = patch_group(L);
    const int co = blockIdx.y;
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= nt) return;
    const float2* src = ys + yspec_offset(co, 0, t, F, G, ntp / G);
    float2 Y[F];
#pragma unroll
    for (int f = 0; f < F; ++f) Y[f] = src[f * G];
    const int b = t % tw;
    const int rest = t / tw;
    const int a = rest % th;
    const int img = rest / th;
    float* slot = aux + (size_t(co) * ntp + t) * (L * L);
#pragma unroll
    for (int m = 0; m < L; ++m) {
        // C_k2 = sum_k1 S(k1, k2) exp(+2 pi i m k1 / L); column 0 is
        // Hermitian in k1, so C_0 is real
        float c0 = Y[bin_odd_col0(L, 0)].x;
#pragma unroll
        for (int k1 = 1; k1 <= H; ++k1) {
            const float2 s = Y[bin_odd_col0(L, k1)];
            c0 = fmaf(2.f * s.x, odd_cos<L>(m * k1), fmaf(-2.f * s.y, odd_sin<L>(m * k1), c0));
        }
        float2 C[H + 1];
#pragma unroll
        for (int k2 = 1; k2 <= H; ++k2) {
            float re = 0.f, im = 0.f;
#pragma unroll
            for (int k1 = 0; k1 < L; ++k1) {
                const float2 s = Y[bin_mid(L, k1, k2)];
                const float cs = odd_cos<L>(m * k1), sn = odd_sin<L>(m * k1);
                re = fmaf(s.x, cs, fmaf(-s.y, sn, re));
                im = fmaf(s.x, sn, fmaf(s.y, cs, im));
            }
            C[k2] = make_float2(re, im);
        }
        // y[m][q] = C_0 + 2 Re sum_{k2=1}^{H} C_k2 exp(+2 pi i q k2 / L)
#pragma unroll
        for (int q = 0; q < L; ++q) {
            float acc = c0;
#pragma unroll
            for (int k2 = 1; k2 <= H; ++k2)
                acc = fmaf(2.f * C[k2].x, odd_cos<L>(q * k2), fmaf(-2.f * C[k2].y, odd_sin<L>(q * k2), acc));
            if (m == 0 && q == 0) {
                // the one pixel only this patch reaches: (aT + P, bT + P)
                const int r = a * T + P, cc = b * T + P;
                if (r < h && cc < w) {
                    float v = acc + (bias ? bias[co] : 0.f);
                    if (relu) v = vmax(v, 0.f);
                    y[((size_t(img) * cout + co) * h + r) * w + cc] = v;
                }
            } else {
                slot[m * L + q] = acc;
            }
        }
    }
}

template <int L>
static hipError_t launch_oaa_forward_L(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                       const LaunchEvents& ev) {
    const dim3 grid(unsigned((p.ntp + 255) / 256), unsigned(p.prob.cin));
    return launch_kernel(oaa_forward_kernel<L>, grid, dim3(256), 0, s, ev.start, ev.stop, x, xs, p.prob.cin,
                         p.prob.h, p.prob.w, p.th, p.tw, p.nt, p.ntp);
}

template <int L>
static hipError_t launch_oaa_inverse_L(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                       float* aux, hipStream_t s, const LaunchEvents& ev) {
    const dim3 grid(unsigned((p.nt + 255) / 256), unsigned(p.prob.cout));
    hipError_t e = launch_kernel(oaa_inverse_kernel<L>, grid, dim3(256), 0, s, ev.start, nullptr, ys, bias, y, aux,
                                 p.prob.cout, p.prob.h, p.prob.w, p.th, p.tw, p.nt, p.ntp, int(p.relu));
    if (e != hipSuccess) return e;
    return launch_seam(p, aux, bias, y, s, ev.stop);
}

hipError_t launch_oaa_forward(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                              const LaunchEvents& ev) {
    if (!p.oaa || p.T != p.prob.k) return hipErrorInvalidValue;
    switch (p.L) {
        case 5: return launch_oaa_forward_L<5>(p, x, xs, s, ev);
        case 9: return launch_oaa_forward_L<9>(p, x, xs, s, ev);
        case 13: return launch_oaa_forward_L<13>(p, x, xs, s, ev);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_oaa_inverse(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y, float* aux,
                              hipStream_t s, const LaunchEvents& ev) {
    if (!p.oaa || p.T != p.prob.k || !aux) return hipErrorInvalidValue;
    switch (p.L) {
        case 5: return launch_oaa_inverse_L<5>(p, ys, bias, y, aux, s, ev);
        case 9: return launch_oaa_inverse_L<9>(p, ys, bias, y, aux, s, ev);
        case 13: return launch_oaa_inverse_L<13>(p, ys, bias, y, aux, s, ev);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
