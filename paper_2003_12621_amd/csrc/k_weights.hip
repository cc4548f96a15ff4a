// Filter spectra, once per layer (Section 3.1, eq. 8 and the filter half of
// eq. 9).
//
// Each K x K filter is zero-padded top-left to L x L and transformed.  The
// padded filter has only K*K nonzeros, so each of its stored bins is a
// direct K*K-term sum, evaluated in double precision with host-computed
// double twiddles and rounded once to fp32.  A CNN layer is a
// cross-correlation, so the stored value is the conjugate spectrum; the
// inverse transform's 1/L^2 is folded in here so the hot path never scales.
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"
#include "launch_util.hpp"

namespace fftsplit {

struct TwiddlesD {
    double c[kTwN];
    double s[kTwN];
};

__global__ __launch_bounds__(256) void weights_kernel(const float* __restrict__ w, float2* __restrict__ wspec,
                                                      int cin, int cout, int coutp, int K, int L, int bins,
                                                      TwiddlesD tw) {
    const size_t total = size_t(bins) * cin * coutp;
    const size_t idx = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int co = int(idx % coutp);
    const size_t rest = idx / coutp;
    const int ci = int(rest % cin);
    const int f = int(rest / cin);
    if (co >= cout) {
        wspec[idx] = make_float2(0.f, 0.f);
        return;
    }
    // Decode the bin from f (order documented in fftsplit.h).  A slot of
    // the real bins holds the (real) values of two bins: (k1, k2) in its
    // real part and (k1b, k2b) in its imaginary part.
    const int h2 = L / 2;
    int k1, k2, k1b = -1, k2b = -1;
    if (L % 2) {   // odd L: complex columns k2 in [1, (L-1)/2], then half of column 0
        if (f < h2 * L) {
            k2 = 1 + f / L;
            k1 = f % L;
        } else {
            k2 = 0;
            k1 = f - h2 * L;
        }
    } else if (f < L * (h2 - 1)) {
        k2 = 1 + f / L;
        k1 = f % L;
    } else if (f < L * (h2 - 1) + h2 - 1) {
        k2 = 0;
        k1 = f - L * (h2 - 1) + 1;
    } else if (f < L * h2 - 2) {
        k2 = h2;
        k1 = f - L * (h2 - 1) - (h2 - 1) + 1;
    } else {
        k1 = 0;
        k1b = h2;
        k2 = k2b = f == L * h2 - 2 ? 0 : h2;
    }
    const int step = L % 2 ? 1 : kTwN / L;   // odd L: the table holds its own L entries
    const float* wp = w + (size_t(co) * cin + ci) * K * K;
    // conj(sum w exp(-2 pi i e / L)) = sum w exp(+2 pi i e / L), e = u k1 + v k2
    auto spectrum = [&](int a, int b, double& re, double& im) {
        re = 0.0;
        im = 0.0;
        for (int u = 0; u < K; ++u) {
            for (int v = 0; v < K; ++v) {
                const int e = ((u * a + v * b) % L) * step;
                const double val = double(wp[u * K + v]);
                re += val * tw.c[e];
                im += val * tw.s[e];
            }
        }
    };
    double re, im;
    spectrum(k1, k2, re, im);
    if (k1b >= 0) {   // two real bins: their imaginary parts are zero
        double re2, im2;
        spectrum(k1b, k2b, re2, im2);
        im = re2;
    }
    const double inv = 1.0 / double(L * L);
    wspec[idx] = make_float2(float(re * inv), float(im * inv));
}

hipError_t launch_weights(const fftsplit_plan_s& p, const float* w, float2* wspec, hipStream_t s,
                          const LaunchEvents& ev) {
    TwiddlesD tw{};
    const double* tc = kTwCosD;
    const double* ts = kTwSinD;
    int nt = kTwN;
    switch (p.L) {
        case 5: tc = kTw5CosD; ts = kTw5SinD; nt = 5; break;
        case 9: tc = kTw9CosD; ts = kTw9SinD; nt = 9; break;
        case 13: tc = kTw13CosD; ts = kTw13SinD; nt = 13; break;
    }
    for (int i = 0; i < nt; ++i) {
        tw.c[i] = tc[i];
        tw.s[i] = ts[i];
    }
    const size_t total = size_t(p.bins) * p.prob.cin * p.coutp;
    const unsigned blocks = unsigned((total + 255) / 256);
    return launch_kernel(weights_kernel, dim3(blocks), dim3(256), 0, s, ev.start, ev.stop, w, wspec, p.prob.cin,
                         p.prob.cout, p.coutp, p.prob.k, p.L, p.bins, tw);
}

}  // namespace fftsplit
