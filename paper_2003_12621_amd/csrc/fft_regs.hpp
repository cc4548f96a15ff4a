// In-register 1-D FFTs of length 8, 16 and 32 for the patch transforms.
//
// One thread owns one length-L sequence in L complex registers.  The
// transform is a radix-2 decimation-in-time network, fully unrolled at
// compile time: every index and every twiddle is a constant, trivial
// twiddles (1 and -i) cost no multiplies, the others are applied with fused
// multiply-adds, and the bit-reversed input order is a renaming of
// registers.  Forward: X[k] = sum_n x[n] exp(-2 pi i n k / L);
// inverse: the same with exp(+...), unnormalised.
#pragma once

#include <hip/hip_runtime.h>

namespace fftsplit {

#include "twiddles.inc"

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }

// One radix-2 decimation-in-time butterfly on (a, b) with twiddle w^e
// applied to b: a, b <- a + w^e b, a - w^e b, where w = exp(-2 pi i / L)
// (forward) or exp(+2 pi i / L) (inverse) and e (0 <= e < L/2) is a
// compile-time constant after unrolling.  w^e = 1 and w^e = -/+i cost four
// adds.  Any other twiddle c + i s is applied in the fused multiply-add form
// of Linzer and Feig: c + i s = m (c/m + i s/m) with m the larger-magnitude
// of c and s, so one of the two parts is exactly 1 and the other is a ratio
// r with |r| <= 1; then w^e b = m t where t costs two FMAs, and a +/- m t two
// FMAs each -- six instructions instead of eight (a complex multiply and
// four adds).
template <int L, bool INV>
__device__ __forceinline__ void butterfly(float2& a, float2& b, int e) {
    const int k = e * (kTwN / L);   // index into the 32-point tables
    const float2 u = a;
    if (k == 0) {
        a = cadd(u, b);
        b = csub(u, b);
        return;
    }
    if (k == kTwN / 4) {             // w^e = -i (forward) or +i (inverse)
        const float2 v = INV ? make_float2(-b.y, b.x) : make_float2(b.y, -b.x);
        a = cadd(u, v);
        b = csub(u, v);
        return;
    }
    const float m = kTwLfScaleF[k];
    const float r = kTwLfRatioF[k];
    const float sg = INV ? 1.f : -1.f;  // w^e = cos + i sg sin of 2 pi k / 32
    float2 t;
    if (kTwLfCos[k]) {  // m = cos, r = sin / cos: w^e b = m (b.x - sg r b.y, b.y + sg r b.x)
        t = make_float2(fmaf(-sg * r, b.y, b.x), fmaf(sg * r, b.x, b.y));
    } else {            // m = sin, r = cos / sin: w^e b = m (r b.x - sg b.y, r b.y + sg b.x)
        t = make_float2(fmaf(r, b.x, -sg * b.y), fmaf(r, b.y, sg * b.x));
    }
    a = make_float2(fmaf(m, t.x, u.x), fmaf(m, t.y, u.y));
    b = make_float2(fmaf(-m, t.x, u.x), fmaf(-m, t.y, u.y));
}

// The DIT stage whose butterflies span SPAN (pairs (s + j, s + j + SPAN) in
// blocks of 2 SPAN, twiddle w^(j L / (2 SPAN))), then the wider stages.
template <int L, bool INV, int SPAN>
struct DitStages {
    __device__ __forceinline__ static void run(float2 (&a)[L]) {
#pragma unroll
        for (int s = 0; s < L; s += 2 * SPAN) {
#pragma unroll
            for (int j = 0; j < SPAN; ++j) butterfly<L, INV>(a[s + j], a[s + j + SPAN], j * (L / (2 * SPAN)));
        }
        DitStages<L, INV, 2 * SPAN>::run(a);
    }
};
template <int L, bool INV>
struct DitStages<L, INV, L> {
    __device__ __forceinline__ static void run(float2 (&)[L]) {}
};

__host__ __device__ constexpr int bitrev(int v, int bits) {
    int r = 0;
    for (int i = 0; i < bits; ++i) r |= ((v >> i) & 1) << (bits - 1 - i);
    return r;
}
template <int L>
__host__ __device__ constexpr int log2i() { return L <= 1 ? 0 : 1 + log2i<L / 2>(); }
template <>
__host__ __device__ constexpr int log2i<1>() { return 0; }

// In-place transform; on return a[k] holds bin k (natural order).  The
// decimation-in-time network takes its input in bit-reversed order, which
// is a renaming of registers.
template <int L, bool INV>
__device__ __forceinline__ void fft(float2 (&a)[L]) {
    float2 t[L];
#pragma unroll
    for (int k = 0; k < L; ++k) t[k] = a[bitrev(k, log2i<L>())];
    DitStages<L, INV, 1>::run(t);
#pragma unroll
    for (int k = 0; k < L; ++k) a[k] = t[k];
}

// Two real sequences packed as z = p + i q: given Z = FFT(z), the spectra of
// p and q at bin k are (Z[k] + conj(Z[-k]))/2 and (Z[k] - conj(Z[-k]))/(2i).
__device__ __forceinline__ void split_two_real(float2 zk, float2 zmk, float2& pk, float2& qk) {
    pk = make_float2(0.5f * (zk.x + zmk.x), 0.5f * (zk.y - zmk.y));
    qk = make_float2(0.5f * (zk.y + zmk.y), 0.5f * (zmk.x - zk.x));
}

}  // namespace fftsplit
