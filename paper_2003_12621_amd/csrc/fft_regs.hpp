// In-register 1-D FFTs of length 8, 16 and 32 for the patch transforms.
//
// One thread owns one length-L sequence in L complex registers.  The
// transform is a radix-2 decimation-in-frequency network, fully unrolled at
// compile time: every index and every twiddle is a constant, trivial
// twiddles (1 and -i) cost no multiplies, and the bit-reversed output order
// is a renaming of registers.  Forward: X[k] = sum_n x[n] exp(-2 pi i n k / L);
// inverse: the same with exp(+...), unnormalised.
#pragma once

#include <hip/hip_runtime.h>

namespace fftsplit {

#include "twiddles.inc"

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }

// v * w^e with w = exp(-2 pi i / L) (forward) or exp(+2 pi i / L) (inverse);
// e is a compile-time constant after unrolling, 0 <= e < L/2.
template <int L, bool INV>
__device__ __forceinline__ float2 twiddle(float2 v, int e) {
    const int k = e * (kTwN / L);          // index into the 32-entry table
    if (k == 0) return v;
    if (k == kTwN / 4) {                    // w^e = -i (forward) or +i (inverse)
        return INV ? make_float2(-v.y, v.x) : make_float2(v.y, -v.x);
    }
    const float c = kTwCosF[k];
    const float s = kTwSinF[k];
    if (INV) return make_float2(c * v.x - s * v.y, c * v.y + s * v.x);
    return make_float2(c * v.x + s * v.y, c * v.y - s * v.x);
}

// One DIF stage with butterfly span SPAN, then the remaining stages.
template <int L, bool INV, int SPAN>
struct DifStages {
    __device__ __forceinline__ static void run(float2 (&a)[L]) {
#pragma unroll
        for (int s = 0; s < L; s += 2 * SPAN) {
#pragma unroll
            for (int j = 0; j < SPAN; ++j) {
                const float2 u = a[s + j];
                const float2 v = a[s + j + SPAN];
                a[s + j] = cadd(u, v);
                a[s + j + SPAN] = twiddle<L, INV>(csub(u, v), j * (L / (2 * SPAN)));
            }
        }
        DifStages<L, INV, SPAN / 2>::run(a);
    }
};
template <int L, bool INV>
struct DifStages<L, INV, 0> {
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

// In-place transform; on return a[k] holds bin k (natural order).
template <int L, bool INV>
__device__ __forceinline__ void fft(float2 (&a)[L]) {
    DifStages<L, INV, L / 2>::run(a);
    float2 t[L];
#pragma unroll
    for (int k = 0; k < L; ++k) t[k] = a[bitrev(k, log2i<L>())];
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
