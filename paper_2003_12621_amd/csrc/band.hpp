// Row bands of the image that a work item touches (overlap-save).
//
// A work item is a run of consecutive patches of one channel; patch t sits
// at tile (a, b) of image img with t = (img * th + a) * tw + b.  The rows a
// run of patches needs lie in at most a few images: a partial first image,
// whole images, a partial last image.  Stacked one after another they form
// the item's band: for overlap-save input, tile rows a*T - P .. a*T + T + P
// (the P-row halo of eqs. 5-6), for output, rows a*T .. a*T + T; always
// clipped to the image.  Every band row ("slot") is a whole image row, so a
// band is read or written as a few contiguous runs of memory.
#pragma once

#include <hip/hip_runtime.h>

namespace fftsplit {

struct BandGeom {
    int img0;    // first image of the run
    int nseg;    // images touched (0 for a run of padding patches only)
    int r0;      // first image row held for image img0
    int rows0;   // rows held for image img0
    int r1last;  // end row (exclusive) held for the last image, if nseg >= 2
    int slots;   // rows held in total
};

// Band of patches [t0, t0 + count) (only those below nt are real), with
// `halo` extra rows above and below each tile row.
__host__ __device__ inline BandGeom band_geom(int t0, int count, int nt, int h, int T, int halo, int th, int tw) {
    BandGeom g{0, 0, 0, 0, 0, 0};
    if (t0 >= nt) return g;
    const int tl = (t0 + count < nt ? t0 + count : nt) - 1;
    const int tr0 = t0 / tw, tr1 = tl / tw;
    g.img0 = tr0 / th;
    const int img1 = tr1 / th;
    const int a0 = tr0 - g.img0 * th, a1 = tr1 - img1 * th;
    g.nseg = img1 - g.img0 + 1;
    const int ahi0 = g.nseg == 1 ? a1 : th - 1;
    const int lo = a0 * T - halo;
    g.r0 = lo > 0 ? lo : 0;
    const int hi0 = ahi0 * T + T + halo;
    g.rows0 = (hi0 < h ? hi0 : h) - g.r0;
    const int hil = a1 * T + T + halo;
    g.r1last = hil < h ? hil : h;
    g.slots = g.rows0 + (g.nseg >= 2 ? (g.nseg - 2) * h + g.r1last : 0);
    return g;
}

// Slot of image row r of the band's image img0 + s.
__host__ __device__ inline int band_slot(const BandGeom& g, int h, int s, int r) {
    return s == 0 ? r - g.r0 : g.rows0 + (s - 1) * h + r;
}

// Column-pass lane roles of the band transforms with patch pairs (work
// items of TG <= 32 patches, TG / 2 pairs): lanes l and l + 32 of a wave take
// patches 2 pm and 2 pm + 1 of the same column, so that one 16-byte access
// of the spectra, whose patches are consecutive in memory, serves both
// lanes after a v_permlane32_swap (swap_halves).  Within each group of 16
// consecutive lanes, min(TG / 2, 8) pairs are fastest, then the columns: with
// an odd patch stride of the half spectra in LDS (TG >= 16; at TG = 8 a
// stride of 2 mod 16), the group's 8-byte accesses of one row then fall in
// 16 distinct bank pairs.
template <int TG>
struct PairRole {
    static constexpr int P = TG / 2, Q = P < 8 ? P : 8, CPW = 64 / TG;
    static_assert(TG <= 32 && TG % 2 == 0, "patch pairs need work items of at most 32 patches");
    int pm, hi, patch, col;
    __host__ __device__ PairRole(int lane, int wave) {
        const int r = lane & 31, s = r / Q;
        hi = lane >> 5;
        pm = (s / CPW) * Q + r % Q;
        patch = 2 * pm + hi;
        col = wave * CPW + s % CPW;
    }
};

// Exchanges the upper half-wave's a with the lower half-wave's b (one
// v_permlane32_swap per 32-bit component).  From per-lane values (a, b) of
// patches 2 pm (lane l < 32) and 2 pm + 1 (lane l + 32) it leaves lane l
// both patches' a and lane l + 32 both patches' b, each a 16-byte run in
// patch order; applied to such runs it restores the per-lane values.
__device__ __forceinline__ void swap_halves(float2& a, float2& b) {
    const auto sx = __builtin_amdgcn_permlane32_swap(__float_as_uint(a.x), __float_as_uint(b.x), false, false);
    const auto sy = __builtin_amdgcn_permlane32_swap(__float_as_uint(a.y), __float_as_uint(b.y), false, false);
    a = make_float2(__uint_as_float(sx[0]), __uint_as_float(sy[0]));
    b = make_float2(__uint_as_float(sx[1]), __uint_as_float(sy[1]));
}

// n / d for 0 <= n < 2^22 and d >= 1 with inv_d = 1.0f / d: the float
// product is within 1/2 of n / d, so one correction step is exact.
__device__ __forceinline__ int div_small(int n, int d, float inv_d) {
    int q = int(float(n) * inv_d);
    const int r = n - q * d;
    q += (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
    return q;
}

}  // namespace fftsplit
