// Inverse patch transform with placement, bias and ReLU (Section 3.1,
// eq. 10 and the concatenation that follows it).
//
// A workgroup owns TG consecutive patches of one output channel, with L/2
// threads per patch:
//   1. column pass (patch index fastest across lanes, so each bin of the TG
//      patches is one contiguous 8*TG-byte read): thread j >= 1 inverse-
//      transforms column k2 = j; thread 0 rebuilds the Hermitian columns
//      k2 = 0 and k2 = L/2 from their stored halves, packs them as one
//      complex sequence and inverse-transforms it (both results are real);
//   2. row pass through LDS: thread j rebuilds rows 2j and 2j+1 over all L
//      bins from Hermitian symmetry, packs them as one complex sequence (row
//      2j real, row 2j+1 imaginary) and inverse-transforms it;
//   3. overlap-save placement: the top-left T x T block of each patch is its
//      output tile (the crop), staged in LDS and written back row by row
//      with bias and ReLU; horizontally adjacent patches of a group land in
//      one contiguous run of the output row (the concatenation).  With the
//      fused max-pool (T even) each 2x2 block of the staged crop is reduced
//      to its maximum first and the [h/2][w/2] output written instead;
//   3'. overlap-add placement (zero-padded patches): entry (p, q) of a
//      patch's L x L result belongs at output (aT+P+p', bT+P+q') with
//      p' = p for p < T and p - L otherwise, so each patch covers the L x L
//      region around its tile.  Entries with p, q < T-2P (the "core") have
//      no other contributor and are written directly with bias and ReLU;
//      the rest (seams, 2P wide, shared by 2 or 4 neighbouring patches) go to
//      a per-patch L x L slot of the aux buffer, and seam_kernel then sums
//      the 1-4 contributions of every seam pixel in a fixed order (no
//      atomics, deterministic) and applies bias and ReLU.
// The inverse's 1/L^2 is already folded into the filter spectra.
#include "band.hpp"
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"
#include "launch_util.hpp"

namespace fftsplit {

template <int L, int TG>
struct InvShape {
    static constexpr int H2 = L / 2;
    static constexpr int NT = TG * H2;
    static constexpr int TP = H2 + 1;             // half-spectrum row pitch (float2)
    static constexpr int TTS = L * TP + 2;        // half-spectrum patch stride (float2)
    static constexpr int SP = L + 1;              // staged tile row pitch (floats)
    static constexpr int STS = L * SP + 1;        // staged tile patch stride (floats)
    // store phase: lanes = q (L) x u_sub (US) x m_sub (MS)
    static constexpr int US = (L == 32) ? 1 : (L == 16 ? 4 : 8);
    static constexpr int MS = NT / (L * US);
    static constexpr int TB_BYTES = TG * TTS * 8;
    static constexpr int ST_BYTES = TG * STS * 4;
    static constexpr int LDS_BYTES = TB_BYTES > ST_BYTES ? TB_BYTES : ST_BYTES;
    static_assert(NT % (L * US) == 0 && TG % US == 0 && L % MS == 0, "store-phase lane split");
};

template <int L, int TG, bool OAA>
__global__ __launch_bounds__(TG * (L / 2)) void inverse_kernel(const float2* __restrict__ ys,
                                                               const float* __restrict__ bias, float* __restrict__ y,
                                                               float* __restrict__ aux, int cout, int coutp, int h,
                                                               int w, int T, int P, int th, int tw, int nt, int ntp,
                                                               int ngroups, int relu, int pool, int y_elems) {
    using S = InvShape<L, TG>;
    constexpr int H2 = S::H2, NT = S::NT, TP = S::TP, TTS = S::TTS, SP = S::SP, STS = S::STS;
    extern __shared__ float4 lds_raw[];
    float2* tb = reinterpret_cast<float2*>(lds_raw);
    float* st = reinterpret_cast<float*>(lds_raw);
    __shared__ int dst_off[TG];
    __shared__ int rows_ok[TG], cols_ok[TG];

    const int tid = threadIdx.x;
    const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
    const int g = lb % ngroups;
    const int co = lb / ngroups;
    const int t0 = g * TG;

    if (tid < TG) {
        const int t = t0 + tid;
        int ro = 0, cw = 0, off = 0;
        if (t < nt) {
            const int b = t % tw;
            const int rest = t / tw;
            const int a = rest % th;
            const int img = rest / th;
            // overlap-save: rows/cols of the crop inside the image;
            // overlap-add: rows/cols of the core (offset P) inside the image.
            ro = OAA ? min(T - 2 * P, h - a * T - P) : min(T, h - a * T);
            cw = OAA ? min(T - 2 * P, w - b * T - P) : min(T, w - b * T);
            // pool (overlap-save, T even): the tile's pooled origin in the
            // [h/2][w/2] output
            off = pool ? ((img * cout + co) * (h >> 1) + ((a * T) >> 1)) * (w >> 1) + ((b * T) >> 1)
                       : ((img * cout + co) * h + a * T) * w + b * T + (OAA ? P * w + P : 0);
        }
        dst_off[tid] = off;
        rows_ok[tid] = ro;
        cols_ok[tid] = cw;
    }

    // 1. column pass: output spectra (co, f, t0 + u) with a per-lane byte
    // offset and the per-bin stride as the scalar offset (always in range).
    {
        const int u = tid % TG;
        const int j = tid / TG;
        const BufRsrc ry = make_rsrc(ys, unsigned(size_t(coutp) * ntp * 8 * stored_bins(L)));
        static_assert(TG == patch_group(L), "a work item is one patch group of the output spectra");
        const unsigned bs8 = unsigned(TG) * 8u;   // bin stride (patch-group-major)
        const unsigned voff = unsigned(yspec_offset(co, 0, t0 + u, stored_bins(L), TG, ngroups)) * 8u;
        float2 cz[L];
        if (j == 0) {
            float2 y0[H2 + 1], yh[H2 + 1];
            // the real bins (k1 = 0, L/2) of both columns share two slots
            const float2 ra = buf_load_f32x2(ry, voff, unsigned(bin_real_a(L)) * bs8);
            const float2 rb = buf_load_f32x2(ry, voff, unsigned(bin_real_b(L)) * bs8);
            y0[0] = make_float2(ra.x, 0.f);
            y0[H2] = make_float2(ra.y, 0.f);
            yh[0] = make_float2(rb.x, 0.f);
            yh[H2] = make_float2(rb.y, 0.f);
#pragma unroll
            for (int k1 = 1; k1 < H2; ++k1) {
                y0[k1] = buf_load_f32x2(ry, voff, unsigned(bin_col0(L, k1)) * bs8);
                yh[k1] = buf_load_f32x2(ry, voff, unsigned(bin_colh(L, k1)) * bs8);
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
            const unsigned vj = voff + unsigned(bin_mid(L, 0, j)) * bs8;
#pragma unroll
            for (int k1 = 0; k1 < L; ++k1) cz[k1] = buf_load_f32x2(ry, vj, unsigned(k1) * bs8);
        }
        fft<L, true>(cz);
        float2* cb = tb + u * TTS;
        if (j == 0) {
#pragma unroll
            for (int m = 0; m < L; ++m) {
                cb[m * TP] = make_float2(cz[m].x, 0.f);
                cb[m * TP + H2] = make_float2(cz[m].y, 0.f);
            }
        } else {
#pragma unroll
            for (int m = 0; m < L; ++m) cb[m * TP + j] = cz[m];
        }
    }
    __syncthreads();

    // 2. row pass (j fastest across lanes)
    {
        const int j = tid % H2;
        const int u = tid / H2;
        float2 z[L];
        const float2* ra = tb + u * TTS + 2 * j * TP;
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
        __syncthreads();  // the staged tiles reuse the half-spectrum LDS
        float* s0 = st + u * STS + 2 * j * SP;
#pragma unroll
        for (int q = 0; q < L; ++q) {
            s0[q] = z[q].x;
            s0[SP + q] = z[q].y;
        }
    }
    __syncthreads();

    // 3. placement: lanes (q, u_sub, m_sub), q fastest
    {
        const int q = tid % L;
        const int us = (tid / L) % S::US;
        const int ms = tid / (L * S::US);
        const float bv = bias ? bias[co] : 0.f;
        const int cs = T - 2 * P;  // overlap-add core size
        const BufRsrc ry_out = make_rsrc(y, unsigned(size_t(y_elems) * 4));
#pragma unroll 4
        for (int ub = 0; ub < TG; ub += S::US) {
            const int u = ub + us;
            const int ro = rows_ok[u], cw = cols_ok[u];
            const int d = dst_off[u];
            const float* s = st + u * STS;
            if (!OAA && pool) {
                // 2x2 max-pool of the crop (T is even, so no pooling window
                // straddles two patches; floor at an odd image edge), then
                // bias and ReLU, which commute with the maximum; lane q < L/2
                // takes pooled column q of pooled rows m
                const int qq = q < L / 2 ? q : 0;
                const unsigned vq = unsigned(d + q) * 4u;
#pragma unroll
                for (int mb = 0; mb < L / 2; mb += S::MS) {
                    const int m = mb + ms;
                    const float* sp = s + 2 * m * SP + 2 * qq;
                    float v = vmax(vmax3(sp[0], sp[1], sp[SP]), sp[SP + 1]) + bv;
                    if (relu) v = vmax(v, 0.f);
                    const bool in = m < (ro >> 1) && q < (cw >> 1);
                    buf_store_f32(v, ry_out, in ? vq + unsigned(m * (w >> 1)) * 4u : kOutOfRange, 0);
                }
            } else if (!OAA) {
                // Output through a descriptor over y: lanes outside the crop
                // (m >= ro or q >= cw) get an out-of-range offset, which drops
                // the store.
                const unsigned vq = unsigned(d + q) * 4u;
#pragma unroll
                for (int mb = 0; mb < L; mb += S::MS) {
                    const int m = mb + ms;
                    float v = s[m * SP + q] + bv;
                    if (relu) v = vmax(v, 0.f);
                    const unsigned vo = (m < ro && q < cw) ? vq + unsigned(m * w) * 4u : kOutOfRange;
                    buf_store_f32(v, ry_out, vo, 0);
                }
            } else if (t0 + u < nt) {
                float* slot = aux + (co * ntp + t0 + u) * (L * L);
#pragma unroll
                for (int mb = 0; mb < L; mb += S::MS) {
                    const int m = mb + ms;
                    const float zv = s[m * SP + q];
                    if (m < cs && q < cs) {
                        if (m < ro && q < cw) {
                            float v = zv + bv;
                            if (relu) v = vmax(v, 0.f);
                            y[d + m * w + q] = v;
                        }
                    } else {
                        slot[m * L + q] = zv;
                    }
                }
            }
        }
    }
}

// Overlap-add seams: every output pixel within P of a tile boundary (in
// either direction) sums the aux entries of the 1-4 patches covering it, in
// the order (a0-1, b0-1), (a0-1, b0), (a0, b0-1), (a0, b0), then adds the
// bias and applies ReLU.  Core pixels were written by inverse_kernel.
// Seam pixels of a plane are enumerated compactly: indices below nsr * w
// walk the seam rows (all columns), the rest walk the seam columns of the
// other rows.  Seam rows are those with (r + P) mod T < 2P; the k-th is
// ((k + P) / 2P) T - P + (k + P) mod 2P (likewise for columns); the k-th
// other row is (k / (T - 2P)) T + P + k mod (T - 2P).  A thread takes
// kSeamPix pixels and issues all their loads before any sum: a missing
// contribution reads an out-of-range offset of a descriptor over the
// plane's patch results, which returns 0, so every pixel sums four terms in
// the fixed order (adding +0 leaves a sum unchanged).
constexpr int kSeamPix = 4;

__global__ __launch_bounds__(256) void seam_kernel(const float* __restrict__ aux, const float* __restrict__ bias,
                                                   float* __restrict__ y, int cout, int h, int w, int T, int P, int L,
                                                   int th, int tw, int ntp, int relu, int nsr, int nsc, int bpp) {
    // blocks run plane-major, bpp blocks per plane
    const int plane = blockIdx.x / bpp;
    const int blk = blockIdx.x - plane * bpp;
    const int img = plane / cout, co = plane % cout;
    const int P2 = 2 * P, LL = L * L;
    const BufRsrc rin = make_rsrc(aux + (size_t(co) * ntp + size_t(img) * th * tw) * LL, unsigned(th * tw * LL * 4));
    const int n_row = nsr * w, n_all = n_row + (h - nsr) * nsc;
    float v[kSeamPix][4];
    int out[kSeamPix];
#pragma unroll
    for (int i = 0; i < kSeamPix; ++i) {
        const int idx = (blk * kSeamPix + i) * 256 + threadIdx.x;
        int r = 0, c = 0;
        bool seam_r = true;
        if (idx < n_row) {
            const int k = idx / w;
            c = idx - k * w;
            r = ((k + P) / P2) * T - P + (k + P) % P2;
        } else if (idx < n_all) {
            const int j = idx - n_row;
            const int k = j / nsc, sc = j - k * nsc;
            const int cs = T - P2;
            r = (k / cs) * T + P + k % cs;
            c = ((sc + P) / P2) * T - P + (sc + P) % P2;
            seam_r = false;
        }
        const bool live = idx < n_all;
        out[i] = live ? r * w + c : -1;
        const bool seam_c = (c + P) % T < P2;
        const int a0 = (r + P) / T, b0 = (c + P) / T;
#pragma unroll
        for (int da = 1; da >= 0; --da) {
            const int a = a0 - da;
            int p = r - a * T - P;
            if (p < 0) p += L;
            const bool ok_a = live && (!da || seam_r) && a >= 0 && a < th;
#pragma unroll
            for (int db = 1; db >= 0; --db) {
                const int b = b0 - db;
                int qq = c - b * T - P;
                if (qq < 0) qq += L;
                const bool ok = ok_a && (!db || seam_c) && b >= 0 && b < tw;
                const unsigned off = ok ? unsigned(((a * tw + b) * L + p) * L + qq) * 4u : kOutOfRange;
                v[i][2 * (1 - da) + (1 - db)] = buf_load_f32(rin, off, 0);
            }
        }
    }
    const float bv = bias ? bias[co] : 0.f;
    float* yp = y + size_t(plane) * h * w;
#pragma unroll
    for (int i = 0; i < kSeamPix; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) acc += v[i][j];
        float o = acc + bv;
        if (relu) o = vmax(o, 0.f);
        if (out[i] >= 0) yp[out[i]] = o;
    }
}


// Overlap-save inverse transform writing whole row bands (width a multiple
// of 4, at most 256; crop width T >= L/2).  Same work items and transforms as inverse_kernel;
// what changes is the memory traffic and how items overlap:
//   * the output spectra of a workgroup's next item are loaded into
//     registers while the current item's rows are transformed and its band
//     is stored (streaming loads: nothing reads them again); a workgroup's
//     items are gridDim.x apart, so the workgroups sweep the spectra and
//     the output in order;
//   * at TG <= 32 the spectra are read in 16-byte patch pairs: lanes l and
//     l + 32 of a wave hold patches 2m and 2m + 1 of one column (PairRole,
//     band.hpp), each loads one bin of both, and one exchange of the
//     half-waves (swap_halves) gives every lane its own patch;
//   * the column pass runs one instruction stream in every lane: lane j = 0,
//     which rebuilds the two Hermitian columns k2 = 0 and k2 = L/2 and packs
//     them as one complex sequence, does so with selects, so no wave
//     executes two paths;
//   * the crops (T x T tiles, eq. 10) are placed in an LDS band of whole
//     output rows (band.hpp, no halo; pitch `obp`, odd) and the band is
//     written with 16-byte streaming stores (kCacheStream: no later kernel
//     of the convolution reads y), lanes along each row, with bias and ReLU;
//     in the first and last tile row of an item only the columns of its own
//     tiles are written;
//   * LDS strides are odd (the half-spectrum patch stride: band_half_stride),
//     so the lanes of a wave spread over the banks.
// POOL: the 2x2 max-pool happens in the store phase (FFTSPLIT_MAXPOOL), and
// ReLU after it.
// NCI > 0 (layers with NCI <= 4 input channels): the per-bin channel sum
// (eq. 9) is done here instead of by the contraction, and the output
// spectra are never stored: each item forms its spectra from the patch
// spectra xsp (held in registers while consecutive items share the patch
// group: items run patch-group-major, so the group's NCI channels are read
// once per workgroup) and the item's filter spectra, staged in LDS from
// wsp.  The products are the contraction's (the two packed slots part by
// part).
template <int L, int TG, int NV, bool POOL, int NCI>
__global__ __launch_bounds__(TG * (L / 2), 2) void inverse_band_kernel(
    const float2* __restrict__ ys, const float* __restrict__ bias, float* __restrict__ y, int cout, int coutp, int h,
    int w, int T, int th, int tw, int nt, int ntp, int ngroups, int nitems, int ipw, int obp, int relu,
    unsigned y_bytes, float inv_h, float inv_tw, float inv_th, const float2* __restrict__ xsp,
    const float2* __restrict__ wsp, int cin, int wl_off) {
    constexpr int H2 = L / 2, NT = TG * H2, NW = NT / 64, TP = H2 + 1;
    constexpr int TTS = band_half_stride(L, TG);  // half-spectrum patch stride (float2)
    constexpr int F = stored_bins(L);
    extern __shared__ float4 lds_raw[];
    float2* tb = reinterpret_cast<float2*>(lds_raw);
    float* ob = reinterpret_cast<float*>(lds_raw);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const BufRsrc ry = make_rsrc(ys, unsigned(size_t(coutp) * ntp * 8 * F));
    const BufRsrc ryo = make_rsrc(y, y_bytes);
    static_assert(TG == patch_group(L), "a work item is one patch group of the output spectra");
    const unsigned bs8 = unsigned(TG) * 8u;   // bin stride (patch-group-major)
    auto opaque = [](int v) {
        asm volatile("" : "+v"(v));
        return v;
    };
    // a uniform value the compiler may not hoist out of the item loop
    auto opaque_s = [](int v) {
        asm volatile("" : "+s"(v));
        return v;
    };

    const int lw = xcd_logical_block(blockIdx.x, gridDim.x);
    // NCI = 0: workgroup lw runs items lw, lw + gridDim.x, lw + 2 gridDim.x,
    // ..., so that at any moment the workgroups together read one contiguous
    // range of the output spectra and write one contiguous range of y (on
    // the VGG-16 layers, whose spectra exceed the last-level cache, 13-16 %
    // faster than a contiguous run of items per workgroup).  NCI > 0: a
    // contiguous run of `ipw` items, so that consecutive items of a
    // workgroup share their patch group's spectra.
    const int istep = NCI > 0 ? 1 : int(gridDim.x);
    const int ibeg = NCI > 0 ? lw * ipw : lw;
    const int iend = NCI > 0 ? min(ibeg + ipw, nitems) : nitems;
    // (channel, first patch) of an item: channel-major, or patch-group-major
    // when the channel sum is done here
    auto decode = [&](int item, int& co, int& t0) {
        if constexpr (NCI > 0) {
            const int gi = item / cout;
            co = item - gi * cout;
            t0 = gi * TG;
        } else {
            co = item / ngroups;
            t0 = (item - co * ngroups) * TG;
        }
    };

    // column-pass roles: patch uc, column jc.  With patch pairs (kPair,
    // band.hpp) lanes l and l + 32 of a wave take patches 2 pm and 2 pm + 1
    // of one column, so that one 16-byte load per lane serves both
    // (load_spectra).  Otherwise the patch is the fastest index across lanes.
    constexpr bool kPair = NCI == 0 && TG <= 32;
    const PairRole<kPair ? TG : 32> pr(lane, wv);
    const int hiw = pr.hi, pm = pr.pm;
    const int uc = kPair ? pr.patch : tid % TG;
    const int jc = kPair ? pr.col : tid / TG;
    const bool j0 = jc == 0;
    // Lane jc >= 1 needs column k2 = jc: pa[k1] = bin (k1, jc) and
    // pb[k1] = bin (k1 + L/2, jc), k1 < L/2.  Lane 0 needs the halves
    // k1 <= L/2 of the real columns k2 = 0 and L/2: pa[0] and pb[0] are the
    // two slots of their real bins, pa[k1] and pb[k1] (k1 >= 1) their
    // complex bins k1.
    float2 pa[H2], pb[H2];
    // kPair: the loaded 16-byte pairs, (pa, pb) of patch 2 pm in the lower
    // half-wave's (x, y) and the upper's (z, w) once exchanged
    float4 pq[kPair ? H2 : 1];
    // slot of pa[k1] / pb[k1] in this lane's column
    auto slot_a = [&](int k1) { return j0 ? (k1 == 0 ? bin_real_a(L) : bin_col0(L, k1)) : bin_mid(L, k1, jc); };
    auto slot_b = [&](int k1) { return j0 ? (k1 == 0 ? bin_real_b(L) : bin_colh(L, k1)) : bin_mid(L, k1 + H2, jc); };
    // NCI > 0: patch spectra of this lane's column for the current patch
    // group, and the next item's filter spectra (WPT per thread)
    constexpr int WPT = NCI > 0 ? (F * NCI + NT - 1) / NT : 1;
    float2 xa[NCI > 0 ? NCI : 1][H2], xb[NCI > 0 ? NCI : 1][H2];
    float2 wpre[WPT];
    float2* wl = reinterpret_cast<float2*>(lds_raw) + wl_off;
    int gcur = -1;
    const BufRsrc rxs = make_rsrc(xsp, NCI > 0 ? unsigned(size_t(kChanBlock) * ntp * 8 * F) : 0u);
    const BufRsrc rws = make_rsrc(wsp, NCI > 0 ? unsigned(size_t(F) * cin * coutp * 8) : 0u);
    auto load_x = [&](int t0) {
        // channel c < 16 of bin f: ((f * 16 + c) * ntp + t) * 8 bytes
        const unsigned lane8 = unsigned(t0 + opaque(uc)) * 8u;
        const unsigned fs8 = unsigned(kChanBlock) * unsigned(ntp) * 8u;
#pragma unroll
        for (int ci = 0; ci < (NCI > 0 ? NCI : 1); ++ci) {
#pragma unroll
            for (int k1 = 0; k1 < H2; ++k1) {
                xa[ci][k1] = buf_load_f32x2(rxs, lane8 + unsigned(slot_a(k1)) * fs8, unsigned(ci * ntp * 8));
                xb[ci][k1] = buf_load_f32x2(rxs, lane8 + unsigned(slot_b(k1)) * fs8, unsigned(ci * ntp * 8));
            }
        }
    };
    auto load_spectra = [&](int item) {
        int co = 0, t0 = 0;
        bool ok = false;
        if (item >= 0) {
            decode(item, co, t0);
            ok = true;
        }
        if constexpr (NCI > 0) {
            // W[f][ci][co] of the item's channel, e = f * NCI + ci
#pragma unroll
            for (int k = 0; k < WPT; ++k) {
                const int e = k * NT + tid;
                const int f = e / NCI, ci = e - (e / NCI) * NCI;
                const bool in = ok && e < F * NCI;
                wpre[k] = buf_load_f32x2(rws, in ? unsigned(((f * cin + ci) * coutp + co) * 8) : kOutOfRange, 0);
            }
            return;
        }
        // item = co * ngroups + t0 / TG: the item's run starts at item * F * TG
        if constexpr (kPair) {
            // lanes l < 32 read the a bins, lanes l + 32 the b bins, each
            // 16 bytes: patches 2 pm and 2 pm + 1 (each 8 consecutive lanes
            // read 128 contiguous bytes of one bin)
            const unsigned pair8 = unsigned(yspec_offset(co, 0, t0 + 2 * opaque(pm), F, TG, ngroups)) * 8u;
            const int s0 = hiw ? (j0 ? bin_real_b(L) : bin_mid(L, H2, jc)) : (j0 ? bin_real_a(L) : bin_mid(L, 0, jc));
            const int s1 = hiw ? (j0 ? bin_colh(L, 1) - 1 : bin_mid(L, H2, jc)) : (j0 ? bin_col0(L, 1) - 1 : bin_mid(L, 0, jc));
            const unsigned v0 = ok ? pair8 + unsigned(s0) * bs8 : kOutOfRange;
            const unsigned v1 = ok ? pair8 + unsigned(s1) * bs8 : kOutOfRange;
            pq[0] = buf_load_f32x4<kCacheStream>(ry, v0, 0);
#pragma unroll
            for (int k1 = 1; k1 < H2; ++k1) pq[k1] = buf_load_f32x4<kCacheStream>(ry, v1, unsigned(k1) * bs8);
            return;
        }
        const unsigned lane8 = unsigned(yspec_offset(co, 0, t0 + opaque(uc), F, TG, ngroups)) * 8u;
        const unsigned va0 = ok ? lane8 + unsigned(j0 ? bin_real_a(L) : bin_mid(L, 0, jc)) * bs8 : kOutOfRange;
        const unsigned vb0 = ok ? lane8 + unsigned(j0 ? bin_real_b(L) : bin_mid(L, H2, jc)) * bs8 : kOutOfRange;
        const unsigned va = ok ? lane8 + unsigned(j0 ? bin_col0(L, 1) - 1 : bin_mid(L, 0, jc)) * bs8 : kOutOfRange;
        const unsigned vb = ok ? lane8 + unsigned(j0 ? bin_colh(L, 1) - 1 : bin_mid(L, H2, jc)) * bs8 : kOutOfRange;
        pa[0] = buf_load_f32x2<kCacheStream>(ry, va0, 0);
        pb[0] = buf_load_f32x2<kCacheStream>(ry, vb0, 0);
#pragma unroll
        for (int k1 = 1; k1 < H2; ++k1) {
            pa[k1] = buf_load_f32x2<kCacheStream>(ry, va, unsigned(k1) * bs8);
            pb[k1] = buf_load_f32x2<kCacheStream>(ry, vb, unsigned(k1) * bs8);
        }
    };

    // store-phase roles: lanes along a band row, 16 bytes each
    const int w4 = w >> 2;
    const int rpi = 64 / w4;
    const int lrow = lane / w4;
    const int c4 = lane - lrow * w4;
    const int slot0 = wv * rpi + lrow;
    const int slot_step = NW * rpi;
    const unsigned cross4 = unsigned(cout - 1) * unsigned(h) * unsigned(w) * 4u;
    const int dq = slot_step / h, dr = slot_step - dq * h;

    auto process = [&](int item) {
        int co, t0;
        decode(item, co, t0);
        const BandGeom g = band_geom(t0, TG, nt, h, T, 0, th, tw);
        if constexpr (kPair) {
            // the lower half-wave holds the a bins of patches (2 pm,
            // 2 pm + 1), the upper their b bins: one exchange leaves each
            // lane (a, b) of its own patch
#pragma unroll
            for (int k1 = 0; k1 < H2; ++k1) {
                pa[k1] = make_float2(pq[k1].x, pq[k1].y);
                pb[k1] = make_float2(pq[k1].z, pq[k1].w);
                swap_halves(pa[k1], pb[k1]);
            }
        }
        if constexpr (NCI > 0) {
            // the item's filter spectra into LDS, the next item's loaded,
            // the patch group's spectra loaded when the group changes
#pragma unroll
            for (int k = 0; k < WPT; ++k)
                if (k * NT + tid < F * NCI) wl[k * NT + tid] = wpre[k];
            if (t0 != gcur) {
                load_x(t0);
                gcur = t0;
            }
            __syncthreads();
            // per-bin channel sum (eq. 9): pa, pb = sum_ci W x, four
            // multiply-adds per complex product.  The two packed slots
            // (lane 0, k1 = 0) multiply part by part: (Wr Xr, Wi Xi), the
            // same multiply-adds with the cross terms' operands zeroed.
            auto cmac = [](float2 s, float2 w, float2 x, bool packed) {
                const float xc = packed ? 0.f : x.y;          // cross term of the real part
                const float xd = packed ? x.y : x.x;          // Wi's partner in the imaginary part
                s.x = fmaf(w.x, x.x, s.x);
                s.x = fmaf(-w.y, xc, s.x);
                s.y = fmaf(w.y, xd, s.y);
                s.y = fmaf(w.x, xc, s.y);
                return s;
            };
#pragma unroll
            for (int k1 = 0; k1 < H2; ++k1) {
                float2 sa = make_float2(0.f, 0.f), sb = make_float2(0.f, 0.f);
                const float2* wa = wl + slot_a(k1) * NCI;
                const float2* wb = wl + slot_b(k1) * NCI;
                const bool packed = k1 == 0 && j0;
#pragma unroll
                for (int ci = 0; ci < NCI; ++ci) {
                    sa = cmac(sa, wa[ci], xa[ci][k1], packed);
                    sb = cmac(sb, wb[ci], xb[ci][k1], packed);
                }
                pa[k1] = sa;
                pb[k1] = sb;
            }
        }

        // column pass
        {
            // lane 0: column spectra Y0[k1], YH[k1] for k1 <= L/2.  The bias
            // enters at bin (0, 0): with the unnormalised inverse, adding b
            // there adds b to every pixel of the patch.
            const float bv = bias ? bias[co] : 0.f;
            auto y0 = [&](int k) {
                return k == 0 ? make_float2(pa[0].x + bv, 0.f) : (k == H2 ? make_float2(pa[0].y, 0.f) : pa[k]);
            };
            auto yh = [&](int k) {
                return k == 0 ? make_float2(pb[0].x, 0.f) : (k == H2 ? make_float2(pb[0].y, 0.f) : pb[k]);
            };
            float2 cz[L];
            // Only the first wave has a lane j = 0.  At L = 16 the other
            // waves skip the Hermitian rebuild and its selects (a branch on
            // the wave index, the same in every lane of a wave); at L = 32
            // that branch made the inverse slower, so every wave runs the
            // selects there.
            if (L != 16 || wv == 0) {
#pragma unroll
                for (int k1 = 0; k1 < L; ++k1) {
                    float2 v0;
                    if (k1 <= H2) {  // lane 0: U = Y0 + i YH
                        const float2 a = y0(k1), b = yh(k1);
                        v0 = make_float2(a.x - b.y, a.y + b.x);
                    } else {         // lane 0: Y0[k1] = conj(Y0[L-k1]), likewise YH
                        const float2 a = y0(L - k1), b = yh(L - k1);
                        v0 = make_float2(a.x + b.y, b.x - a.y);
                    }
                    const float2 v1 = k1 < H2 ? pa[k1] : pb[k1 - H2];
                    cz[k1] = j0 ? v0 : v1;
                }
            } else {
#pragma unroll
                for (int k1 = 0; k1 < L; ++k1) cz[k1] = k1 < H2 ? pa[k1] : pb[k1 - H2];
            }
            // NCI > 0: the next item's filter spectra stay in flight
            // through this whole item
            if constexpr (NCI > 0) load_spectra(item + istep < iend ? item + istep : -1);
            fft<L, true>(cz);
            // lane 0's result is the two real columns packed (column 0 +
            // i * column L/2): it stays packed in slot 0 for the row pass
            float2* cbw = tb + opaque(uc * TTS);
#pragma unroll
            for (int m = 0; m < L; ++m) cbw[m * TP + jc] = cz[m];
            // NCI = 0: the next item's output spectra are issued here, after
            // this item's column transform rather than before it, and stay
            // in flight through its row pass and store phase; the registers
            // they fill are then not live across the column transform.
            if constexpr (NCI == 0) load_spectra(item + istep < iend ? item + istep : -1);
        }
        __syncthreads();

        // row pass (j fastest across lanes): rows j and j + L/2 (a stride of
        // L/2 rows, so that the 16 lanes of a patch spread over all banks),
        // and placement of the crop in the band
        {
            const int j = tid % H2;
            const int u = tid / H2;
            float2 z[L];
            const float2* ra = tb + opaque(u * TTS + j * TP);
            const float2* rb = ra + H2 * TP;
            // slot 0 holds (column 0, column L/2), both real in a row: the
            // packed row sequence takes row j's value as its real part and
            // row j + L/2's as its imaginary part
            const float2 p0 = ra[0], q0 = rb[0];
            z[0] = make_float2(p0.x, q0.x);
            z[H2] = make_float2(p0.y, q0.y);
#pragma unroll
            for (int k2 = 1; k2 < L; ++k2) {
                if (k2 < H2) {
                    const float2 a = ra[k2], b = rb[k2];
                    z[k2] = make_float2(a.x - b.y, a.y + b.x);
                } else if (k2 > H2) {
                    const float2 a = ra[L - k2], b = rb[L - k2];
                    z[k2] = make_float2(a.x + b.y, b.x - a.y);
                }
            }
            __syncthreads();  // the output band reuses the half-spectrum LDS
            fft<L, true>(z);
            // ReLU on the transform's results; with the max-pool it comes
            // after the pooling instead (relu(max(.)) = max(relu(.)), on a
            // quarter of the values)
            if (!POOL && relu) {
#pragma unroll
                for (int q = 0; q < L; ++q) z[q] = make_float2(vmax(z[q].x, 0.f), vmax(z[q].y, 0.f));
            }
            const int t = t0 + u;
            if (t < nt && j < T) {
                const int tr = div_small(t, tw, inv_tw);
                const int b = t - tr * tw;
                const int img = div_small(tr, th, inv_th);
                const int a = tr - img * th;
                const int r = a * T + j;
                // rows run through the images in order: row r of image
                // img0 + sg sits at slot sg * h + r - r0
                const int sl = __umul24(img - g.img0, h) - g.r0 + r;
                const bool ok0 = r < h;
                const bool ok1 = r + H2 < h && j + H2 < T;
                // one exec-mask branch per row, and the crop width T (at
                // least L/2) as a scalar loop bound re-read per item, so the
                // tail's bound checks stay scalar compares
                float* d = ob + opaque(sl * obp + b * T);
                const int tq = opaque_s(T);
                if (ok0) {
#pragma unroll
                    for (int q = 0; q < L; ++q) {
                        if (q >= H2 && q >= tq) break;
                        d[q] = z[q].x;
                    }
                }
                if (ok1) {
#pragma unroll
                    for (int q = 0; q < L; ++q) {
                        if (q >= H2 && q >= tq) break;
                        d[H2 * obp + q] = z[q].y;
                    }
                }
            }
        }
        __syncthreads();

        // store phase with the 2x2 max-pool (POOL): the band's slots pair up
        // into pooled rows (tile rows start on even image rows and hold an
        // even number of rows, and the image height is even), each lane
        // reads 4 columns of 2 slots and writes 2 pooled values (8 bytes)
        if constexpr (POOL) {
            const int hp = h >> 1, wp = w >> 1;
            const int tl = (t0 + TG < nt ? t0 + TG : nt) - 1;
            const int tr0 = t0 / tw, tr1 = tl / tw;
            // pooled columns of this item's tiles in its first and last tile rows
            const int lo0 = ((t0 - tr0 * tw) * T) >> 1;
            const int hi_last = min((tl - tr1 * tw + 1) * T, w) >> 1;
            const int hi_first = tr1 == tr0 ? hi_last : wp;
            const int rows_first = min(T, h - (tr0 % th) * T) >> 1;
            const int rows_last = min(T, h - (tr1 % th) * T) >> 1;
            const int pslots = g.slots >> 1;
            const int last0 = pslots - rows_last;
            const bool edge = ((lo0 | hi_last) & 1) != 0;
            const int col = 2 * c4;
            const bool in_first = col >= lo0 && col + 2 <= hi_first;
            const bool in_last = col + 2 <= hi_last;
            const bool lane_ok = lrow < rpi;
            const unsigned crossp = unsigned(cout - 1) * unsigned(hp) * unsigned(wp) * 4u;
            const int dqp = slot_step / hp, drp = slot_step - dqp * hp;
            const int sl0 = opaque(slot0);
            // the lane writes whole pairs at pooled slots [sbeg, send): the
            // first (last) tile row's slots only where its columns lie in
            // the item's range; one unsigned compare per slot
            const int sbeg = in_first ? 0 : rows_first;
            const int send = lane_ok ? (in_last ? pslots : min(last0, pslots)) : 0;
            const unsigned span = unsigned(max(send - sbeg, 0));
            const int xs0 = sl0 - sbeg;
            const int x0 = sl0 + (g.r0 >> 1);
            const int qd = div_small(x0, hp, 2.f * inv_h);
            const int rr0 = x0 - qd * hp;
            const unsigned voff0 = unsigned((((g.img0 * cout + co) * hp + (g.r0 >> 1)) * wp) * 4) +
                                   unsigned(sl0 * wp * 4) + unsigned(8 * c4) + unsigned(qd) * crossp;
            const unsigned dq_off = unsigned(dqp) * crossp;
            const float* src = ob + 2 * sl0 * obp + 4 * c4;
            // 2x2 maximum, then ReLU: with -inf as the floor (no ReLU) the
            // second maximum leaves its other operands as they are
            const float lo = relu ? 0.f : -__builtin_inff();
            auto pool4 = [&](const float* sp) {
                return make_float2(vmax3(vmax3(sp[0], sp[1], sp[obp]), sp[obp + 1], lo),
                                   vmax3(vmax3(sp[2], sp[3], sp[obp + 2]), sp[obp + 3], lo));
            };
            {
                // batches of SB pooled slots, LDS reads before stores
                constexpr int SB = 4, NP = (NV + 1) / 2;
                int rr = rr0;
                unsigned voff = voff0;
#pragma unroll
                for (int k0 = 0; k0 < NP; k0 += SB) {
                    float2 v[SB];
                    bool full[SB];
#pragma unroll
                    for (int i = 0; i < SB && k0 + i < NP; ++i) {
                        const int k = k0 + i;
                        full[i] = unsigned(xs0 + k * slot_step) < span;
                        v[i] = pool4(full[i] ? src + 2 * k * slot_step * obp : ob);
                    }
#pragma unroll
                    for (int i = 0; i < SB && k0 + i < NP; ++i) {
                        const int k = k0 + i;
                        buf_store_f32x2<kCacheStream>(v[i], ryo, full[i] ? voff : kOutOfRange, unsigned(k * slot_step * wp * 4));
                        rr += drp;
                        voff += dq_off;
                        const bool carry = rr >= hp;
                        rr -= carry ? hp : 0;
                        voff += carry ? crossp : 0u;
                    }
                }
            }
            if (edge) {
                // pairs that straddle the item's first or last column
                int rr = rr0;
                unsigned voff = voff0;
#pragma unroll
                for (int k = 0; k < (NV + 1) / 2; ++k) {
                    const int ps = sl0 + k * slot_step;
                    const bool full = unsigned(xs0 + k * slot_step) < span;
                    const bool first = ps < rows_first;
                    const bool last = ps >= last0;
                    const int lo = first ? lo0 : 0;
                    const int hi = first ? hi_first : (last ? hi_last : wp);
                    if (lane_ok && ps < pslots && !full && col + 2 > lo && col < hi) {
                        const float2 ve = pool4(src + 2 * k * slot_step * obp);
                        const unsigned soff = unsigned(k * slot_step * wp * 4);
                        buf_store_f32<kCacheStream>(ve.x, ryo, col >= lo && col < hi ? voff : kOutOfRange, soff);
                        buf_store_f32<kCacheStream>(ve.y, ryo, col + 1 >= lo && col + 1 < hi ? voff + 4u : kOutOfRange, soff);
                    }
                    rr += drp;
                    voff += dq_off;
                    const bool carry = rr >= hp;
                    rr -= carry ? hp : 0;
                    voff += carry ? crossp : 0u;
                }
            }
        } else
        // store phase: whole band rows (bias and ReLU are already applied:
        // the bias is in the DC bin, so every pixel of every patch carries
        // it, and ReLU came after the row transform)
        {
            const int tl = (t0 + TG < nt ? t0 + TG : nt) - 1;
            const int tr0 = t0 / tw, tr1 = tl / tw;
            // columns of this item's tiles in its first and last tile rows
            const int lo0 = (t0 - tr0 * tw) * T;
            const int hi_last = min((tl - tr1 * tw + 1) * T, w);
            const int hi_first = tr1 == tr0 ? hi_last : w;
            const int rows_first = min(T, h - (tr0 % th) * T);
            const int rows_last = min(T, h - (tr1 % th) * T);
            const int last0 = g.slots - rows_last;
            // whether some float4 of the first or last tile row straddles the
            // item's column range (the same for every lane of the item)
            const bool edge = ((lo0 | hi_last) & 3) != 0;
            const int col = 4 * c4;
            const bool in_first = col >= lo0 && col + 4 <= hi_first;
            const bool in_last = col + 4 <= hi_last;
            const bool lane_ok = lrow < rpi;
            const int sl0 = opaque(slot0);
            // the lane writes whole float4s at slots [sbeg, send): the first
            // (last) tile row's slots only where its columns lie in the
            // item's range; one unsigned compare per slot
            const int sbeg = in_first ? 0 : rows_first;
            const int send = lane_ok ? (in_last ? g.slots : min(last0, g.slots)) : 0;
            const unsigned span = unsigned(max(send - sbeg, 0));
            const int xs0 = sl0 - sbeg;
            const int x0 = sl0 + g.r0;
            const int qd = div_small(x0, h, inv_h);
            const int rr0 = x0 - qd * h;
            const unsigned voff0 = unsigned((((g.img0 * cout + co) * h + g.r0) * w) * 4) + unsigned(sl0 * w * 4) +
                                   unsigned(16 * c4) + unsigned(qd) * cross4;
            const unsigned dq_off = unsigned(dq) * cross4;
            const float* src = ob + sl0 * obp + 4 * c4;
            // Slot k of this lane goes to byte offset voff + k * slot_step *
            // w * 4 of y, where voff advances by whole images (cross4) as the
            // lane's rows cross into the next image.
            //
            // Every lane issues one 16-byte store per slot (dropped through an
            // out-of-range offset where it has nothing to write, after a read
            // of the band's first float4), so the count of stores after this
            // item's spectrum loads is fixed.  Slots go in batches of SB whose
            // LDS reads are all issued before their stores (the compiler does
            // not move LDS reads above buffer stores), so SB reads are in
            // flight at once.
            {
                constexpr int SB = 4;
                int rr = rr0;
                unsigned voff = voff0;
#pragma unroll
                for (int k0 = 0; k0 < NV; k0 += SB) {
                    float4 v[SB];
                    bool full[SB];
#pragma unroll
                    for (int i = 0; i < SB && k0 + i < NV; ++i) {
                        const int k = k0 + i;
                        full[i] = unsigned(xs0 + k * slot_step) < span;
                        const float* sp = full[i] ? src + k * slot_step * obp : ob;
                        v[i] = make_float4(sp[0], sp[1], sp[2], sp[3]);
                    }
#pragma unroll
                    for (int i = 0; i < SB && k0 + i < NV; ++i) {
                        const int k = k0 + i;
                        buf_store_f32x4<kCacheStream>(v[i], ryo, full[i] ? voff : kOutOfRange, unsigned(k * slot_step * w * 4));
                        rr += dr;
                        voff += dq_off;
                        const bool carry = rr >= h;
                        rr -= carry ? h : 0;
                        voff += carry ? cross4 : 0u;
                    }
                }
            }
            // Only where a float4 straddles an item's first or last column
            // (never when items start and end on tile-row boundaries whose
            // columns are multiples of 4) are 4-byte stores added.
            if (edge) {
                int rr = rr0;
                unsigned voff = voff0;
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    const int sl = sl0 + k * slot_step;
                    const bool full = unsigned(xs0 + k * slot_step) < span;
                    const bool first = sl < rows_first;
                    const bool last = sl >= last0;
                    const int lo = first ? lo0 : 0;
                    const int hi = first ? hi_first : (last ? hi_last : w);
                    if (lane_ok && sl < g.slots && !full && col + 4 > lo && col < hi) {
                        const float* se = src + k * slot_step * obp;
                        const unsigned soff = unsigned(k * slot_step * w * 4);
                        buf_store_f32<kCacheStream>(se[0], ryo, col >= lo && col < hi ? voff : kOutOfRange, soff);
                        buf_store_f32<kCacheStream>(se[1], ryo, col + 1 >= lo && col + 1 < hi ? voff + 4u : kOutOfRange, soff);
                        buf_store_f32<kCacheStream>(se[2], ryo, col + 2 >= lo && col + 2 < hi ? voff + 8u : kOutOfRange, soff);
                        buf_store_f32<kCacheStream>(se[3], ryo, col + 3 >= lo && col + 3 < hi ? voff + 12u : kOutOfRange, soff);
                    }
                    rr += dr;
                    voff += dq_off;
                    const bool carry = rr >= h;
                    rr -= carry ? h : 0;
                    voff += carry ? cross4 : 0u;
                }
            }
        }
        __syncthreads();  // the next item's column pass reuses the band's LDS
    };

    // The first item is peeled off the loop so that, inside the loop, the
    // wait for an item's spectra leaves the previous item's stores in flight.
    if (ibeg < iend) {
        load_spectra(ibeg);
        process(ibeg);
        for (int item = ibeg + istep; item < iend; item += istep) process(item);
    }
}

template <int L, int TG, int NV, bool POOL, int NCI = 0>
static hipError_t launch_inverse_band_v(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                        hipStream_t s, const LaunchEvents& ev, const float2* xs = nullptr,
                                        const float2* ws = nullptr) {
    constexpr int NT = TG * (L / 2);
    auto kern = inverse_band_kernel<L, TG, NV, POOL, NCI>;
    const int wl_off = (p.inv_lds + 15) / 16 * 2;   // float2 offset of the filter-spectrum stage
    const int lds = NCI > 0 ? (wl_off + stored_bins(L) * NCI) * 8 : p.inv_lds;
    if (lds > 64 * 1024) {
        const hipError_t attr = allow_dynamic_lds(kern, lds);
        if (attr != hipSuccess) return attr;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern), NT, lds) !=
            hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    const int ngroups = p.ntp / TG;
    const int nitems = ngroups * p.prob.cout;
    const int ipw = items_per_workgroup(nitems, p.cus * per_cu);
    const dim3 grid(unsigned((nitems + ipw - 1) / ipw));
    const unsigned y_bytes = unsigned(size_t(p.prob.n) * p.prob.cout * (POOL ? (p.prob.h / 2) * (p.prob.w / 2)
                                                                             : p.prob.h * p.prob.w) * 4);
    return launch_kernel(kern, grid, dim3(NT), unsigned(lds), s, ev.start, ev.stop, ys, bias, y, p.prob.cout, p.coutp,
                         p.prob.h, p.prob.w, p.T, p.th, p.tw, p.nt, p.ntp, ngroups, nitems, ipw, p.inv_obp,
                         int(p.relu), y_bytes, 1.0f / float(p.prob.h), 1.0f / float(p.tw), 1.0f / float(p.th), xs,
                         ws, p.prob.cin, wl_off);
}

template <int L, int TG, int NV>
static hipError_t launch_inverse_band(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                      hipStream_t s, const LaunchEvents& ev) {
    return p.pool_fused ? launch_inverse_band_v<L, TG, NV, true>(p, ys, bias, y, s, ev)
                        : launch_inverse_band_v<L, TG, NV, false>(p, ys, bias, y, s, ev);
}

template <int L, int TG, int NV, bool POOL>
static hipError_t launch_inverse_fused_p(const fftsplit_plan_s& p, const float2* xs, const float2* ws,
                                         const float* bias, float* y, hipStream_t s, const LaunchEvents& ev) {
    switch (p.prob.cin) {
        case 1: return launch_inverse_band_v<L, TG, NV, POOL, 1>(p, nullptr, bias, y, s, ev, xs, ws);
        case 2: return launch_inverse_band_v<L, TG, NV, POOL, 2>(p, nullptr, bias, y, s, ev, xs, ws);
        case 3: return launch_inverse_band_v<L, TG, NV, POOL, 3>(p, nullptr, bias, y, s, ev, xs, ws);
        case 4:
            if constexpr (L == 8) return launch_inverse_band_v<L, TG, NV, POOL, 4>(p, nullptr, bias, y, s, ev, xs, ws);
            break;
    }
    return hipErrorInvalidValue;
}

hipError_t launch_inverse_fused(const fftsplit_plan_s& p, const float2* xs, const float2* ws, const float* bias,
                                float* y, hipStream_t s, const LaunchEvents& ev) {
    if (!p.fuse_cin) return hipErrorInvalidValue;
    switch (p.L) {
        case 8:
            return p.pool_fused ? launch_inverse_fused_p<8, 64, kBandNV8, true>(p, xs, ws, bias, y, s, ev)
                                : launch_inverse_fused_p<8, 64, kBandNV8, false>(p, xs, ws, bias, y, s, ev);
        case 16:
            return p.pool_fused ? launch_inverse_fused_p<16, 32, kBandNV16, true>(p, xs, ws, bias, y, s, ev)
                                : launch_inverse_fused_p<16, 32, kBandNV16, false>(p, xs, ws, bias, y, s, ev);
    }
    return hipErrorInvalidValue;
}

template <int L, int TG, bool OAA>
static hipError_t launch_inverse_v(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                   float* aux, hipStream_t s, const LaunchEvents& ev) {
    using S = InvShape<L, TG>;
    auto kern = inverse_kernel<L, TG, OAA>;
    static hipError_t attr = allow_dynamic_lds(kern, S::LDS_BYTES);
    if (attr != hipSuccess) return attr;
    const int ngroups = p.ntp / TG;
    const dim3 grid(unsigned(ngroups) * unsigned(p.prob.cout));
    const bool pool = !OAA && p.pool_fused;
    const int y_elems = pool ? p.prob.n * p.prob.cout * (p.prob.h / 2) * (p.prob.w / 2)
                             : p.prob.n * p.prob.cout * p.prob.h * p.prob.w;
    hipError_t e = launch_kernel(kern, grid, dim3(S::NT), S::LDS_BYTES, s, ev.start, OAA ? nullptr : ev.stop, ys,
                                 bias, y, aux, p.prob.cout, p.coutp, p.prob.h, p.prob.w, p.T, p.P, p.th, p.tw, p.nt,
                                 p.ntp, ngroups, int(p.relu), int(pool), y_elems);
    if (e != hipSuccess || !OAA) return e;
    return launch_seam(p, aux, bias, y, s, ev.stop);
}

hipError_t launch_seam(const fftsplit_plan_s& p, const float* aux, const float* bias, float* y, hipStream_t s,
                       hipEvent_t stop) {
    // seam rows (columns): r in [0, h) with (r + P) mod T < 2P, counted as
    // u = r + P over [P, h + P) with u mod T < 2P
    const int T = p.T, P2 = 2 * p.P;
    auto below = [&](int n) { return (n / T) * (P2 < T ? P2 : T) + (n % T < P2 ? n % T : P2); };
    const int nsr = below(p.prob.h + p.P) - below(p.P);
    const int nsc = below(p.prob.w + p.P) - below(p.P);
    const long long count = (long long)nsr * p.prob.w + (long long)(p.prob.h - nsr) * nsc;
    const long long per_block = 256LL * kSeamPix;
    const long long bpp = count > 0 ? (count + per_block - 1) / per_block : 1;
    const long long blocks = bpp * p.prob.n * p.prob.cout;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    return launch_kernel(seam_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, nullptr, stop, aux, bias, y,
                         p.prob.cout, p.prob.h, p.prob.w, p.T, p.P, p.L, p.th, p.tw, p.ntp, int(p.relu), nsr, nsc,
                         int(bpp));
}

template <int L, int TG>
static hipError_t launch_inverse_L(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y,
                                   float* aux, hipStream_t s, const LaunchEvents& ev) {
    return p.oaa ? launch_inverse_v<L, TG, true>(p, ys, bias, y, aux, s, ev)
                 : launch_inverse_v<L, TG, false>(p, ys, bias, y, aux, s, ev);
}

hipError_t launch_inverse(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y, void* aux,
                          hipStream_t s, const LaunchEvents& ev) {
    float* a = static_cast<float*>(aux);
    if (p.oaa && !a) return hipErrorInvalidValue;
    if (p.L % 2) return launch_oaa_inverse(p, ys, bias, y, a, s, ev);
    if (p.inv_band) {
        switch (p.L) {
            case 8: return launch_inverse_band<8, 64, kBandNV8>(p, ys, bias, y, s, ev);
            case 16: return launch_inverse_band<16, 32, kBandNV16>(p, ys, bias, y, s, ev);
            case 32: return launch_inverse_band<32, 16, kBandNV32>(p, ys, bias, y, s, ev);
        }
        return hipErrorInvalidValue;
    }
    switch (p.L) {
        case 8: return launch_inverse_L<8, 64>(p, ys, bias, y, a, s, ev);
        case 16: return launch_inverse_L<16, 32>(p, ys, bias, y, a, s, ev);
        case 32: return launch_inverse_L<32, 16>(p, ys, bias, y, a, s, ev);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
