// Forward patch transform (Section 3.1: split, eq. 4; pad, eqs. 5-6; the
// transform of each padded patch, first factor of eq. 9).
//
// Work item: TG consecutive patches of one input channel.  A workgroup
// (TG * L/2 threads, L/2 per patch) processes `ipw` consecutive items and
// software-pipelines them: the window loads of item i+1 are issued into
// registers before item i is transformed, so they are in flight during
// item i's transforms and stores.  Per item:
//   1. the gathered windows (registers) go to LDS, one window row per L
//      consecutive lanes.  Overlap-save: the L x L window that starts P
//      rows/cols before the tile, zeros outside the image.  Overlap-add:
//      the T x T tile, zeros up to L x L.  Every load is issued
//      unconditionally from a clamped in-image address and masked after,
//      so all of a thread's loads are in flight together;
//   2. row pass: thread j transforms rows 2j and 2j+1 packed as one complex
//      sequence (real part row 2j, imaginary part row 2j+1) and separates
//      the two half spectra (bins 0..L/2) into LDS;
//   3. column pass: thread j >= 1 transforms column k2 = j; thread 0 the two
//      real-valued columns k2 = 0 and k2 = L/2 packed as one complex
//      sequence, then separates them;
//   4. each bin goes to the patch spectra (channel-blocked, fftsplit.h):
//      the TG lanes with consecutive patch index write one contiguous
//      8*TG-byte segment.
// Items are numbered channel-major (consecutive items are neighbouring
// patch groups of one channel) and each accelerator die (XCD) receives a
// contiguous range of workgroups, so the halo rows and columns shared by
// neighbouring groups hit in that die's L2.
#include "band.hpp"
#include "fftsplit_internal.hpp"
#include "fft_regs.hpp"
#include "launch_util.hpp"

namespace fftsplit {

template <int L, int TG>
struct FwdShape {
    static constexpr int H2 = L / 2;
    static constexpr int NT = TG * H2;            // threads
    static constexpr int WP = L + 1;              // window row pitch (floats)
    static constexpr int WTS = L * WP + 1;        // window patch stride (floats)
    static constexpr int TP = H2 + 1;             // half-spectrum row pitch (float2)
    static constexpr int TTS = L * TP + 2;        // half-spectrum patch stride (float2)
    static constexpr int NLOAD = TG * L * L / NT; // window elements per thread (= 2L)
    static constexpr int WIN_BYTES = TG * WTS * 4;
    static constexpr int TB_BYTES = TG * TTS * 8;
    static constexpr int LDS_BYTES = WIN_BYTES > TB_BYTES ? WIN_BYTES : TB_BYTES;
    static_assert(NT % L == 0, "thread count must be a multiple of L");
};

template <int L, int TG, bool OAA>
__global__ __launch_bounds__(TG * (L / 2)) void forward_kernel(const float* __restrict__ x, float2* __restrict__ xs,
                                                               int cin, int h, int w, int T, int P, int th, int tw,
                                                               int nt, int ntp, int ngroups, int nitems, int ipw) {
    using S = FwdShape<L, TG>;
    constexpr int H2 = S::H2, WP = S::WP, WTS = S::WTS, TP = S::TP, TTS = S::TTS;
    constexpr int RPI = 64 / L;               // window rows per wave-wide load
    constexpr int TPW = TG / (S::NT / 64);    // patches per wave
    extern __shared__ float4 lds_raw[];
    float* win = reinterpret_cast<float*>(lds_raw);
    float2* tb = reinterpret_cast<float2*>(lds_raw);

    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int q = lane % L;
    const int mr = lane / L;
    const unsigned row_step = unsigned(RPI * w * 4);
    const BufRsrc rx = make_rsrc(xs, unsigned(size_t(round_up_block(cin)) * ntp * 8 * stored_bins(L)));
    const unsigned bs8 = unsigned(kChanBlock) * unsigned(ntp) * 8u;   // bin stride (channel-blocked)

    // Gather of one item into registers.  Wave wv reads the windows of its
    // own TPW patches; each wave-wide load covers RPI consecutive window
    // rows of one patch (L consecutive lanes per row), so the patch
    // geometry is wave-uniform.  Each patch gets a buffer descriptor whose
    // range ends where its valid rows end; rows before it wrap to huge
    // offsets, and lanes whose column is outside the image (or, for
    // overlap-add, beyond the tile) use an always-out-of-range offset -- all
    // of those read 0.
    float v[S::NLOAD];
    // item < 0 issues the same loads with an empty range (they return 0
    // without touching memory), which keeps the pipelined loop free of a
    // branch around its prefetch.
    auto gather = [&](int item) {
        const int c = item / ngroups;
        const int t0 = (item - c * ngroups) * TG;
#pragma unroll
        for (int pi = 0; pi < TPW; ++pi) {
            const int t = t0 + wv * TPW + pi;
            const float* base = x;
            unsigned bytes = 0, voff = kOutOfRange;   // padding patches read nothing
            if (item >= 0 && t < nt) {
                const int b = t % tw;
                const int rest = t / tw;
                const int a = rest % th;
                const int img = rest / th;
                const int plane = (img * cin + c) * h * w;
                if (OAA) {
                    // rows a*T .. min(a*T + T, h) - 1 of the plane, cols b*T + q for q < T
                    base = x + plane + a * T * w;
                    bytes = unsigned(min(T, h - a * T) * w * 4);
                    const int col = b * T + q;
                    if (q < T && col < w) voff = unsigned((mr * w + col) * 4);
                } else {
                    // rows a*T - P + m of the plane; rows < 0 wrap out of range
                    base = x + plane;
                    bytes = unsigned(h * w * 4);
                    const int col = b * T - P + q;
                    if (unsigned(col) < unsigned(w)) voff = unsigned(((a * T - P + mr) * w + col) * 4);
                }
            }
            const BufRsrc rs = make_rsrc(base, bytes);
#pragma unroll
            for (int ri = 0; ri < L / RPI; ++ri)
                v[pi * (L / RPI) + ri] = buf_load_f32(rs, voff + unsigned(ri) * row_step, 0);
        }
    };

    const int lw = xcd_logical_block(blockIdx.x, gridDim.x);
    const int ibeg = lw * ipw;
    const int iend = min(ibeg + ipw, nitems);

    auto process = [&](int item) {
        const int c = item / ngroups;
        const int t0 = (item - c * ngroups) * TG;

        // 1. this item's windows to LDS (waits for its loads only)
#pragma unroll
        for (int pi = 0; pi < TPW; ++pi) {
            const int u = wv * TPW + pi;
#pragma unroll
            for (int ri = 0; ri < L / RPI; ++ri) win[u * WTS + (ri * RPI + mr) * WP + q] = v[pi * (L / RPI) + ri];
        }
        __syncthreads();
        // the next item's loads stay in flight through steps 2-4
        gather(item + 1 < iend ? item + 1 : -1);

        // 2. row pass (j fastest across lanes)
        {
            const int j = tid % H2;
            const int u = tid / H2;
            float2 z[L];
            const float* r0 = win + u * WTS + 2 * j * WP;
#pragma unroll
            for (int qq = 0; qq < L; ++qq) z[qq] = make_float2(r0[qq], r0[WP + qq]);
            __syncthreads();  // the half-spectrum buffer reuses the window's LDS
            fft<L, false>(z);
            float2* ra = tb + u * TTS + 2 * j * TP;
#pragma unroll
            for (int k = 0; k <= H2; ++k) {
                float2 a, b;
                split_two_real(z[k], z[(L - k) % L], a, b);
                ra[k] = a;
                ra[TP + k] = b;
            }
        }
        __syncthreads();

        // 3. column pass (patch index fastest across lanes) and 4. store
        {
            const int u = tid % TG;
            const int j = tid / TG;
            const float2* cb = tb + u * TTS;
            float2 cz[L];
            if (j == 0) {
#pragma unroll
                for (int m = 0; m < L; ++m) cz[m] = make_float2(cb[m * TP].x, cb[m * TP + H2].x);
            } else {
#pragma unroll
                for (int m = 0; m < L; ++m) cz[m] = cb[m * TP + j];
            }
            __syncthreads();  // every read of the spectra is done before the next item's windows land
            fft<L, false>(cz);
            // (c, f, t0 + u): per-lane byte offset, per-bin stride as the
            // scalar offset (always in range).
            const unsigned voff = unsigned(spec_offset(c, 0, t0 + u, stored_bins(L), ntp)) * 8u;
            if (j == 0) {
                // the real bins (k1 = 0, L/2) of both columns share two slots
                float2 a0, b0, ah, bh;
                split_two_real(cz[0], cz[0], a0, b0);
                split_two_real(cz[H2], cz[H2], ah, bh);
                buf_store_f32x2(make_float2(a0.x, ah.x), rx, voff, unsigned(bin_real_a(L)) * bs8);
                buf_store_f32x2(make_float2(b0.x, bh.x), rx, voff, unsigned(bin_real_b(L)) * bs8);
#pragma unroll
                for (int k1 = 1; k1 < H2; ++k1) {
                    float2 a, b;
                    split_two_real(cz[k1], cz[L - k1], a, b);
                    buf_store_f32x2(a, rx, voff, unsigned(bin_col0(L, k1)) * bs8);
                    buf_store_f32x2(b, rx, voff, unsigned(bin_colh(L, k1)) * bs8);
                }
            } else {
                const unsigned vj = voff + unsigned(bin_mid(L, 0, j)) * bs8;
#pragma unroll
                for (int k1 = 0; k1 < L; ++k1) buf_store_f32x2(cz[k1], rx, vj, unsigned(k1) * bs8);
            }
        }
    };

    // The first item is peeled off the loop so that, inside the loop, the
    // wait for an item's loads leaves the previous item's stores in flight
    // (the memory counter is in order, and the loads were issued first).
    if (ibeg < iend) {
        gather(ibeg);
        process(ibeg);
        for (int item = ibeg + 1; item < iend; ++item) process(item);
    }
}


// Overlap-save forward transform reading whole row bands (width a multiple
// of 4, at most 256).  Same work items, transforms and output layout as
// forward_kernel; what changes is how the input arrives and how items
// overlap:
//   * input: the item's band (band.hpp: the tile rows of its patches plus
//     the P-row halo, as whole image rows -- a few contiguous runs of
//     memory) is read with 16-byte loads, lanes along each row, and kept in
//     LDS with `co` zero columns on the left and zeros up to the pitch `bp`
//     on the right; a zero row (slot `zslot`) stands in for rows outside
//     the image.  The row pass cuts each patch's L x L window out of it;
//   * pipelining: the band loads of a workgroup's next item are issued into
//     registers before the current item is transformed, and its spectra
//     are stored straight from the column pass, so loads, transforms and
//     stores of neighbouring items overlap; `sweep` (set by the plan where
//     input and spectra exceed the last-level cache) spaces a workgroup's
//     items a grid apart, so the workgroups sweep input and spectra in
//     order, otherwise a workgroup runs a contiguous run of items; with XS
//     (an input larger than the last-level cache) the input is read
//     non-temporally, so that it does not take the cache's room from the
//     spectra the contraction reads next;
//   * LDS banks (32 four-byte banks): the row pass pairs rows j and
//     j + L/2 (not 2j and 2j+1); with the odd band pitch the L/2 row-pass
//     lanes of a patch, which read rows j, hit distinct banks, and with the
//     odd row stride of the half spectra (L/2+1 float2) its row writes do
//     too; the patch stride of the half spectra (band_half_stride) puts
//     the column-pass reads of the patches and columns that share a bank
//     sweep in distinct banks; the band is written with 4-byte stores (odd
//     rows are not 8-byte aligned).
template <int L, int TG, int NV, bool XS>
__global__ __launch_bounds__(TG * (L / 2), 2) void forward_band_kernel(
    const float* __restrict__ x, float2* __restrict__ xs, int cin, int h, int w, int T, int P, int th, int tw, int nt,
    int ntp, int ngroups, int nitems, int ipw, int bp, int co, int zslot, unsigned x_bytes, float inv_h, float inv_tw,
    float inv_th, int sweep) {
    using S = FwdShape<L, TG>;
    constexpr int NT = S::NT, NW = NT / 64, H2 = S::H2, TP = S::TP;
    constexpr int TTS = band_half_stride(L, TG);  // half-spectrum patch stride (float2)
    constexpr int F = stored_bins(L);
    extern __shared__ float4 lds_raw[];
    float* band = reinterpret_cast<float*>(lds_raw);
    float2* tb = reinterpret_cast<float2*>(lds_raw);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int w4 = w >> 2;
    const int rpi = 64 / w4;                 // band rows per wave-wide load
    const int lrow = lane / w4;              // this lane's row within a load
    const int c4 = lane - lrow * w4;         // this lane's float4 column
    const BufRsrc rxin = make_rsrc(x, x_bytes);
    const BufRsrc rx = make_rsrc(xs, unsigned(size_t(round_up_block(cin)) * ntp * 8 * F));
    const unsigned bs8 = unsigned(kChanBlock) * unsigned(ntp) * 8u;   // bin stride (channel-blocked)
    // An opaque copy of a per-lane value: offsets derived from it are
    // recomputed inside the item loop instead of being hoisted out of it
    // and held in registers for the whole loop.
    auto opaque = [](int v) {
        asm volatile("" : "+v"(v));
        return v;
    };

    // sweep: workgroup lw runs items lw, lw + gridDim.x, ...; otherwise a
    // contiguous run of ipw items, in XCD-aware order
    const int lw = sweep ? int(blockIdx.x) : xcd_logical_block(blockIdx.x, gridDim.x);
    const int istep = sweep ? int(gridDim.x) : 1;
    const int ibeg = sweep ? lw : lw * ipw;
    const int iend = sweep ? nitems : min(ibeg + ipw, nitems);

    float4 v[NV];
    // Slot k of this lane is band row slot0 + k * slot_step.
    const int slot0 = wv * rpi + lrow;
    const int slot_step = NW * rpi;
    // Issue the band loads of `item` (item < 0: empty loads that return 0
    // without touching memory).  Band slot `sl` holds image row
    // (r0 + sl) mod h of image img0 + (r0 + sl) / h (slots run through the
    // images' rows in order), so its byte offset in x is
    //   4 * (((img0 * cin + c) * h + r0) * w + sl * w) + q * 4 * (cin - 1) * h * w
    // with q = (r0 + sl) / h.  Along this lane's slots q and the row
    // advance incrementally; the sl * w part of each step is a uniform
    // scalar offset.
    const unsigned cross4 = unsigned(cin - 1) * unsigned(h) * unsigned(w) * 4u;
    const int dq = slot_step / h, dr = slot_step - dq * h;
    auto load_band = [&](int item) {
        int c = 0, t0 = 0;
        BandGeom g{0, 0, 0, 0, 0, 0};
        if (item >= 0) {
            c = item / ngroups;
            t0 = (item - c * ngroups) * TG;
            g = band_geom(t0, TG, nt, h, T, P, th, tw);
        }
        const int sl0 = opaque(slot0);
        const int x0 = sl0 + g.r0;
        int q = div_small(x0, h, inv_h);
        int r = x0 - q * h;
        unsigned voff = unsigned((((g.img0 * cin + c) * h + g.r0) * w) * 4) + unsigned(sl0 * w * 4) +
                        unsigned(16 * c4) + unsigned(q) * cross4;
        const bool lane_ok = lrow < rpi;
        const unsigned dq_off = unsigned(dq) * cross4;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const bool ok = lane_ok && sl0 + k * slot_step < g.slots;
            v[k] = buf_load_f32x4<XS ? kCacheStream : kCacheDefault>(rxin, ok ? voff : kOutOfRange,
                                                                     unsigned(k * slot_step * w * 4));
            r += dr;
            voff += dq_off;
            const bool carry = r >= h;
            r -= carry ? h : 0;
            voff += carry ? cross4 : 0u;
        }
    };
    // The loaded band and its zero padding into LDS.
    auto write_band = [&](const BandGeom& g) {
        const int sl0 = opaque(slot0);
        float* dst = band + sl0 * bp + co + 4 * c4;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            if (lrow < rpi && sl0 + k * slot_step < g.slots) {
                float* d = dst + k * slot_step * bp;
                d[0] = v[k].x;
                d[1] = v[k].y;
                d[2] = v[k].z;
                d[3] = v[k].w;
            }
        }
        // columns [0, co) and [co + w, bp) of every slot, and the zero slot
        const int pw = bp - w;
        const float inv_pw = 1.0f / float(pw);
        for (int e = tid; e < g.slots * pw; e += NT) {
            const int sl = div_small(e, pw, inv_pw);
            const int k = e - sl * pw;
            band[sl * bp + (k < co ? k : w + k)] = 0.f;
        }
        for (int e = tid; e < bp; e += NT) band[zslot * bp + e] = 0.f;
    };

    auto process = [&](int item) {
        const int c = item / ngroups;
        const int t0 = (item - c * ngroups) * TG;
        const BandGeom g = band_geom(t0, TG, nt, h, T, P, th, tw);
        write_band(g);
        __syncthreads();
        // the next item's loads stay in flight through this item's transforms
        load_band(item + istep < iend ? item + istep : -1);

        // row pass (j fastest across lanes): rows j and j + L/2 of patch u's
        // window (rows a stride of L/2 apart, not adjacent ones, so that with
        // the odd band pitch and half-spectrum row stride the 16 lanes of a
        // patch spread over all banks)
        {
            const int j = tid % H2;
            const int u = tid / H2;
            const int t = t0 + u;
            int s0 = zslot, s1 = zslot, cb = co;
            if (t < nt) {
                const int tr = div_small(t, tw, inv_tw);
                const int b = t - tr * tw;
                const int img = div_small(tr, th, inv_th);
                const int a = tr - img * th;
                // the band's rows run through the images in order: image row
                // r of image img0 + sg sits at slot sg * h + r - r0
                const int r = a * T - P + j;
                const int sb = __umul24(img - g.img0, h) - g.r0 + r;
                s0 = unsigned(r) < unsigned(h) ? sb : zslot;
                s1 = unsigned(r + H2) < unsigned(h) ? sb + H2 : zslot;
                cb = co + b * T - P;
            }
            const float* r0 = band + s0 * bp + cb;
            const float* r1 = band + s1 * bp + cb;
            float2 z[L];
#pragma unroll
            for (int qq = 0; qq < L; ++qq) z[qq] = make_float2(r0[qq], r1[qq]);
            __syncthreads();  // the half-spectrum buffer reuses the band's LDS
            fft<L, false>(z);
            // A real row's spectrum is real at k = 0 and k = L/2: those two
            // values share slot 0 as (re, im), already the packed sequence
            // (column 0 + i * column L/2) the column pass transforms there.
            float2* ra = tb + opaque(u * TTS + j * TP);
            ra[0] = make_float2(z[0].x, z[H2].x);
            ra[H2 * TP] = make_float2(z[0].y, z[H2].y);
#pragma unroll
            for (int k = 1; k < H2; ++k) {
                float2 a, b;
                split_two_real(z[k], z[L - k], a, b);
                ra[k] = a;
                ra[H2 * TP + k] = b;
            }
        }
        __syncthreads();

        // column pass (patch index fastest across lanes).  Lane j >= 1
        // transforms column k2 = j; lane j = 0 the two real columns k2 = 0
        // and k2 = L/2, which the row pass left packed in slot 0 as one
        // complex sequence (column 0 + i * column L/2).  Both kinds of lane
        // run one instruction stream -- separating the two real spectra is
        // a select -- so no wave executes two paths.  Each bin goes to
        // (c, f, t0 + u): the TG lanes of consecutive patches write one
        // contiguous 8*TG-byte segment.
        {
            const int u = tid % TG;
            const int j = tid / TG;
            const bool j0 = j == 0;
            const float2* ca = tb + opaque(u * TTS) + j;
            float2 cz[L];
#pragma unroll
            for (int m = 0; m < L; ++m) cz[m] = ca[m * TP];
            __syncthreads();  // the next item's band reuses the half-spectrum LDS
            fft<L, false>(cz);
            // Lane j >= 1 stores bins (k1, j) and (k1 + L/2, j); lane 0 the
            // complex bins k1 in [1, L/2-1] of the two real columns, and at
            // k1 = 0 their four real bins packed into two slots.
            const unsigned lane8 = unsigned(spec_offset(c, 0, t0 + u, F, ntp)) * 8u;
            const unsigned va0 = lane8 + unsigned(j0 ? bin_real_a(L) : bin_mid(L, 0, j)) * bs8;
            const unsigned vb0 = lane8 + unsigned(j0 ? bin_real_b(L) : bin_mid(L, H2, j)) * bs8;
            const unsigned va = lane8 + unsigned(j0 ? bin_col0(L, 1) - 1 : bin_mid(L, 0, j)) * bs8;
            const unsigned vb = lane8 + unsigned(j0 ? bin_colh(L, 1) - 1 : bin_mid(L, H2, j)) * bs8;
            {
                float2 sa0, sb0, sah, sbh;
                split_two_real(cz[0], cz[0], sa0, sb0);
                split_two_real(cz[H2], cz[H2], sah, sbh);
                buf_store_f32x2(j0 ? make_float2(sa0.x, sah.x) : cz[0], rx, va0, 0);
                buf_store_f32x2(j0 ? make_float2(sb0.x, sbh.x) : cz[H2], rx, vb0, 0);
            }
#pragma unroll
            for (int k1 = 1; k1 < H2; ++k1) {
                float2 sa, sb;
                split_two_real(cz[k1], cz[L - k1], sa, sb);
                buf_store_f32x2(j0 ? sa : cz[k1], rx, va, unsigned(k1) * bs8);
                buf_store_f32x2(j0 ? sb : cz[k1 + H2], rx, vb, unsigned(k1) * bs8);
            }
        }
    };

    // The first item is peeled off the loop so that, inside the loop, the
    // wait for an item's band leaves the previous item's stores in flight
    // (the memory counter is in order, and the loads were issued first).
    if (ibeg < iend) {
        load_band(ibeg);
        process(ibeg);
        for (int item = ibeg + istep; item < iend; item += istep) process(item);
    }
}

template <int L, int TG, bool OAA>
static hipError_t launch_forward_v(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                   const LaunchEvents& ev) {
    using S = FwdShape<L, TG>;
    auto kern = forward_kernel<L, TG, OAA>;
    static hipError_t attr = allow_dynamic_lds(kern, S::LDS_BYTES);
    if (attr != hipSuccess) return attr;
    static int per_cu = resident_blocks(kern, S::NT, S::LDS_BYTES);
    const int ngroups = p.ntp / TG;
    const int nitems = ngroups * p.prob.cin;
    const int ipw = items_per_workgroup(nitems, p.cus * per_cu);
    const dim3 grid(unsigned((nitems + ipw - 1) / ipw));
    return launch_kernel(kern, grid, dim3(S::NT), S::LDS_BYTES, s, ev.start, ev.stop, x, xs, p.prob.cin, p.prob.h,
                         p.prob.w, p.T, p.P, p.th, p.tw, p.nt, p.ntp, ngroups, nitems, ipw);
}

template <int L, int TG>
static hipError_t launch_forward_L(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                   const LaunchEvents& ev) {
    return p.oaa ? launch_forward_v<L, TG, true>(p, x, xs, s, ev) : launch_forward_v<L, TG, false>(p, x, xs, s, ev);
}

template <int L, int TG, int NV, bool XS>
static hipError_t launch_forward_band_v(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                      const LaunchEvents& ev) {
    using S = FwdShape<L, TG>;
    auto kern = forward_band_kernel<L, TG, NV, XS>;
    const int lds = p.fwd_lds;
    if (lds > 64 * 1024) {
        const hipError_t attr = allow_dynamic_lds(kern, lds);
        if (attr != hipSuccess) return attr;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kern), S::NT, lds) !=
            hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    const int ngroups = p.ntp / TG;
    const int nitems = ngroups * p.prob.cin;
    const int ipw = items_per_workgroup(nitems, p.cus * per_cu);
    const dim3 grid(unsigned((nitems + ipw - 1) / ipw));
    const unsigned x_bytes = unsigned(size_t(p.prob.n) * p.prob.cin * p.prob.h * p.prob.w * 4);
    return launch_kernel(kern, grid, dim3(S::NT), unsigned(lds), s, ev.start, ev.stop, x, xs, p.prob.cin, p.prob.h,
                         p.prob.w, p.T, p.P, p.th, p.tw, p.nt, p.ntp, ngroups, nitems, ipw, p.fwd_bp, p.fwd_co,
                         p.fwd_zslot, x_bytes, 1.0f / float(p.prob.h), 1.0f / float(p.tw), 1.0f / float(p.th),
                         p.fwd_sweep ? 1 : 0);
}

// XS where the input exceeds the last-level cache (plan fwd_stream): the
// input is read non-temporally, so that it does not evict the spectra the
// contraction reads next.
template <int L, int TG, int NV>
static hipError_t launch_forward_band(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                      const LaunchEvents& ev) {
    return p.fwd_stream ? launch_forward_band_v<L, TG, NV, true>(p, x, xs, s, ev)
                       : launch_forward_band_v<L, TG, NV, false>(p, x, xs, s, ev);
}

hipError_t launch_forward(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                          const LaunchEvents& ev) {
    if (p.L % 2) return launch_oaa_forward(p, x, xs, s, ev);
    if (p.fwd_band) {
        switch (p.L) {
            case 8: return launch_forward_band<8, forward_group(8), kBandNV8>(p, x, xs, s, ev);
            case 16: return launch_forward_band<16, forward_group(16), kBandNV16>(p, x, xs, s, ev);
            case 32: return launch_forward_band<32, forward_group(32), kBandNV32>(p, x, xs, s, ev);
        }
        return hipErrorInvalidValue;
    }
    switch (p.L) {
        case 8: return launch_forward_L<8, forward_group(8)>(p, x, xs, s, ev);
        case 16: return launch_forward_L<16, forward_group(16)>(p, x, xs, s, ev);
        case 32: return launch_forward_L<32, forward_group(32)>(p, x, xs, s, ev);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
