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
// so every operand fragment is 32 consecutive complex values of one input
// channel row, and every stored output row is 32 consecutive patches.
//
// The last two bins each hold two real bins (re, im) -- the four real bins
// of the two Hermitian columns, fftsplit.h -- whose products are taken
// component by component: Y = (sum Wr Xr, sum Wi Xi).
//
// With G3 the complex product takes three real products instead (Gauss):
//     P1 = Wr Xr, P2 = Wi Xi, P3 = (Wr + Wi)(Xr + Xi);  Y = (P1 - P2, P3 - P1 - P2)
// which cuts the matrix-core work by a quarter for two vector adds per
// operand fragment; the plan's default.
//
// Workgroup tile: BM output channels x BN patches of one bin, 4 waves in a
// WM x (4/WM) grid.  The input-channel loop runs in stages of KC channels.
// PF = 2 (the default where a tile has it): stages are loaded two ahead
// straight into three LDS stage buffers, one barrier per stage.  PF = 1:
// stage s+1 is loaded from memory into registers while stage s is
// multiplied out of LDS, then written to the other LDS buffer.  Inside a
// stage the operand fragments of the next channel pair are read from LDS
// while the current pair's MFMAs run.  The filter spectra, the bulk of the
// bytes, are loaded non-temporally where each block of them is read by one
// or two workgroups, so they do not evict the patch and output spectra; with XS (a
// single 64-channel output block, so every patch spectrum is read by one
// workgroup) the patch spectra are too, so that they do not evict the
// output spectra the inverse reads next.  The
// workgroups of one bin run on the same XCD, so the bin's patch spectra
// are fetched from HBM once and reused from L2, and the bins are dealt to
// the XCDs in turn, so that together they sweep the spectra in order.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

// s_waitcnt immediate that waits until at most n (< 64) vector memory
// instructions are outstanding and leaves the other counters alone (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int vmcnt_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// 16 bytes per lane from global memory straight into LDS: lane l writes
// LDS bytes [base + 16 l, base + 16 l + 16) with base the wave's LDS
// address (the low 32 bits of a generic pointer into LDS are its LDS
// offset).  Written as inline assembly rather than with the compiler's
// builtin: for the builtin the compiler cannot tell which LDS buffer a load
// fills and waits for all of them before every LDS read, which would
// serialise the stages loaded ahead; here the caller waits (s_waitcnt
// vmcnt) before the barrier that publishes a buffer.  One wait state
// separates the M0 write from the load.
template <bool NT>
__device__ __forceinline__ void lds_dma16(const void* g, const void* lds_wave_base) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane(unsigned(reinterpret_cast<uintptr_t>(lds_wave_base)));
    if constexpr (NT)
        asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(m0)
                     : "memory", "m0");
    else
        asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m0)
                     : "memory", "m0");
}

template <int BM, int BN, int KC, int WM>
struct ConShape {
    static constexpr int NT = 256;
    static constexpr int WN = 4 / WM;
    static constexpr int TM = BM / WM / 32;      // 32-row MFMA tiles per wave
    static constexpr int TN = BN / WN / 32;      // 32-col MFMA tiles per wave
    static constexpr int WE = KC * BM;           // W stage elements (complex)
    static constexpr int XE = KC * BN;           // X stage elements (complex)
    static constexpr int WL = WE / 2 / NT;       // 16-byte loads per thread per stage
    static constexpr int XL = XE / 2 / NT;
    static constexpr int LDS_BYTES = 2 * (WE + XE) * 8;
    static_assert(WM * WN == 4, "four waves");
    static_assert(TM >= 1 && TN >= 1 && WL >= 1 && XL >= 1, "tile shape");
    static_assert((WE / 2) % NT == 0 && (XE / 2) % NT == 0, "loads divide evenly");
};

// Writes a wave's TM x TN MFMA tiles of output spectra (rows from co_base,
// patches from t_base) in the patch-group-major layout: the 32 lanes of a
// row write 32 consecutive patches (32 / G runs of G, or half a run).
// With G3, Y = (P1 - P2, P3 - P1 - P2), except in the two slots of packed
// real bins, whose parts are P1 and P2 themselves.
template <int TM, int TN, bool G3>
__device__ __forceinline__ void store_output_tile(float2* __restrict__ ys, const floatx16 (&accR)[TM][TN],
                                                  const floatx16 (&accI)[TM][TN],
                                                  const floatx16 (&acc3)[G3 ? TM : 1][G3 ? TN : 1], int co_base,
                                                  int t_base, int f, int nbins, int ygroup, int ntp, int krow,
                                                  int col, bool packed) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int cb0 = co_base + i * 32;
            float2* yb = ys + yspec_offset(cb0, f, t_base + j * 32 + col, nbins, ygroup, ntp / ygroup);
            const size_t cstride = size_t(nbins) * ntp;   // next channel
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                // row ii = 8 (r / 4) + 4 krow + r % 4 of the 32
                const int ii = 8 * (r >> 2) + 4 * krow + (r & 3);
                float2* dst = yb + size_t(ii) * cstride;
                if (G3) {
                    const float p1 = accR[i][j][r], p2 = accI[i][j][r];
                    *dst = packed ? make_float2(p1, p2)
                                  : make_float2(p1 - p2, acc3[G3 ? i : 0][G3 ? j : 0][r] - p1 - p2);
                } else {
                    *dst = make_float2(accR[i][j][r], accI[i][j][r]);
                }
            }
        }
    }
}

// One input-channel stage (KC channels) of a wave's TM x TN MFMA tiles,
// from the stage buffer in LDS (W rows of BM channels, then X rows of BN
// patches).  The fragments of the next channel pair are read while the
// current pair is multiplied.
template <int BM, int BN, int KC, int TM, int TN, bool G3>
__device__ __forceinline__ void multiply_stage(const float2* stage, floatx16 (&accR)[TM][TN],
                                               floatx16 (&accI)[TM][TN],
                                               floatx16 (&acc3)[G3 ? TM : 1][G3 ? TN : 1], int krow, int col,
                                               int wm, int wn, bool packed) {
    const float2* sw = stage + krow * BM + wm * (TM * 32) + col;
    const float2* sx = stage + KC * BM + krow * BN + wn * (TN * 32) + col;
    float2 a[2][TM], b[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) a[0][i] = sw[i * 32];
#pragma unroll
    for (int j = 0; j < TN; ++j) b[0][j] = sx[j * 32];
#pragma unroll
    for (int kp = 0; kp < KC / 2; ++kp) {
        const int cur = kp & 1;
        if (kp + 1 < KC / 2) {
#pragma unroll
            for (int i = 0; i < TM; ++i) a[cur ^ 1][i] = sw[(2 * kp + 2) * BM + i * 32];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[cur ^ 1][j] = sx[(2 * kp + 2) * BN + j * 32];
        }
        // the next channel pair's fragment reads stay ahead of this
        // pair's matrix products
        __builtin_amdgcn_sched_barrier(0);
        if (G3) {
            float bs_[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j) bs_[j] = b[cur][j].x + b[cur][j].y;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const float ar = a[cur][i].x, ai = a[cur][i].y, as_ = ar + ai;
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    accR[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(ar, b[cur][j].x, accR[i][j], 0, 0, 0);
                    accI[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(ai, b[cur][j].y, accI[i][j], 0, 0, 0);
                    acc3[G3 ? i : 0][G3 ? j : 0] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                        as_, bs_[j], acc3[G3 ? i : 0][G3 ? j : 0], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                // a slot of two real bins: accR = sum Wr Xr, accI = sum Wi Xi
                const float ar = a[cur][i].x, ai = a[cur][i].y;
                const float a2 = packed ? ai : ar, nai = packed ? 0.f : -ai, ai4 = packed ? 0.f : ai;
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    accR[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(ar, b[cur][j].x, accR[i][j], 0, 0, 0);
                    accI[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a2, b[cur][j].y, accI[i][j], 0, 0, 0);
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    accR[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(nai, b[cur][j].y, accR[i][j], 0, 0, 0);
                    accI[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(ai4, b[cur][j].x, accI[i][j], 0, 0, 0);
                }
            }
        }
    }
}

template <int BM, int BN, int KC, int WM, bool G3, int PF, bool XS>
__global__ __launch_bounds__(256) void contract_kernel(const float2* __restrict__ xs, const float2* __restrict__ ws,
                                                       float2* __restrict__ ys, int cin, int coutp, int ntp,
                                                       int nbco, int nbt, int nbins, int ygroup, int npacked) {
    using S = ConShape<BM, BN, KC, WM>;
    constexpr int TM = S::TM, TN = S::TN;
    extern __shared__ float4 lds_raw[];   // max(PF + 1, 2) stage buffers

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / S::WN, wn = wave % S::WN;

    // Logical block lb = (bin, patch block, channel block), channel blocks
    // fastest.  The hardware deals workgroup i to XCD i % 8; the bins are
    // dealt to the XCDs in turn (bin f to XCD f % 8, its workgroups
    // consecutive there), so that a bin's workgroups share that XCD's L2
    // and the XCDs together sweep the bins in order.  Grids that the turns
    // do not divide keep one contiguous range of bins per XCD.
    const int per_bin = nbco * nbt;
    int lb;
    if (int(gridDim.x) % (kNumXcd * per_bin) == 0) {
        const int x = int(blockIdx.x) % kNumXcd, j = int(blockIdx.x) / kNumXcd;
        lb = ((j / per_bin) * kNumXcd + x) * per_bin + j % per_bin;
    } else {
        lb = xcd_logical_block(blockIdx.x, gridDim.x);
    }
    const int cbk = lb % nbco;
    const int rest = lb / nbco;
    const int tbk = rest % nbt;
    const int f = rest / nbt;
    // the last two bins (even L) are slots of two real bins each
    // (fftsplit.h): their products are taken component by component
    const bool packed = f >= nbins - npacked;
    const int co0 = cbk * BM;
    const int t0 = tbk * BN;

    const float4* wsrc = reinterpret_cast<const float4*>(ws + size_t(f) * cin * coutp + co0);
    // The filter spectra are streamed (non-temporal) when each block of them
    // is read by at most two workgroups (one or two patch blocks per bin):
    // the two run side by side on the bin's XCD, so the second still finds
    // the block in L2, and the last-level cache is spared the stream (VGG-16
    // layers at 28^2, 128 patches: up to 6 us each).  With more patch
    // blocks per bin the block has to stay in the caches.
    const bool w_once = nbt <= 2;
    const int wrow4 = coutp / 2;   // row pitch in float4
    // Patch spectra are channel-blocked (fftsplit.h): input channel ci of
    // bin f starts at spec_offset(ci, f, 0); within a block of 16 channels
    // the rows are ntp apart.
    auto xrow = [&](int ci) {
        return reinterpret_cast<const float4*>(xs + spec_offset(ci, f, t0, nbins, ntp));
    };

    // register sets for the stages loaded ahead (the second only with PF 2)
    typedef uint4 WRegs[S::WL];
    typedef uint4 XRegs[S::XL];
    WRegs wreg0, wreg1;
    XRegs xreg0, xreg1;
    // A stage that runs past cin reads its missing rows from row cin-1
    // (always in range) and store_stage writes zeros for them.  The loads
    // are never used before store_stage, so both kinds of stage leave them
    // in flight through the multiply.
    auto load_stage = [&](int k0, WRegs& wreg, XRegs& xreg) {
        const bool full = k0 + KC <= cin;
#pragma unroll
        for (int i = 0; i < S::WL; ++i) {
            const int e = i * S::NT + tid;
            const int ci = k0 + e / (BM / 2);
            const uint4* g = reinterpret_cast<const uint4*>(wsrc) + (full ? ci : min(ci, cin - 1)) * wrow4 + e % (BM / 2);
            wreg[i] = w_once ? load_stream_u4(g) : *g;
        }
#pragma unroll
        for (int i = 0; i < S::XL; ++i) {
            const int e = i * S::NT + tid;
            const int ci = k0 + e / (BN / 2);
            xreg[i] = reinterpret_cast<const uint4*>(xrow(full ? ci : min(ci, cin - 1)))[e % (BN / 2)];
        }
    };
    auto store_stage = [&](float2* stage, const WRegs& wreg, const XRegs& xreg, int k0) {
        uint4* sw = reinterpret_cast<uint4*>(stage);
        uint4* sx = reinterpret_cast<uint4*>(stage + S::WE);
        auto masked = [](uint4 v, bool keep) {
            const unsigned m = keep ? 0xffffffffu : 0u;
            return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
        };
        if (k0 + KC <= cin) {
#pragma unroll
            for (int i = 0; i < S::WL; ++i) sw[i * S::NT + tid] = wreg[i];
#pragma unroll
            for (int i = 0; i < S::XL; ++i) sx[i * S::NT + tid] = xreg[i];
        } else {
#pragma unroll
            for (int i = 0; i < S::WL; ++i) {
                const int e = i * S::NT + tid;
                sw[e] = masked(wreg[i], k0 + e / (BM / 2) < cin);
            }
#pragma unroll
            for (int i = 0; i < S::XL; ++i) {
                const int e = i * S::NT + tid;
                sx[e] = masked(xreg[i], k0 + e / (BN / 2) < cin);
            }
        }
    };

    // 4M: accR = sum Wr Xr - Wi Xi, accI = sum Wr Xi + Wi Xr.
    // 3M: accR = sum Wr Xr, accI = sum Wi Xi, acc3 = sum (Wr + Wi)(Xr + Xi);
    //     Y = (accR - accI, acc3 - accR - accI).
    floatx16 accR[TM][TN], accI[TM][TN], acc3[G3 ? TM : 1][G3 ? TN : 1];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                accR[i][j][r] = 0.f;
                accI[i][j][r] = 0.f;
                if (G3) acc3[G3 ? i : 0][G3 ? j : 0][r] = 0.f;
            }

    const int nstage = (cin + KC - 1) / KC;
    const int krow = lane >> 5;
    const int col = lane & 31;
    // the multiply of the stage held in LDS buffer `stage`
    auto multiply = [&](const float2* stage) {
        multiply_stage<BM, BN, KC, TM, TN, G3>(stage, accR, accI, acc3, krow, col, wm, wn, packed);
    };
    if constexpr (PF == 1) {
        float2* lds = reinterpret_cast<float2*>(lds_raw);   // [2][WE + XE]
        load_stage(0, wreg0, xreg0);
        store_stage(lds, wreg0, xreg0, 0);
        __syncthreads();
        for (int s = 0; s < nstage; ++s) {
            float2* cur = lds + (s & 1) * (S::WE + S::XE);
            float2* nxt = lds + ((s + 1) & 1) * (S::WE + S::XE);
            if (s + 1 < nstage) load_stage((s + 1) * KC, wreg0, xreg0);
            multiply(cur);
            if (s + 1 < nstage) store_stage(nxt, wreg0, xreg0, (s + 1) * KC);
            __syncthreads();
        }
    } else {
        // PF stages ahead, loaded straight into LDS (global_load_lds_dwordx4:
        // lane l of a wave writes the 16 bytes at the wave's LDS base + 16 l,
        // the layout store_stage writes), PF + 1 stage buffers in the dynamic
        // LDS.  The loop is unrolled by PF + 1, so the buffers are fixed at
        // every step; the wait for a stage's own loads and the barrier are
        // explicit (__syncthreads() would wait for every outstanding load,
        // the stages ahead included).
        constexpr int NB = PF + 1;
        float2* const lds = reinterpret_cast<float2*>(lds_raw);
        float2* const bufs[4] = {lds, lds + (S::WE + S::XE), lds + 2 * (S::WE + S::XE), lds + 3 * (S::WE + S::XE)};
        static_assert(NB <= 4, "at most four stage buffers");
        constexpr int LPS = S::WL + S::XL;   // memory instructions per stage and thread
        const int nfull = cin / KC;          // stages [0, nfull) are whole
        auto dma_stage = [&](int k0, float2* stage) {
            uint4* sw = reinterpret_cast<uint4*>(stage);
            uint4* sx = reinterpret_cast<uint4*>(stage + S::WE);
            const int wbase = tid & ~63;
#pragma unroll
            for (int i = 0; i < S::WL; ++i) {
                const int e = i * S::NT + tid;
                const uint4* g = reinterpret_cast<const uint4*>(wsrc) + (k0 + e / (BM / 2)) * wrow4 + e % (BM / 2);
                if (w_once) lds_dma16<true>(g, sw + i * S::NT + wbase);   // non-temporal, as load_stream_u4
                else lds_dma16<false>(g, sw + i * S::NT + wbase);
            }
#pragma unroll
            for (int i = 0; i < S::XL; ++i) {
                const int e = i * S::NT + tid;
                const uint4* g = reinterpret_cast<const uint4*>(xrow(k0 + e / (BN / 2))) + e % (BN / 2);
                lds_dma16<XS>(g, sx + i * S::NT + wbase);
            }
        };
        // full stage s in buffer `cur`; stage s + PF goes into `ahead` (the
        // buffer of stage s - 1, which every wave has finished once past the
        // barrier).  No register loads happen in this loop, so the compiler
        // has no loads of its own to wait for.
        auto step = [&](int s, float2* cur, float2* ahead) {
            // this stage's loads are done when at most those of the stages
            // issued after it remain (the memory counter retires in order)
            const int later = min(s + PF - 1, nfull - 1) - s;
            if (PF >= 3 && later >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_wait(2 * LPS));
            else if (later == 1) __builtin_amdgcn_s_waitcnt(vmcnt_wait(LPS));
            else __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
            asm volatile("s_barrier" ::: "memory");
            if (s + PF < nfull) dma_stage((s + PF) * KC, ahead);
            multiply(cur);
        };
#pragma unroll
        for (int d = 0; d < PF; ++d)
            if (d < nfull) dma_stage(d * KC, bufs[d]);
        for (int s0 = 0; s0 < nfull; s0 += NB) {
#pragma unroll
            for (int r = 0; r < NB; ++r)
                if (s0 + r < nfull) step(s0 + r, bufs[r], bufs[(r + PF) % NB]);
        }
        if (nfull < nstage) {
            // the partial last stage, through registers (masked rows), once
            // every wave is done with the buffers
            __syncthreads();
            load_stage(nfull * KC, wreg0, xreg0);
            store_stage(bufs[0], wreg0, xreg0, nfull * KC);
            __syncthreads();
            multiply(bufs[0]);
        }
    }

    store_output_tile<TM, TN, G3>(ys, accR, accI, acc3, co0 + wm * (TM * 32), t0 + wn * (TN * 32), f, nbins, ygroup,
                                  ntp, krow, col, packed);
}

template <int BM, int BN, int KC, int WM, bool G3 = false, int PF = 1, bool XS = false>
static hipError_t launch_contract_v(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                                    hipStream_t s, const LaunchEvents& ev) {
    using S = ConShape<BM, BN, KC, WM>;
    auto kern = contract_kernel<BM, BN, KC, WM, G3, PF, XS>;
    constexpr int lds = (PF > 1 ? PF + 1 : 2) * (S::WE + S::XE) * 8;
    static hipError_t attr = allow_dynamic_lds(kern, lds);
    if (attr != hipSuccess) return attr;
    if (p.coutp % BM != 0 || p.ntp % BN != 0) return hipErrorInvalidValue;
    const int nbco = p.coutp / BM, nbt = p.ntp / BN;
    const size_t nb = size_t(nbco) * nbt * p.bins;
    return launch_kernel(kern, dim3(unsigned(nb)), dim3(S::NT), lds, s, ev.start, ev.stop, xs, ws, ys,
                         p.prob.cin, p.coutp, p.ntp, nbco, nbt, p.bins, patch_group(p.L), packed_slots(p.L));
}

// The variants launch_contract dispatches (checked at plan time, so that a
// plan never names a tile without a kernel).
bool contract_variant_exists(int bm, int bn, int kc, int products) {
    const int v = bm * 1000000 + bn * 1000 + kc;
    if (bm <= 0 || bn <= 0 || kc <= 0) return false;
    if (products == 3) return v == 64064016 || v == 64064008 || v == 128064016 || v == 64128016 || v == 128032016;
    if (products == 4)
        return v == 64064016 || v == 64064032 || v == 128064016 || v == 128064032 || v == 64128016 ||
               v == 128128016 || v == 256064016 || v == 128032016;
    return false;
}

hipError_t launch_contract(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                           hipStream_t s, const LaunchEvents& ev) {
    const int v = p.con_bm * 1000000 + p.con_bn * 1000 + p.con_kc;
    if (p.con_products == 3) {
        switch (v) {
            case 64064016:
                if (p.con_prefetch == 2 && p.coutp == 64)
                    return launch_contract_v<64, 64, 16, 2, true, 2, true>(p, xs, ws, ys, s, ev);
                if (p.con_prefetch == 2) return launch_contract_v<64, 64, 16, 2, true, 2>(p, xs, ws, ys, s, ev);
                if (p.con_prefetch == 3) return launch_contract_v<64, 64, 16, 2, true, 3>(p, xs, ws, ys, s, ev);
                return launch_contract_v<64, 64, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 64064008:
                if (p.con_prefetch == 3 && p.coutp == 64)
                    return launch_contract_v<64, 64, 8, 2, true, 3, true>(p, xs, ws, ys, s, ev);
                if (p.con_prefetch == 3) return launch_contract_v<64, 64, 8, 2, true, 3>(p, xs, ws, ys, s, ev);
                if (p.con_prefetch == 2) return launch_contract_v<64, 64, 8, 2, true, 2>(p, xs, ws, ys, s, ev);
                return launch_contract_v<64, 64, 8, 2, true>(p, xs, ws, ys, s, ev);
            case 128064016:
                if (p.con_prefetch == 2) return launch_contract_v<128, 64, 16, 2, true, 2>(p, xs, ws, ys, s, ev);
                return launch_contract_v<128, 64, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 64128016:
                if (p.con_prefetch == 2) return launch_contract_v<64, 128, 16, 2, true, 2>(p, xs, ws, ys, s, ev);
                return launch_contract_v<64, 128, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 128032016:
                if (p.con_prefetch == 2) return launch_contract_v<128, 32, 16, 4, true, 2>(p, xs, ws, ys, s, ev);
                return launch_contract_v<128, 32, 16, 4, true>(p, xs, ws, ys, s, ev);
        }
    } else {
        switch (v) {
            case 64064016: return launch_contract_v<64, 64, 16, 2>(p, xs, ws, ys, s, ev);
            case 64064032: return launch_contract_v<64, 64, 32, 2>(p, xs, ws, ys, s, ev);
            case 128064016: return launch_contract_v<128, 64, 16, 2>(p, xs, ws, ys, s, ev);
            case 128064032: return launch_contract_v<128, 64, 32, 2>(p, xs, ws, ys, s, ev);
            case 64128016: return launch_contract_v<64, 128, 16, 2>(p, xs, ws, ys, s, ev);
            case 128128016: return launch_contract_v<128, 128, 16, 2>(p, xs, ws, ys, s, ev);
            case 256064016: return launch_contract_v<256, 64, 16, 4>(p, xs, ws, ys, s, ev);
            case 128032016: return launch_contract_v<128, 32, 16, 4>(p, xs, ws, ys, s, ev);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
