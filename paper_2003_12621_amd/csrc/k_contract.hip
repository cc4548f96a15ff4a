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
// WM x (4/WM) grid.  The input-channel loop runs in stages of KC channels;
// stage s+1 is loaded from memory into registers while stage s is
// multiplied out of LDS, then written to the other LDS buffer (one barrier
// per stage).  Inside a stage the operand fragments of the next channel
// pair are read from LDS while the current pair's MFMAs run.  The filter
// spectra, the bulk of the bytes and each read once, are loaded
// non-temporally so they do not evict the patch and output spectra.  The channel
// blocks of one bin are consecutive logical workgroups on the same XCD, so
// the bin's patch spectra are fetched from HBM once and reused from L2.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

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

template <int BM, int BN, int KC, int WM, bool G3>
__global__ __launch_bounds__(256) void contract_kernel(const float2* __restrict__ xs, const float2* __restrict__ ws,
                                                       float2* __restrict__ ys, int cin, int coutp, int ntp,
                                                       int nbco, int nbt, int nbins, int ygroup, int npacked) {
    using S = ConShape<BM, BN, KC, WM>;
    constexpr int TM = S::TM, TN = S::TN;
    extern __shared__ float4 lds_raw[];
    float2* lds = reinterpret_cast<float2*>(lds_raw);   // [2][WE + XE]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / S::WN, wn = wave % S::WN;

    const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
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
    const int wrow4 = coutp / 2;   // row pitch in float4
    // Patch spectra are channel-blocked (fftsplit.h): input channel ci of
    // bin f starts at spec_offset(ci, f, 0); within a block of 16 channels
    // the rows are ntp apart.
    auto xrow = [&](int ci) {
        return reinterpret_cast<const float4*>(xs + spec_offset(ci, f, t0, nbins, ntp));
    };

    uint4 wreg[S::WL], xreg[S::XL];
    // A full stage is loaded as is; only a stage that runs past cin reads
    // its missing rows from row cin-1 (always in range) and zeroes them.
    // The branch is uniform, and in the full case the loaded registers are
    // first used when the stage is written to LDS after the MFMAs, so the
    // loads stay in flight during the multiply.
    auto load_stage = [&](int k0) {
        if (k0 + KC <= cin) {
#pragma unroll
            for (int i = 0; i < S::WL; ++i) {
                const int e = i * S::NT + tid;
                wreg[i] = load_stream_u4(reinterpret_cast<const uint4*>(wsrc) + (k0 + e / (BM / 2)) * wrow4 +
                                         e % (BM / 2));
            }
#pragma unroll
            for (int i = 0; i < S::XL; ++i) {
                const int e = i * S::NT + tid;
                xreg[i] = reinterpret_cast<const uint4*>(xrow(k0 + e / (BN / 2)))[e % (BN / 2)];
            }
        } else {
#pragma unroll
            for (int i = 0; i < S::WL; ++i) {
                const int e = i * S::NT + tid;
                const int ci = k0 + e / (BM / 2);
                const uint4 v = load_stream_u4(reinterpret_cast<const uint4*>(wsrc) + min(ci, cin - 1) * wrow4 +
                                               e % (BM / 2));
                const unsigned m = ci < cin ? 0xffffffffu : 0u;
                wreg[i] = make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
            }
#pragma unroll
            for (int i = 0; i < S::XL; ++i) {
                const int e = i * S::NT + tid;
                const int ci = k0 + e / (BN / 2);
                const uint4 v = reinterpret_cast<const uint4*>(xrow(min(ci, cin - 1)))[e % (BN / 2)];
                const unsigned m = ci < cin ? 0xffffffffu : 0u;
                xreg[i] = make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
            }
        }
    };
    auto store_stage = [&](int buf) {
        uint4* sw = reinterpret_cast<uint4*>(lds + buf * (S::WE + S::XE));
        uint4* sx = reinterpret_cast<uint4*>(lds + buf * (S::WE + S::XE) + S::WE);
#pragma unroll
        for (int i = 0; i < S::WL; ++i) sw[i * S::NT + tid] = wreg[i];
#pragma unroll
        for (int i = 0; i < S::XL; ++i) sx[i * S::NT + tid] = xreg[i];
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
    load_stage(0);
    store_stage(0);
    __syncthreads();

    const int krow = lane >> 5;
    const int col = lane & 31;
    for (int s = 0; s < nstage; ++s) {
        const int buf = s & 1;
        if (s + 1 < nstage) load_stage((s + 1) * KC);
        const float2* sw = lds + buf * (S::WE + S::XE) + krow * BM + wm * (TM * 32) + col;
        const float2* sx = lds + buf * (S::WE + S::XE) + S::WE + krow * BN + wn * (TN * 32) + col;
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
        if (s + 1 < nstage) store_stage(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            // output spectra, patch-group-major: the 32 lanes of a row write
            // 32 consecutive patches (32 / G runs of G, or half a run)
            const int cb0 = co0 + wm * (TM * 32) + i * 32;
            float2* yb = ys + yspec_offset(cb0, f, t0 + wn * (TN * 32) + j * 32 + col, nbins, ygroup,
                                           ntp / ygroup);
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

template <int BM, int BN, int KC, int WM, bool G3 = false>
static hipError_t launch_contract_v(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                                    hipStream_t s, const LaunchEvents& ev) {
    using S = ConShape<BM, BN, KC, WM>;
    auto kern = contract_kernel<BM, BN, KC, WM, G3>;
    static hipError_t attr = allow_dynamic_lds(kern, S::LDS_BYTES);
    if (attr != hipSuccess) return attr;
    if (p.coutp % BM != 0 || p.ntp % BN != 0) return hipErrorInvalidValue;
    const int nbco = p.coutp / BM, nbt = p.ntp / BN;
    const size_t nb = size_t(nbco) * nbt * p.bins;
    return launch_kernel(kern, dim3(unsigned(nb)), dim3(S::NT), S::LDS_BYTES, s, ev.start, ev.stop, xs, ws, ys,
                         p.prob.cin, p.coutp, p.ntp, nbco, nbt, p.bins, patch_group(p.L), packed_slots(p.L));
}

hipError_t launch_contract(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                           hipStream_t s, const LaunchEvents& ev) {
    const int v = p.con_bm * 1000000 + p.con_bn * 1000 + p.con_kc;
    if (p.con_products == 3) {
        switch (v) {
            case 64064016: return launch_contract_v<64, 64, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 128064016: return launch_contract_v<128, 64, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 64128016: return launch_contract_v<64, 128, 16, 2, true>(p, xs, ws, ys, s, ev);
            case 128032016: return launch_contract_v<128, 32, 16, 4, true>(p, xs, ws, ys, s, ev);
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
