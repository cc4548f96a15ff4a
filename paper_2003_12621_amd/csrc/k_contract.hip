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
// Workgroup tile: BM output channels x BN patches of one bin, 4 waves in a
// 2 x 2 grid.  The input-channel loop runs in stages of KC channels; stage
// s+1 is loaded from memory into registers while stage s is multiplied out
// of LDS, then written to the other LDS buffer (one barrier per stage).
// The channel blocks of one bin are consecutive logical workgroups on the
// same XCD, so the bin's patch spectra are fetched from HBM once and reused
// from that die's L2.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

template <int BM, int BN, int KC>
struct ConShape {
    static constexpr int NT = 256;
    static constexpr int TM = BM / 64;           // 32-row MFMA tiles per wave (2 waves along co)
    static constexpr int TN = BN / 64;           // 32-col MFMA tiles per wave (2 waves along t)
    static constexpr int WE = KC * BM;           // W stage elements (complex)
    static constexpr int XE = KC * BN;           // X stage elements (complex)
    static constexpr int WL = WE / 2 / NT;       // 16-byte loads per thread per stage
    static constexpr int XL = XE / 2 / NT;
    static constexpr int LDS_BYTES = 2 * (WE + XE) * 8;
    static_assert(TM >= 1 && TN >= 1 && WL >= 1 && XL >= 1, "tile shape");
    static_assert((WE / 2) % NT == 0 && (XE / 2) % NT == 0, "loads divide evenly");
};

template <int BM, int BN, int KC>
__global__ __launch_bounds__(256) void contract_kernel(const float2* __restrict__ xs, const float2* __restrict__ ws,
                                                       float2* __restrict__ ys, int cin, int coutp, int ntp,
                                                       int nbco, int nbt) {
    using S = ConShape<BM, BN, KC>;
    extern __shared__ float4 lds_raw[];
    float2* lds = reinterpret_cast<float2*>(lds_raw);   // [2][WE + XE]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
    const int cbk = lb % nbco;
    const int rest = lb / nbco;
    const int tbk = rest % nbt;
    const int f = rest / nbt;
    const int co0 = cbk * BM;
    const int t0 = tbk * BN;

    const float4* wsrc = reinterpret_cast<const float4*>(ws + size_t(f) * cin * coutp + co0);
    const float4* xsrc = reinterpret_cast<const float4*>(xs + size_t(f) * cin * ntp + t0);
    const int wrow4 = coutp / 2, xrow4 = ntp / 2;   // row pitch in float4

    float4 wreg[S::WL], xreg[S::XL];
    auto load_stage = [&](int k0) {
#pragma unroll
        for (int i = 0; i < S::WL; ++i) {
            const int e = i * S::NT + tid;
            const int kk = e / (BM / 2), c2 = e % (BM / 2);
            const int ci = k0 + kk;
            const float4 v = wsrc[size_t(min(ci, cin - 1)) * wrow4 + c2];
            wreg[i] = ci < cin ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < S::XL; ++i) {
            const int e = i * S::NT + tid;
            const int kk = e / (BN / 2), c2 = e % (BN / 2);
            const int ci = k0 + kk;
            const float4 v = xsrc[size_t(min(ci, cin - 1)) * xrow4 + c2];
            xreg[i] = ci < cin ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    auto store_stage = [&](int buf) {
        float4* sw = reinterpret_cast<float4*>(lds + buf * (S::WE + S::XE));
        float4* sx = reinterpret_cast<float4*>(lds + buf * (S::WE + S::XE) + S::WE);
#pragma unroll
        for (int i = 0; i < S::WL; ++i) sw[i * S::NT + tid] = wreg[i];
#pragma unroll
        for (int i = 0; i < S::XL; ++i) sx[i * S::NT + tid] = xreg[i];
    };

    floatx16 accR[S::TM][S::TN], accI[S::TM][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                accR[i][j][r] = 0.f;
                accI[i][j][r] = 0.f;
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
        const float2* sw = lds + buf * (S::WE + S::XE) + wm * (S::TM * 32) + col;
        const float2* sx = lds + buf * (S::WE + S::XE) + S::WE + wn * (S::TN * 32) + col;
#pragma unroll
        for (int kk = 0; kk < KC; kk += 2) {
            float2 a[S::TM], b[S::TN];
#pragma unroll
            for (int i = 0; i < S::TM; ++i) a[i] = sw[(kk + krow) * BM + i * 32];
#pragma unroll
            for (int j = 0; j < S::TN; ++j) b[j] = sx[(kk + krow) * BN + j * 32];
#pragma unroll
            for (int i = 0; i < S::TM; ++i) {
                const float nai = -a[i].y;
#pragma unroll
                for (int j = 0; j < S::TN; ++j) {
                    accR[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i].x, b[j].x, accR[i][j], 0, 0, 0);
                    accR[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(nai, b[j].y, accR[i][j], 0, 0, 0);
                    accI[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i].x, b[j].y, accI[i][j], 0, 0, 0);
                    accI[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i].y, b[j].x, accI[i][j], 0, 0, 0);
                }
            }
        }
        if (s + 1 < nstage) store_stage(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < S::TM; ++i) {
#pragma unroll
        for (int j = 0; j < S::TN; ++j) {
            float2* yb = ys + (size_t(f) * coutp + co0 + wm * (S::TM * 32) + i * 32) * ntp + t0 +
                         wn * (S::TN * 32) + j * 32 + col;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int ii = 8 * (r >> 2) + 4 * krow + (r & 3);
                yb[size_t(ii) * ntp] = make_float2(accR[i][j][r], accI[i][j][r]);
            }
        }
    }
}

template <int BM, int BN, int KC>
static hipError_t launch_contract_v(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                                    hipStream_t s) {
    using S = ConShape<BM, BN, KC>;
    auto kern = contract_kernel<BM, BN, KC>;
    static hipError_t attr = allow_dynamic_lds(kern, S::LDS_BYTES);
    if (attr != hipSuccess) return attr;
    const int nbco = p.coutp / BM, nbt = p.ntp / BN;
    const size_t nb = size_t(nbco) * nbt * p.bins;
    hipLaunchKernelGGL(kern, dim3(unsigned(nb)), dim3(S::NT), S::LDS_BYTES, s, xs, ws, ys, p.prob.cin, p.coutp, p.ntp,
                       nbco, nbt);
    return hipGetLastError();
}

hipError_t launch_contract(const fftsplit_plan_s& p, const float2* xs, const float2* ws, float2* ys,
                           hipStream_t s) {
    if (p.coutp % 128 == 0) return launch_contract_v<128, 64, 16>(p, xs, ws, ys, s);
    return launch_contract_v<64, 64, 16>(p, xs, ws, ys, s);
}

}  // namespace fftsplit
