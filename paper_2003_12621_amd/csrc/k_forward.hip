// Forward patch transform (Section 3.1: split, eq. 4; pad, eqs. 5-6; the
// transform of each padded patch, first factor of eq. 9).
//
// A workgroup owns TG consecutive patches of one input channel, with L/2
// threads per patch:
//   1. gather: the TG windows are read cooperatively into LDS, one window
//      row per L consecutive lanes.  Overlap-save: the L x L window that
//      starts P rows/cols before the tile, zeros outside the image.
//      Overlap-add: the T x T tile, zeros up to L x L.  Every load is issued
//      unconditionally from a clamped in-image address and masked after, so
//      all of a thread's loads are in flight together;
//   2. row pass: thread j transforms rows 2j and 2j+1 packed as one complex
//      sequence (real part row 2j, imaginary part row 2j+1) and separates
//      the two half spectra (bins 0..L/2) into LDS;
//   3. column pass: thread j >= 1 transforms column k2 = j; thread 0 the two
//      real-valued columns k2 = 0 and k2 = L/2 packed as one complex
//      sequence, then separates them;
//   4. each bin goes to X[f][c][t]: the TG lanes with consecutive patch
//      index write one contiguous 8*TG-byte segment.
// Workgroups are laid out so that each accelerator die (XCD) processes a
// contiguous run of patch groups of one channel: the windows' halo rows and
// columns shared between neighbouring groups then hit in that die's L2.
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
                                                               int nt, int ntp, int ngroups) {
    using S = FwdShape<L, TG>;
    constexpr int H2 = S::H2, WP = S::WP, WTS = S::WTS, TP = S::TP, TTS = S::TTS;
    constexpr int RPI = 64 / L;               // window rows per wave-wide load
    constexpr int TPW = TG / (S::NT / 64);    // patches per wave
    extern __shared__ float4 lds_raw[];
    float* win = reinterpret_cast<float*>(lds_raw);
    float2* tb = reinterpret_cast<float2*>(lds_raw);

    const int tid = threadIdx.x;
    const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
    const int g = lb % ngroups;
    const int c = lb / ngroups;
    const int t0 = g * TG;

    // 1. gather.  Wave wv reads the windows of its own TPW patches; each
    // wave-wide load covers RPI consecutive window rows of one patch (L
    // consecutive lanes per row), so the patch geometry is wave-uniform.
    // Each patch gets a buffer descriptor whose range ends where its valid
    // rows end; rows before it wrap to huge offsets, and lanes whose column
    // is outside the image (or, for overlap-add, beyond the tile) use an
    // always-out-of-range offset -- all of those read 0.
    {
        const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int lane = tid & 63;
        const int q = lane % L;
        const int mr = lane / L;
        const unsigned row_step = unsigned(RPI * w * 4);
        float v[S::NLOAD];
#pragma unroll
        for (int pi = 0; pi < TPW; ++pi) {
            const int t = t0 + wv * TPW + pi;
            const float* base = x;
            unsigned bytes = 0, voff = kOutOfRange;   // padding patches read nothing
            if (t < nt) {
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
#pragma unroll
        for (int pi = 0; pi < TPW; ++pi) {
            const int u = wv * TPW + pi;
#pragma unroll
            for (int ri = 0; ri < L / RPI; ++ri) win[u * WTS + (ri * RPI + mr) * WP + q] = v[pi * (L / RPI) + ri];
        }
    }
    __syncthreads();

    // 2. row pass (j fastest across lanes)
    {
        const int j = tid % H2;
        const int u = tid / H2;
        float2 z[L];
        const float* r0 = win + u * WTS + 2 * j * WP;
#pragma unroll
        for (int q = 0; q < L; ++q) z[q] = make_float2(r0[q], r0[WP + q]);
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
        fft<L, false>(cz);
        // X[f][c][t0 + u]: per-lane byte offset, per-bin stride as the
        // scalar offset (always in range).
        const BufRsrc rx = make_rsrc(xs, unsigned(size_t(cin) * ntp * 8 * stored_bins(L)));
        const unsigned bs8 = unsigned(cin) * unsigned(ntp) * 8u;
        const unsigned voff = unsigned(c * ntp + t0 + u) * 8u;
        if (j == 0) {
#pragma unroll
            for (int k1 = 0; k1 <= H2; ++k1) {
                float2 a, b;
                split_two_real(cz[k1], cz[(L - k1) % L], a, b);
                buf_store_f32x2(a, rx, voff, unsigned(bin_col0(L, k1)) * bs8);
                buf_store_f32x2(b, rx, voff, unsigned(bin_colh(L, k1)) * bs8);
            }
        } else {
            const unsigned vj = voff + unsigned(bin_mid(L, 0, j)) * bs8;
#pragma unroll
            for (int k1 = 0; k1 < L; ++k1) buf_store_f32x2(cz[k1], rx, vj, unsigned(k1) * bs8);
        }
    }
}

template <int L, int TG, bool OAA>
static hipError_t launch_forward_v(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                   const LaunchEvents& ev) {
    using S = FwdShape<L, TG>;
    auto kern = forward_kernel<L, TG, OAA>;
    static hipError_t attr = allow_dynamic_lds(kern, S::LDS_BYTES);
    if (attr != hipSuccess) return attr;
    const int ngroups = p.ntp / TG;
    const dim3 grid(unsigned(ngroups) * unsigned(p.prob.cin));
    return launch_kernel(kern, grid, dim3(S::NT), S::LDS_BYTES, s, ev.start, ev.stop, x, xs, p.prob.cin, p.prob.h,
                         p.prob.w, p.T, p.P, p.th, p.tw, p.nt, p.ntp, ngroups);
}

template <int L, int TG>
static hipError_t launch_forward_L(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                                   const LaunchEvents& ev) {
    return p.oaa ? launch_forward_v<L, TG, true>(p, x, xs, s, ev) : launch_forward_v<L, TG, false>(p, x, xs, s, ev);
}

hipError_t launch_forward(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                          const LaunchEvents& ev) {
    switch (p.L) {
        case 8: return launch_forward_L<8, 64>(p, x, xs, s, ev);
        case 16: return launch_forward_L<16, 32>(p, x, xs, s, ev);
        case 32: return launch_forward_L<32, 16>(p, x, xs, s, ev);
    }
    return hipErrorInvalidValue;
}

}  // namespace fftsplit
