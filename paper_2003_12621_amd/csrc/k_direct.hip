// Direct spatial cross-correlation on the fp32 matrix cores: the spatial
// convolution the paper compares the split method against (Section 2,
// eq. 1; Section 4, Table 1 and Fig. 4).
//
//     y[n][co][p] = b[co] + sum_{ci, u, v} w[co][ci][u][v] * x[n][ci][py + u - P][px + v - P]
//
// as an implicit GEMM: rows = output channels, columns = output pixels
// (flattened over image, row, column), reduction over (u, v, ci).  The
// filters are rearranged once per layer into Wd[u][v][ci16][coutp]
// (direct_weights_kernel), so that a stage of 16 input channels of one tap
// (u, v) is a contiguous 16 x 64 block; the input operand of a stage is
// gathered from x with the tap's shift, zero outside the image.
//
// Workgroup tile: 64 output channels x 64 pixels, 4 waves of 32 x 32, one
// v_mfma_f32_32x32x2_f32 per two input channels (operand layout as in the
// contraction kernel).  Stages are double-buffered through registers and
// LDS: the next stage's loads are in flight while the current one is
// multiplied.  Bias and ReLU are applied in the epilogue.
#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

namespace fftsplit {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kDirBM = 64, kDirBN = 64, kDirKC = 16;

// w [cout][cin][k][k] -> Wd[k*k][cin16][coutp], zero for padded channels.
__global__ __launch_bounds__(256) void direct_weights_kernel(const float* __restrict__ w, float* __restrict__ wd,
                                                             int cin, int cout, int cin16, int coutp, int kk) {
    const size_t total = size_t(kk) * cin16 * coutp;
    const size_t idx = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int co = int(idx % coutp);
    const size_t rest = idx / coutp;
    const int ci = int(rest % cin16);
    const int uv = int(rest / cin16);
    wd[idx] = (co < cout && ci < cin) ? w[(size_t(co) * cin + ci) * kk + uv] : 0.f;
}

__global__ __launch_bounds__(256) void direct_kernel(const float* __restrict__ x, const float* __restrict__ wd,
                                                     const float* __restrict__ bias, float* __restrict__ y, int n,
                                                     int cin, int h, int w, int cout, int coutp, int k, int relu,
                                                     unsigned x_bytes, int nbco, int npix) {
    constexpr int BM = kDirBM, BN = kDirBN, KC = kDirKC, NT = 256;
    __shared__ float lds[2][KC * (BM + BN)];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
    const int cbk = lb % nbco;
    const int pbk = lb / nbco;
    const int co0 = cbk * BM;
    const int p0 = pbk * BN;
    const int P = k / 2;
    const int hw = h * w;
    const int cin16 = (cin + KC - 1) / KC * KC;
    const int nchunk = cin16 / KC;
    const int nstage = k * k * nchunk;

    // B loads: thread -> (row kr = tid / 16, 4 consecutive pixels at 4 * (tid % 16))
    const int kr = tid >> 4;
    const int pj = (tid & 15) * 4;
    int pimg[4], py[4], px[4];
    bool pok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int p = p0 + pj + e;
        pok[e] = p < npix;
        const int pp = pok[e] ? p : 0;
        pimg[e] = pp / hw;
        const int r = pp - pimg[e] * hw;
        py[e] = r / w;
        px[e] = r - py[e] * w;
    }
    const BufRsrc rxs = make_rsrc(x, x_bytes);
    // A loads: thread -> (row tid / 16, 4 consecutive channels at 4 * (tid % 16))
    const float* wsrc = wd + co0 + (tid & 15) * 4;

    float4 areg;
    float breg[4];
    auto load_stage = [&](int s) {
        const int uv = s / nchunk;
        const int c0 = (s - uv * nchunk) * KC;
        const int u = uv / k, v = uv - u * k;
        areg = *reinterpret_cast<const float4*>(wsrc + (size_t(uv) * cin16 + c0 + kr) * coutp);
        const int ci = c0 + kr;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int yy = py[e] + u - P, xx = px[e] + v - P;
            const bool ok = pok[e] && ci < cin && unsigned(yy) < unsigned(h) && unsigned(xx) < unsigned(w);
            const unsigned off = ok ? unsigned(((pimg[e] * cin + ci) * h + yy) * w + xx) * 4u : kOutOfRange;
            breg[e] = buf_load_f32(rxs, off, 0);
        }
    };
    auto store_stage = [&](int buf) {
        *reinterpret_cast<float4*>(&lds[buf][kr * BM + (tid & 15) * 4]) = areg;
        *reinterpret_cast<float4*>(&lds[buf][KC * BM + kr * BN + pj]) =
            make_float4(breg[0], breg[1], breg[2], breg[3]);
    };

    floatx16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const int krow = lane >> 5;
    const int col = lane & 31;

    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int s = 0; s < nstage; ++s) {
        const int buf = s & 1;
        if (s + 1 < nstage) load_stage(s + 1);
        const float* sa = &lds[buf][krow * BM + wm * 32 + col];
        const float* sb = &lds[buf][KC * BM + krow * BN + wn * 32 + col];
        float a[KC / 2], b[KC / 2];
#pragma unroll
        for (int kp = 0; kp < KC / 2; ++kp) {
            a[kp] = sa[2 * kp * BM];
            b[kp] = sb[2 * kp * BN];
        }
#pragma unroll
        for (int kp = 0; kp < KC / 2; ++kp) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[kp], b[kp], acc, 0, 0, 0);
        if (s + 1 < nstage) store_stage(buf ^ 1);
        __syncthreads();
    }

    // epilogue: D[i][j], register r: i = 8 (r / 4) + 4 krow + r % 4, j = col
    const int p = p0 + wn * 32 + col;
    if (p < npix) {
        const int img = p / hw;
        const int rem = p - img * hw;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int co = co0 + wm * 32 + 8 * (r >> 2) + 4 * krow + (r & 3);
            if (co < cout) {
                float v = acc[r] + (bias ? bias[co] : 0.f);
                if (relu) v = vmax(v, 0.f);
                y[(size_t(img) * cout + co) * hw + rem] = v;
            }
        }
    }
}

size_t direct_wspec_bytes(const fftsplit_plan_s& p) {
    return size_t(p.prob.k) * p.prob.k * round_up_block(p.prob.cin) * p.coutp * 4;
}

hipError_t launch_direct_weights(const fftsplit_plan_s& p, const float* w, float* wd, hipStream_t s) {
    const int kk = p.prob.k * p.prob.k;
    const size_t total = size_t(kk) * round_up_block(p.prob.cin) * p.coutp;
    const unsigned blocks = unsigned((total + 255) / 256);
    hipLaunchKernelGGL(direct_weights_kernel, dim3(blocks), dim3(256), 0, s, w, wd, p.prob.cin, p.prob.cout,
                       round_up_block(p.prob.cin), p.coutp, kk);
    return hipGetLastError();
}

hipError_t launch_direct(const fftsplit_plan_s& p, const float* x, const float* wd, const float* bias, float* y,
                         hipStream_t s, const LaunchEvents& ev) {
    const int npix = p.prob.n * p.prob.h * p.prob.w;
    const int nbco = p.coutp / kDirBM;
    const int nbp = (npix + kDirBN - 1) / kDirBN;
    const unsigned x_bytes = unsigned(size_t(p.prob.n) * p.prob.cin * p.prob.h * p.prob.w * 4);
    return launch_kernel(direct_kernel, dim3(unsigned(nbco) * unsigned(nbp)), dim3(256), 0, s, ev.start, ev.stop, x,
                         wd, bias, y, p.prob.n, p.prob.cin, p.prob.h, p.prob.w, p.prob.cout, p.coutp, p.prob.k,
                         int(p.relu), x_bytes, nbco, npix);
}

}  // namespace fftsplit
