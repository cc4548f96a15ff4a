// Internal declarations shared by the host library and the kernel files.
#pragma once

#include <cstddef>
#include <string>

#include <hip/hip_runtime.h>

#include "../../include/fftsplit.h"

#define FFTSPLIT_EXPORT extern "C" __attribute__((visibility("default")))

struct fftsplit_plan_s {
    fftsplit_problem_t prob;
    int device;                 // HIP ordinal, or -1 for an architecture-only plan
    int cus;                    // compute units of the device (256 for an architecture-only plan)
    char arch[64];
    int T, L, P;                // tile, FFT size, K/2
    int th, tw, nt, ntp;        // tile grid, tiles, padded tiles
    int bins, coutp;            // stored bins, padded output channels
    bool oaa, bias, relu, pool;
    size_t wspec_bytes;
    size_t xspec_off, xspec_bytes, yspec_off, yspec_bytes, aux_off, aux_bytes;
    size_t ws_bytes;
    // contraction kernel variant: tile BM x BN, KC channels per stage, and
    // 3 (Gauss) or 4 real products per complex multiply-add; con_prefetch
    // stages loaded ahead of the one being multiplied (1 to 3)
    int con_bm, con_bn, con_kc, con_products, con_prefetch;
    // overlap-save band variant of the forward transform (band.hpp):
    // used if fwd_band; LDS row pitch, left zero columns, zero-row slot and
    // dynamic LDS bytes; fwd_sweep: items a grid apart instead of a
    // contiguous run per workgroup; fwd_stream: the input read
    // non-temporally
    bool fwd_band, fwd_sweep, fwd_stream;
    int fwd_bp, fwd_co, fwd_zslot, fwd_lds;
    // overlap-save band variant of the inverse transform: used if
    // inv_band; LDS pitch of the output band and dynamic LDS bytes
    bool inv_band;
    int inv_obp, inv_lds;
    // FFTSPLIT_MAXPOOL: pooled inside the overlap-save inverse's store
    // phase (band or general kernel) if pool_fused, else the inverse writes
    // the unpooled output to the workspace at pre_off and a pooling pass
    // follows
    bool pool_fused;
    size_t pre_off, pre_bytes;
    // inputs of at most 4 (L = 8) or 3 (L = 16) channels (overlap-save,
    // band inverse):
    // conv2d sums the channels inside the inverse and skips the contraction
    bool fuse_cin;
    // the cost model's terms for the chosen L (fftsplit_plan_info_t)
    double model_con_flops, model_xfer_bytes, model_seconds;
};

namespace fftsplit {

// Granularity of the contraction's output tiles (patches x channels).
constexpr int kTileGranule = 64;
constexpr int kCoutGranule = 64;
// Patches are padded to 64, or to 32 where the transforms' patch groups
// allow it (L = 16, 32) and the output channels fill 128-wide tiles: the
// contraction then runs 128 x 32 tiles, which halves the padding of layers
// with few patches (a 14 x 14 image at T = 14 is one patch).
constexpr int kTileGranuleSmall = 32;

// Patches per work item of the forward/inverse transforms (L/2 threads
// each), by FFT size; the odd sizes of the OaAConv configuration transform
// one patch per thread and group patches in 64s.
__host__ __device__ constexpr int patch_group(int L) {
    return L % 2 ? 64 : (L == 8 ? 64 : (L == 16 ? 32 : 16));
}
// Patches per work item of the forward transform (L/2 threads each).  At
// L = 32 it is half the output-spectra group: 128-thread workgroups of 35 KB
// of LDS, four per compute unit, whose barriers span two waves (forward
// 22.5-23.6 -> 20.9-22.4 us on the 16x256x56^2 layer, warm).
__host__ __device__ constexpr int forward_group(int L) { return L == 32 ? 8 : patch_group(L); }

// Patch stride (float2) of the half spectra in the band transforms, for
// work items of TG patches: L rows of L/2+1 bins plus a pad that spreads the
// column pass over the LDS banks.  There, 16 consecutive lanes (one bank
// sweep of 8-byte accesses over 32 four-byte banks) hold min(TG, 16)
// patches u and 16 / min(TG, 16) columns j, at float2 index u * stride + j;
// with L (L/2 + 1) a multiple of 16 at L = 16 and 32, a pad of 16 / TG for
// TG < 16 and of 1 otherwise puts them in distinct bank pairs.
__host__ __device__ constexpr int band_half_stride(int L, int TG) {
    return L * (L / 2 + 1) + (TG < 16 ? 16 / TG : 1);
}

// Band loads per thread (16 bytes each) the band variant of the forward
// transform holds in registers, by FFT size.
constexpr int kBandNV8 = 8;
constexpr int kBandNV16 = 8;
constexpr int kBandNV32 = 16;

// Patch and output spectra are channel-blocked (fftsplit.h):
// [c / 16][bin][c % 16][patch], so the bins of one channel lie 16 * ntp
// elements apart.  Element offset of (channel c, bin f, patch t):
constexpr int kChanBlock = 16;
__host__ __device__ inline size_t spec_offset(int c, int f, int t, int bins, int ntp) {
    return ((size_t(c / kChanBlock) * bins + f) * kChanBlock + c % kChanBlock) * size_t(ntp) + t;
}
__host__ __device__ constexpr int round_up_block(int c) { return (c + kChanBlock - 1) / kChanBlock * kChanBlock; }

// Output spectra are patch-group-major (fftsplit.h): [c][t / G][bin][t % G]
// with G = patch_group(L), so one inverse work item (channel c, patches
// [gG, gG + G)) reads one contiguous run of bins * G elements.  The
// contraction, which is bound by its matrix products, writes them as
// G-element runs instead.  Element offset of (channel c, bin f, patch t):
__host__ __device__ inline size_t yspec_offset(int c, int f, int t, int bins, int G, int ngroups) {
    return ((size_t(c) * ngroups + t / G) * bins + f) * size_t(G) + t % G;
}

// Stored frequency bins of an L x L real transform: L*L/2 (layout in
// fftsplit.h).  Bins with k2 in [1, L/2-1] (all k1) are stored as they are;
// of the columns k2 = 0 and k2 = L/2, which are Hermitian in k1, the
// complex bins k1 in [1, L/2-1] are stored, and their four real bins
// (k1, k2 in {0, L/2}) share two slots: real_a = (S(0,0), S(L/2,0)),
// real_b = (S(0,L/2), S(L/2,L/2)) as (re, im).
//
// Odd L (the OaAConv configuration, L = 2K - 1): no column is real, only
// the bin (0, 0); (L*L+1)/2 slots, none packed:
//   f = (k2-1)*L + k1      S(k1, k2)  for k2 in [1, (L-1)/2], k1 in [0, L)
//   f = (L-1)/2*L + k1     S(k1, 0)   for k1 in [0, (L-1)/2]
__host__ __device__ constexpr int stored_bins(int L) { return L % 2 ? (L * L + 1) / 2 : L * L / 2; }
// slots at the end that each hold two real bins (multiplied part by part)
__host__ __device__ constexpr int packed_slots(int L) { return L % 2 ? 0 : 2; }
__host__ __device__ constexpr int bin_odd_col0(int L, int k1) { return (L / 2) * L + k1; }
__host__ __device__ constexpr int bin_mid(int L, int k1, int k2) { return (k2 - 1) * L + k1; }
// complex bins of the real columns, k1 in [1, L/2-1]
__host__ __device__ constexpr int bin_col0(int L, int k1) { return L * (L / 2 - 1) + k1 - 1; }
__host__ __device__ constexpr int bin_colh(int L, int k1) { return L * (L / 2 - 1) + L / 2 - 1 + k1 - 1; }
// the two slots holding pairs of real bins
__host__ __device__ constexpr int bin_real_a(int L) { return L * L / 2 - 2; }
__host__ __device__ constexpr int bin_real_b(int L) { return L * L / 2 - 1; }

// Thread-local error detail for fftsplit_last_error().
void set_error(const std::string& msg);
fftsplit_status_t fail(fftsplit_status_t st, const std::string& msg);

// Makes the plan's device current for the duration of a call.
class DeviceGuard {
  public:
    explicit DeviceGuard(int dev) {
        ok_ = hipGetDevice(&prev_) == hipSuccess;
        if (ok_ && prev_ != dev) ok_ = hipSetDevice(dev) == hipSuccess;
        changed_ = ok_ && prev_ != dev;
    }
    ~DeviceGuard() {
        if (changed_) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }

  private:
    int prev_ = 0;
    bool ok_ = false, changed_ = false;
};

// fftsplit_conv2d in two parts (api.cpp): the checks of every argument but
// the workspace, and the launch sequence into a workspace of at least
// plan->ws_bytes bytes on the plan's device, which must be current.
fftsplit_status_t check_conv2d_args(fftsplit_plan_t plan, const float* x, const void* wspec, const float* bias,
                                    const float* y);
fftsplit_status_t enqueue_conv2d(fftsplit_plan_t plan, const float* x, const void* wspec, const float* bias, float* y,
                                 void* workspace, hipStream_t stream);

// Kernel launchers (one per .hip file); return hipSuccess or the launch
// error.  `ev` optionally times the launch sequence (see launch_util.hpp).
struct LaunchEvents;
hipError_t launch_weights(const fftsplit_plan_s& p, const float* w, float2* wspec, hipStream_t s,
                          const LaunchEvents& ev);
hipError_t launch_forward(const fftsplit_plan_s& p, const float* x, float2* xspec, hipStream_t s,
                          const LaunchEvents& ev);
hipError_t launch_contract(const fftsplit_plan_s& p, const float2* xspec, const float2* wspec, float2* yspec,
                           hipStream_t s, const LaunchEvents& ev);
// whether launch_contract has a kernel for tile bm x bn, stages of kc and
// 3 or 4 real products per complex multiply-add
bool contract_variant_exists(int bm, int bn, int kc, int products);
hipError_t launch_inverse(const fftsplit_plan_s& p, const float2* yspec, const float* bias, float* y, void* aux,
                          hipStream_t s, const LaunchEvents& ev);
hipError_t launch_maxpool(const float* x, float* y, int n, int c, int h, int w, hipStream_t s,
                          hipEvent_t stop = nullptr);
// OaAConv configuration (odd L = 2K - 1, T = K, overlap-add): k_oaa.hip
hipError_t launch_oaa_forward(const fftsplit_plan_s& p, const float* x, float2* xs, hipStream_t s,
                              const LaunchEvents& ev);
hipError_t launch_oaa_inverse(const fftsplit_plan_s& p, const float2* ys, const float* bias, float* y, float* aux,
                              hipStream_t s, const LaunchEvents& ev);
// the band inverse with the per-bin channel sum for plans with fuse_cin:
// reads the patch spectra xs and the filter spectra ws, not output spectra
hipError_t launch_inverse_fused(const fftsplit_plan_s& p, const float2* xs, const float2* ws, const float* bias,
                                float* y, hipStream_t s, const LaunchEvents& ev);
// overlap-add seams from the per-patch L x L results in aux (k_inverse.hip)
hipError_t launch_seam(const fftsplit_plan_s& p, const float* aux, const float* bias, float* y, hipStream_t s,
                       hipEvent_t stop);
size_t direct_wspec_bytes(const fftsplit_plan_s& p);
hipError_t launch_direct_weights(const fftsplit_plan_s& p, const float* w, float* wd, hipStream_t s);
hipError_t launch_direct(const fftsplit_plan_s& p, const float* x, const float* wd, const float* bias, float* y,
                         hipStream_t s, const LaunchEvents& ev);

}  // namespace fftsplit
