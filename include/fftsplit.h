/*
 * fftsplit.h -- C ABI of the split-FFT 2-D convolution library for AMD
 * MI355X (gfx950).
 *
 * Method: Chitsaz et al., "Acceleration of Convolutional Neural Network Using
 * FFT-Based Split Convolutions" (arXiv:2003.12621), Section 3.1.  A stride-1
 * 'same' convolution layer (CNN cross-correlation, odd K x K kernel, K//2
 * zeros of padding) is computed by
 *   1. splitting each input plane into T x T patches (eq. 4),
 *   2. padding each patch to L x L, L = T + K - 1 (eqs. 5-6),
 *   3. a 2-D real FFT of every padded patch, and of every zero-padded filter
 *      (eq. 8, done once per layer by fftsplit_transform_weights),
 *   4. the entry-wise product of patch and filter spectra (eq. 9), summed
 *      over input channels: per frequency bin a Cin -> Cout complex matrix
 *      product batched over patches,
 *   5. an inverse FFT per (patch, output channel), crop and concatenation of
 *      the valid T x T tile (eq. 10 and the text after it) -- or, with
 *      FFTSPLIT_OVERLAP_ADD, zero-padded patches whose L x L results are
 *      overlap-added (the discipline of Section 2, Fig. 1, at tile size T),
 *   6. optional bias and ReLU, fused into the inverse stage.
 *
 * Result: y = relu?(conv2d(x, w, bias, stride=1, padding=K//2)) with
 * PyTorch's cross-correlation convention, in fp32.
 *
 * Conventions for every entry point:
 *   - Tensors are fp32 and densely packed (C order).  Pointers marked
 *     "device" are device addresses on the plan's device; "host" pointers
 *     are host memory.  Device buffers must be 16-byte aligned.
 *   - The caller owns every buffer.  The library never allocates device
 *     memory; a plan owns host memory only.
 *   - Work is enqueued asynchronously on the given stream (0 = the null
 *     stream).  The return status covers argument checks and launch errors;
 *     a fault inside a kernel surfaces at the caller's next synchronisation.
 *   - No C++ exception crosses this ABI.  On any status other than
 *     FFTSPLIT_SUCCESS, fftsplit_last_error() returns a message for the
 *     calling thread and nothing has been enqueued.
 *   - A plan is immutable after creation and may be used from several
 *     threads and streams at once, as long as each concurrent call has its
 *     own workspace and output.
 */
#ifndef FFTSPLIT_H
#define FFTSPLIT_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fftsplit_plan_s* fftsplit_plan_t;   /* opaque, host-side */

typedef enum {
    FFTSPLIT_SUCCESS = 0,
    FFTSPLIT_ERROR_INVALID_VALUE = 1,        /* bad dimension, NULL/misaligned pointer, aliasing */
    FFTSPLIT_ERROR_NOT_SUPPORTED = 2,        /* even K, stride != 1, pad != K/2, unsupported L */
    FFTSPLIT_ERROR_INSUFFICIENT_WORKSPACE = 3,
    FFTSPLIT_ERROR_DEVICE = 4,               /* a HIP runtime call or kernel launch failed */
    FFTSPLIT_ERROR_ARCH = 5                  /* the device is not gfx950 */
} fftsplit_status_t;

/* Problem flags. */
enum {
    FFTSPLIT_OVERLAP_SAVE = 0,   /* halo'd patches, crop + concatenate (Section 3.1); default */
    FFTSPLIT_OVERLAP_ADD  = 1,   /* zero-padded patches, overlap-add of the L x L results */
    FFTSPLIT_BIAS         = 2,   /* add bias[co] in the inverse stage */
    FFTSPLIT_RELU         = 4,   /* apply max(., 0) after the bias */
    FFTSPLIT_MAXPOOL      = 8    /* then a 2x2 stride-2 max-pool (floor): y is
                                  * [n][cout][h/2][w/2] (the VGG stage ends);
                                  * needs h, w >= 2 */
};

/* The layer, as the paper states the problem: batch n, channels cin -> cout,
 * an h x w input, a k x k filter, the patch (tile) size, stride 1 and zero
 * padding of k/2 (Section 2, eq. 1; Section 3.1). */
typedef struct {
    int n, cin, h, w, cout, k;
    int tile;        /* T; 0 lets the plan choose among L = 8, 16, 32.  With
                      * FFTSPLIT_OVERLAP_ADD, tile = k (k = 3, 5, 7) selects the
                      * OaAConv configuration the paper compares against
                      * (Section 2, Fig. 1): patches of the filter's size,
                      * L = 2k - 1 = 5, 9, 13 */
    int stride;      /* must be 1 */
    int pad;         /* must be k/2 ('same') */
    unsigned flags;  /* FFTSPLIT_* flags above */
} fftsplit_problem_t;

/* What a plan decided.  Spectra are complex64 (re, im float pairs).
 *
 * Frequency bins: the 2-D real transform S of an L x L patch has
 * L*(L/2+1) bins (k1 in [0,L), k2 in [0,L/2]); columns k2 = 0 and k2 = L/2
 * are Hermitian in k1, so only their k1 <= L/2 halves are kept, and the
 * four of those that are real (k1, k2 in {0, L/2}) share two slots, leaving
 * bins = L*L/2 slots.  Slot f holds
 *   f = (k2-1)*L + k1             S(k1, k2)   for k2 in [1, L/2-1], k1 in [0, L)
 *   f = L*(L/2-1) + k1 - 1        S(k1, 0)    for k1 in [1, L/2-1]
 *   f = L*(L/2-1) + L/2-2 + k1    S(k1, L/2)  for k1 in [1, L/2-1]
 *   f = L*L/2 - 2                 (S(0, 0), S(L/2, 0))     as (re, im)
 *   f = L*L/2 - 1                 (S(0, L/2), S(L/2, L/2)) as (re, im)
 * The two last slots are multiplied part by part in the per-bin product
 * (a product of two real bins is real), the others as complex numbers.
 * For odd L (the OaAConv configuration) only S(0, 0) is real, nothing is
 * packed, and bins = (L*L+1)/2:
 *   f = (k2-1)*L + k1             S(k1, k2)   for k2 in [1, (L-1)/2], k1 in [0, L)
 *   f = (L-1)/2*L + k1            S(k1, 0)    for k1 in [0, (L-1)/2]
 *
 * Patch index t = (img * tiles_h + a) * tiles_w + b for the patch whose
 * top-left output pixel is (a*T, b*T); t in [tiles, tiles_padded) are zero
 * padding.
 *
 * Layouts (all complex64, innermost index last):
 *   weight spectra  W[bins][cin][cout_padded]        (wspec, wspec_bytes)
 *       = conj(DFT of w[co][ci] zero-padded top-left to L x L) / L^2,
 *         zero for co >= cout
 *   patch spectra   X[cin16/16][bins][16][tiles_padded]  (workspace + xspec_offset)
 *       channel-blocked: channel c of bin f is row c % 16 of block c / 16
 *       (cin16 = cin rounded up to a multiple of 16), so the slots of one
 *       channel are 16 * tiles_padded elements apart
 *   output spectra  Y[cout_padded][tiles_padded/G][bins][G] (workspace + yspec_offset)
 *       patch-group-major, G = spec_group (64, 32, 16 for L = 8, 16, 32):
 *       all slots of one channel and G consecutive patches are one
 *       contiguous run (the unit of work of the inverse transform)
 * The DFT is unnormalised, exp(-2 pi i (m k1 + q k2) / L). */
typedef struct {
    int tile;            /* T */
    int nfft;            /* L = T + k - 1 */
    int tiles_h, tiles_w;/* ceil(h/T), ceil(w/T) */
    int tiles;           /* n * tiles_h * tiles_w */
    int tiles_padded;    /* tiles rounded up to the contraction's tile granularity */
    int bins;            /* L*L/2 ((L*L+1)/2 for odd L) */
    int cout_padded;     /* cout rounded up to the contraction's tile granularity */
    unsigned flags;
    size_t wspec_bytes;
    size_t workspace_bytes;
    size_t xspec_offset, xspec_bytes;
    size_t yspec_offset, yspec_bytes;
    size_t aux_offset, aux_bytes;   /* overlap-add seam partials (0 for overlap-save) */
    /* Contraction kernel variant chosen by the plan: output tile
     * contract_tile_m channels x contract_tile_n patches, input channels in
     * stages of contract_stage_k, and 3 (Gauss) or 4 real matrix products
     * per complex multiply-add.  The environment variable
     * FFTSPLIT_CONTRACT_TILE=[g3:|g4:]MxNxK overrides it at plan time. */
    int contract_tile_m, contract_tile_n, contract_stage_k, contract_real_products;
    int spec_group;      /* G of the output-spectra layout */
    /* 1 if fftsplit_conv2d sums the input channels inside the inverse stage
     * (layers of at most 4 input channels at L = 8, 3 at L = 16, on the
     * overlap-save band path): no contraction launch, and the output
     * spectra region of the workspace is left untouched.  The stage entry
     * points are unaffected. */
    int fused_channel_sum;
    /* Bytes of the filter layout of the direct (spatial) convolution,
     * fftsplit_direct_transform_weights. */
    size_t direct_wspec_bytes;
    /* Input-channel stages the contraction loads ahead of the one it
     * multiplies: 1 (through registers), or 2 or 3 straight into LDS (2 the
     * default where the tile has that variant, 3 with the 8-channel stages
     * the plan picks for layers of at most 128 input channels and at least
     * 8192 workgroups).  The environment variable
     * FFTSPLIT_CONTRACT_PREFETCH=1..3 overrides it at plan time. */
    int contract_prefetch;
    /* The plan's cost model for the chosen L (Section 3.2 weighs the
     * operations and memory accesses of a patch size; here they are priced
     * at an effective HBM rate and matrix-core rate):
     *   model_contract_flops  = 8 * bins * cin * cout_padded * tiles_padded
     *                           (8 flops per complex multiply-add),
     *   model_transform_bytes = forward bytes (x read once, patch spectra
     *                           written once) + inverse bytes (output spectra
     *                           read once, y written once),
     *   model_seconds         = the modelled time the tile choice minimises. */
    double model_contract_flops;
    double model_transform_bytes;
    double model_seconds;
    /* Transform kernel variants: 1 if the forward / inverse stage runs the
     * row-band kernel (overlap-save, image width a multiple of 4 and at most
     * 256), else the general one; forward_sweep is 1 if the row-band forward
     * spaces each workgroup's work items a grid apart (chosen where the
     * input and the patch spectra together exceed 256 MB;
     * FFTSPLIT_FORWARD_SWEEP=1 / 0 forces it at plan time). */
    int forward_band, forward_sweep, inverse_band;
    /* 1 if the row-band forward reads its input non-temporally (an input
     * larger than the 256 MB last-level cache). */
    int forward_stream;
} fftsplit_plan_info_t;

/* Validate `prob` (host) and create a plan for `device` (a HIP ordinal).
 * The paper leaves the patch size free, to be chosen from the resources of
 * the hardware (Section 3.1, first paragraph), and weighs a patch size by
 * its operation count and memory accesses (Section 3.2, eqs. 13-14).  Here
 * the choice is among the FFT sizes the kernels implement.
 * Queries the device: its gcnArchName must start with "gfx950", else
 * FFTSPLIT_ERROR_ARCH.  With prob->tile == 0 the plan picks T from a cost
 * model over L = 8, 16, 32 (the model_* fields of fftsplit_plan_info_t);
 * the environment variable FFTSPLIT_TILE forces a tile size.  No device memory is touched.  *out is set only on success.
 * Other environment variables read here (for experiments; the defaults are
 * the measured best): FFTSPLIT_CONTRACT_TILE (see contract_tile_m),
 * FFTSPLIT_CONTRACT_PREFETCH (see contract_prefetch),
 * FFTSPLIT_FORWARD_BAND=0 / FFTSPLIT_INVERSE_BAND=0 (general forward /
 * inverse kernels instead of the row-band ones), FFTSPLIT_FORWARD_SWEEP=1 / 0
 * (the row-band forward's workgroups run items a grid apart, or contiguous
 * runs; by default the former where input and patch spectra exceed 256 MB),
 * FFTSPLIT_FUSE_CIN=0 (no channel sum in the inverse), FFTSPLIT_LOG=1 (print
 * the plan to stderr). */
fftsplit_status_t fftsplit_plan(const fftsplit_problem_t* prob, int device, fftsplit_plan_t* out);

/* As fftsplit_plan, but for a named architecture string (host-only, no HIP
 * call).  The resulting plan can be queried but not executed: the entry
 * points that launch work return FFTSPLIT_ERROR_INVALID_VALUE for it. */
fftsplit_status_t fftsplit_plan_for_arch(const fftsplit_problem_t* prob, const char* arch,
                                         fftsplit_plan_t* out);

/* What the plan decided (Section 3.1: patch size T and FFT size
 * L = T + K - 1; Section 3.2: the cost that chose them), the buffer sizes
 * and layouts the caller must provide, and the kernel variants.  Fails with
 * FFTSPLIT_ERROR_INVALID_VALUE on a NULL argument. */
fftsplit_status_t fftsplit_plan_info(fftsplit_plan_t plan, fftsplit_plan_info_t* out /* host */);

/* Frees a plan's host memory.  NULL is ignored. */
void fftsplit_plan_destroy(fftsplit_plan_t plan);

/* Eq. (8) and the filter half of eq. (9), once per layer:
 * w (device) [cout][cin][k][k] -> wspec (device, info.wspec_bytes).  The
 * spectra are evaluated in double precision and rounded once to fp32. */
fftsplit_status_t fftsplit_transform_weights(fftsplit_plan_t plan, const float* w, void* wspec,
                                             hipStream_t stream);

/* The hot path, Section 3.1 steps 1-6:
 *   x (device) [n][cin][h][w], wspec from fftsplit_transform_weights,
 *   bias (device) [cout] or NULL (required iff FFTSPLIT_BIAS),
 *   y (device) [n][cout][h][w] (must not overlap x),
 *   workspace (device) of at least info.workspace_bytes.
 * Enqueues the forward patch transform, the per-bin contraction and the
 * inverse transform with placement on `stream`. */
fftsplit_status_t fftsplit_conv2d(fftsplit_plan_t plan, const float* x, const void* wspec,
                                  const float* bias, float* y, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/* Bytes of the static device scratch behind fftsplit_conv2d_noalloc. */
#define FFTSPLIT_NOALLOC_MAX_WORKSPACE (256u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fftsplit_conv2d with the workspace taken from a static device array of
 * FFTSPLIT_NOALLOC_MAX_WORKSPACE bytes (256 MiB) that the library holds on
 * each device it runs on until the process ends.  Same arguments, layouts,
 * kernels and results as fftsplit_conv2d, minus the workspace; calls no
 * allocating routine.  Plans whose info.workspace_bytes exceed the limit
 * get FFTSPLIT_ERROR_INSUFFICIENT_WORKSPACE (nothing enqueued).  Every call
 * on a device shares that device's array: calls that overlap on one device
 * (concurrent streams, or threads) race and must be serialised by the
 * caller.  The array needs no clearing between calls.  The first call on a
 * device looks up the array's device address (hipGetSymbolAddress). */
fftsplit_status_t fftsplit_conv2d_noalloc(fftsplit_plan_t plan, const float* x, const void* wspec,
                                          const float* bias, float* y, hipStream_t stream);

/* The three stages of fftsplit_conv2d, separately (same arguments and
 * workspace layout; running them in order is exactly fftsplit_conv2d).
 * They exist for stage-by-stage testing and per-kernel timing.
 *   forward:  x -> patch spectra at workspace + xspec_offset (eqs. 4-6, FFT)
 *   contract: patch spectra, wspec -> output spectra at yspec_offset (eq. 9)
 *   inverse:  output spectra -> y, with crop/concatenate or overlap-add,
 *             bias and ReLU (eq. 10). */
fftsplit_status_t fftsplit_forward(fftsplit_plan_t plan, const float* x, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);
fftsplit_status_t fftsplit_contract(fftsplit_plan_t plan, const void* wspec, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream);
fftsplit_status_t fftsplit_inverse(fftsplit_plan_t plan, const float* bias, float* y,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The spatial convolution the paper compares the split method against
 * (Section 2, eq. 1 computed directly; Section 4): the same layer as the
 * plan's, as an implicit matrix product on the fp32 matrix cores, with the
 * plan's bias and ReLU flags.  The filters are first rearranged once per
 * layer:
 *   fftsplit_direct_transform_weights: w (device) [cout][cin][k][k] ->
 *     wd (device, info.direct_wspec_bytes) = [k*k][cin16][cout_padded],
 *     zero for padded channels;
 *   fftsplit_direct_conv2d: x (device) [n][cin][h][w], wd, bias (device,
 *     [cout] or NULL; required iff FFTSPLIT_BIAS), y (device)
 *     [n][cout][h][w] (must not overlap x or wd).  No workspace.  x must be
 *     under 2 GiB (FFTSPLIT_ERROR_NOT_SUPPORTED otherwise).
 * The plan's tile size and overlap mode do not apply. */
fftsplit_status_t fftsplit_direct_transform_weights(fftsplit_plan_t plan, const float* w, float* wd,
                                                    hipStream_t stream);
fftsplit_status_t fftsplit_direct_conv2d(fftsplit_plan_t plan, const float* x, const float* wd, const float* bias,
                                         float* y, hipStream_t stream);

/* 2x2, stride-2 max-pool (floor), used between the stages of a VGG-16
 * stack; not part of the method.  x (device) [n][c][h][w] ->
 * y (device) [n][c][h/2][w/2].  x and y must not overlap. */
fftsplit_status_t fftsplit_maxpool2x2(const float* x, float* y, int n, int c, int h, int w,
                                      hipStream_t stream);

/* Benchmark hook (host, per calling thread): until called again with
 * NULL, NULL, every later fftsplit_transform_weights / fftsplit_conv2d /
 * stage call made by this thread records `start` (if non-NULL) when its
 * first kernel begins executing and `stop` (if non-NULL) when its last
 * kernel ends, using the kernels' own dispatch timestamps
 * (hipExtLaunchKernel) rather than separate event packets; the two
 * measurement probes below are timed the same way.  The events
 * must be valid hipEvents created with timing enabled, on the plan's
 * device.  Always returns FFTSPLIT_SUCCESS. */
fftsplit_status_t fftsplit_set_timing_events(hipEvent_t start, hipEvent_t stop);

/* Measurement hooks: the practical ceilings the path's kernels are
 * measured against, on the device they run on.  Neither computes anything
 * of the method.
 *
 * fftsplit_probe_matrix: enqueues on `stream` (on the plan's device) one
 * kernel with the plan's contraction launch -- the same grid of 256-thread
 * workgroups and the same dynamic LDS, hence the same workgroups per
 * compute unit -- in which every wave issues as many fp32 matrix
 * operations (v_mfma_f32_32x32x2f32) as a wave of fftsplit_contract does,
 * with operands in registers and no other memory traffic.  Its duration is
 * the time the matrix cores need for the contraction's executed
 * operations at this launch shape.  `sink` (device, one float) is written
 * only if the sum of a wave's accumulators is exactly -1, which it never
 * is.  INVALID_VALUE for a NULL plan or sink or an architecture-only plan;
 * NOT_SUPPORTED for a plan whose channel sum runs inside the inverse (it
 * has no contraction).
 *
 * fftsplit_probe_stream: enqueues on `stream` (current device) a plain
 * streaming kernel that loads `read_bytes` from src and stores
 * `write_bytes` to dst, 16 bytes per lane, from 8192 workgroups of 256
 * threads: dst[i] = src[i] for the first min(read_bytes, write_bytes)
 * bytes, zero for the rest of dst.  Its duration is what HBM needs for
 * that read/write mix (e.g. a transform's bytes).  Both pointers device,
 * 16-byte aligned, sizes multiples of 16, not overlapping; INVALID_VALUE
 * otherwise. */
fftsplit_status_t fftsplit_probe_matrix(fftsplit_plan_t plan, float* sink, hipStream_t stream);
fftsplit_status_t fftsplit_probe_stream(const void* src, void* dst, size_t read_bytes, size_t write_bytes,
                                        hipStream_t stream);

/* Static description of a status code. */
const char* fftsplit_status_string(fftsplit_status_t status);

/* Detail of the calling thread's last failure (empty string if none).
 * Valid until the thread's next call into the library. */
const char* fftsplit_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FFTSPLIT_H */
