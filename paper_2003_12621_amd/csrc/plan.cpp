// Plan creation: argument validation, tile-size choice and buffer sizes.
//
// The paper leaves the patch size free, to be picked from the hardware's
// constraints (Section 3.1, first paragraph; Section 3.2).  Here the FFT
// size L is restricted to the register transforms the kernels implement
// (8, 16, 32), so T = L - K + 1, and a plan without an explicit tile picks
// the L whose modelled time (streamed bytes at an effective bandwidth plus
// contraction flops at an effective matrix-core rate) is smallest.
#include <cerrno>
#include <cstdint>
#include <climits>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include "band.hpp"
#include "fftsplit_internal.hpp"

namespace fftsplit {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

fftsplit_status_t fail(fftsplit_status_t st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

static size_t round_up(size_t v, size_t g) { return (v + g - 1) / g * g; }

// Multiply with overflow detection.
static bool mul_ok(size_t a, size_t b, size_t* out) {
    if (a != 0 && b > SIZE_MAX / a) return false;
    *out = a * b;
    return true;
}

// Effective rates of the cost model (bytes/s and flop/s) -- deliberately
// conservative fractions of the 8 TB/s HBM and 157 TFLOP/s fp32 matrix peaks.
static constexpr double kModelBandwidth = 5.0e12;
static constexpr double kModelMatrixRate = 100.0e12;

struct Geometry {
    int T, L, th, tw, nt, ntp, bins, coutp;
    double con_flops, xfer_bytes, model_seconds;
};

static Geometry geometry(const fftsplit_problem_t& p, int L) {
    Geometry g{};
    g.L = L;
    g.T = L - p.k + 1;
    g.th = (p.h + g.T - 1) / g.T;
    g.tw = (p.w + g.T - 1) / g.T;
    const double nt = double(p.n) * g.th * g.tw;
    g.nt = nt > INT_MAX ? -1 : int(nt);
    g.bins = stored_bins(L);
    g.coutp = int(round_up(size_t(p.cout), kCoutGranule));
    const bool small_granule = (L == 16 || L == 32) && g.coutp % 128 == 0;
    g.ntp = g.nt < 0 ? -1 : int(round_up(size_t(g.nt), small_granule ? kTileGranuleSmall : kTileGranule));
    const double F = g.bins, ntp = double(g.ntp), cin = p.cin, coutp = g.coutp;
    const double img = double(p.n) * p.h * p.w;
    const double fwd = 4.0 * img * cin + 8.0 * F * cin * ntp;
    const double con_b = 8.0 * F * (cin * ntp + cin * coutp + coutp * ntp);
    const double con_f = 8.0 * F * cin * coutp * ntp;
    const double inv = 8.0 * F * coutp * ntp + 4.0 * img * p.cout;
    const double con = con_f / kModelMatrixRate > con_b / kModelBandwidth ? con_f / kModelMatrixRate
                                                                          : con_b / kModelBandwidth;
    g.con_flops = con_f;
    g.xfer_bytes = fwd + inv;
    g.model_seconds = fwd / kModelBandwidth + con + inv / kModelBandwidth;
    return g;
}

static bool supported_L(int L) { return L == 8 || L == 16 || L == 32; }

// The OaAConv configuration (the paper's comparison method, Section 2 and
// Fig. 1): overlap-add with patches of the filter's size, T = K, so the
// transforms are L = 2K - 1 = 5, 9 or 13 points.
static bool oaaconv_L(int L, int k, bool oaa) { return oaa && L == 2 * k - 1 && (k == 3 || k == 5 || k == 7); }

// The band variant of the inverse transform (overlap-save, width a multiple
// of 4 and at most 256, crop at least L/2 wide): used when the output band of any work item fits the
// store slots it assigns and its LDS stays within two workgroups per compute
// unit.  FFTSPLIT_INVERSE_BAND=0 turns it off.
static void choose_inverse_band(fftsplit_plan_s& p) {
    p.inv_band = false;
    const int w = p.prob.w, L = p.L, T = p.T;
    // (the row pass stores the first L/2 columns of a crop unconditionally,
    // so the crop must be at least that wide: K <= L/2 + 1)
    if (p.oaa || w % 4 != 0 || w > 256 || 2 * T < L || p.nt >= (1 << 22) || p.prob.h >= (1 << 22) ||
        p.yspec_bytes >= (size_t(1) << 31))
        return;
    if (const char* e = std::getenv("FFTSPLIT_INVERSE_BAND"))
        if (*e == '0') return;
    const int tg = patch_group(L);
    const int nw = tg * (L / 2) / 64;
    const int rpi = 64 / (w / 4);
    const int nv = L == 8 ? kBandNV8 : (L == 16 ? kBandNV16 : kBandNV32);
    int slots = 0;
    for (int t0 = 0; t0 < p.nt; t0 += tg) {
        const BandGeom g = band_geom(t0, tg, p.nt, p.prob.h, T, 0, p.th, p.tw);
        if (g.slots > slots) slots = g.slots;
    }
    if ((slots + nw * rpi - 1) / (nw * rpi) > nv) return;
    int obp = p.tw * T;
    if (obp % 2 == 0) ++obp;   // odd pitch: a patch's row-pass lanes write distinct banks
    const size_t band = size_t(slots) * obp * 4;
    const size_t half = size_t(tg) * band_half_stride(L, tg) * 8;
    const size_t lds = band > half ? band : half;
    if (lds > 80 * 1024) return;
    p.inv_band = true;
    p.inv_obp = obp;
    p.inv_lds = int(lds);
}

// The band variant of the forward transform (overlap-save, image width a
// multiple of 4 and at most 256) is used when its band of any work item fits
// the registers it prefetches into and its LDS stays within two workgroups
// per compute unit.  FFTSPLIT_FORWARD_BAND=0 turns it off.
static void choose_forward_band(fftsplit_plan_s& p) {
    p.fwd_band = false;
    p.fwd_sweep = false;
    p.fwd_stream = false;
    const int w = p.prob.w, L = p.L, T = p.T, P = p.P;
    // (offsets are 32-bit; the tile and row arithmetic uses exact float
    // division, valid below 2^22; stores dropped with an out-of-range
    // offset need spectra below 2 GiB)
    if (p.oaa || w % 4 != 0 || w > 256 || p.nt >= (1 << 22) || p.prob.h >= (1 << 22) ||
        p.xspec_bytes >= (size_t(1) << 31))
        return;
    if (const char* e = std::getenv("FFTSPLIT_FORWARD_BAND"))
        if (*e == '0') return;
    const int tg = forward_group(L);
    const int nw = tg * (L / 2) / 64;
    const int rpi = 64 / (w / 4);
    const int nv = L == 8 ? kBandNV8 : (L == 16 ? kBandNV16 : kBandNV32);
    int slots = 0;
    for (int t0 = 0; t0 < p.nt; t0 += tg) {
        const BandGeom g = band_geom(t0, tg, p.nt, p.prob.h, T, P, p.th, p.tw);
        if (g.slots > slots) slots = g.slots;
    }
    if ((slots + nw * rpi - 1) / (nw * rpi) > nv) return;
    const int co = P;
    int bp = co + p.tw * T + P;
    if (bp % 2 == 0) ++bp;   // odd pitch: a patch's row-pass lanes read distinct banks
    const size_t band = size_t(slots + 1) * bp * 4;
    const size_t half = size_t(tg) * band_half_stride(L, tg) * 8;
    const size_t lds = band > half ? band : half;
    if (lds > 80 * 1024) return;
    p.fwd_band = true;
    // Where the input and the patch spectra together exceed the 256 MB
    // last-level cache, both stream from and to HBM: then workgroup lw runs
    // items lw, lw + grid, ..., so that the workgroups together read one
    // contiguous range of the input and write one of the spectra at a time.
    // Otherwise each workgroup runs a contiguous run of items and the XCD
    // remap keeps neighbouring items, which share halo rows, on one L2.
    const size_t x_bytes = size_t(p.prob.n) * p.prob.cin * p.prob.h * p.prob.w * 4;
    p.fwd_sweep = x_bytes + p.xspec_bytes > (size_t(256) << 20);
    if (const char* e = std::getenv("FFTSPLIT_FORWARD_SWEEP")) p.fwd_sweep = *e == '1';
    // An input larger than the last-level cache is read non-temporally: it
    // could not stay cached anyway, and so it does not take the room of the
    // spectra the contraction reads next (VGG-16 layer 2, 411 MB: forward
    // and contraction 8-11 us faster; with inputs that fit, such as the
    // 205 MB of layer 4, keeping them cached measured as fast or faster).
    p.fwd_stream = x_bytes > (size_t(256) << 20);
    p.fwd_bp = bp;
    p.fwd_co = co;
    p.fwd_zslot = slots;
    p.fwd_lds = int(lds);
}

static fftsplit_status_t build_plan(const fftsplit_problem_t* prob, int device, const char* arch,
                                    fftsplit_plan_t* out) {
    if (!prob || !out) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "problem and output pointers must be non-NULL");
    const fftsplit_problem_t p = *prob;
    if (p.n <= 0 || p.cin <= 0 || p.h <= 0 || p.w <= 0 || p.cout <= 0 || p.k <= 0)
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "all dimensions must be positive");
    if (p.tile < 0) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "tile must be >= 0 (0 = choose)");
    const unsigned known = FFTSPLIT_OVERLAP_ADD | FFTSPLIT_BIAS | FFTSPLIT_RELU | FFTSPLIT_MAXPOOL;
    if (p.flags & ~known) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "unknown flag bits");
    if (p.k % 2 == 0) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "kernel size must be odd");
    if (p.stride != 1) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "only stride 1 is supported");
    if (p.pad != p.k / 2) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "only 'same' padding (pad = k/2) is supported");
    if (p.k > 31) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "kernel larger than the largest FFT size");
    if (size_t(p.h) * size_t(p.w) > size_t(INT_MAX))
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "image planes above 2^31 pixels are not supported");
    if (p.cin > 65535 || p.cout > 65535)
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "channel counts above 65535 are not supported");
    const bool oaa = (p.flags & FFTSPLIT_OVERLAP_ADD) != 0;
    const bool pool = (p.flags & FFTSPLIT_MAXPOOL) != 0;
    if (pool && (p.h < 2 || p.w < 2)) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "max-pool needs h, w >= 2");

    int tile = p.tile;
    if (tile == 0) {
        const char* env = std::getenv("FFTSPLIT_TILE");
        if (env && *env) {
            char* end = nullptr;
            errno = 0;
            long v = std::strtol(env, &end, 10);
            if (errno || !end || *end || v <= 0 || v > 32)
                return fail(FFTSPLIT_ERROR_INVALID_VALUE, "FFTSPLIT_TILE must be a positive integer <= 32");
            tile = int(v);
        }
    }
    Geometry g{};
    if (tile > 0) {
        const int L = tile + p.k - 1;
        if (!supported_L(L) && !oaaconv_L(L, p.k, oaa))
            return fail(FFTSPLIT_ERROR_NOT_SUPPORTED,
                        "tile + k - 1 must be 8, 16 or 32, or tile = k for k in {3, 5, 7} with overlap-add "
                        "(got " + std::to_string(L) + ")");
        g = geometry(p, L);
    } else {
        bool have = false;
        for (int L : {8, 16, 32}) {
            const int T = L - p.k + 1;
            if (T < 1 || (oaa && T < p.k - 1)) continue;
            Geometry c = geometry(p, L);
            if (c.nt < 0) continue;
            if (!have || c.model_seconds < g.model_seconds) { g = c; have = true; }
        }
        if (!have) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "no FFT size in {8,16,32} fits this kernel");
    }
    if (oaa && g.T < p.k - 1)
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "overlap-add needs tile >= k - 1");
    if (g.nt < 0 || g.ntp < 0 || g.ntp / kTileGranuleSmall > INT_MAX / 2)
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "too many patches");
    // The overlap-add seam buffer is indexed with 32-bit offsets.
    if (oaa && size_t(p.cout) * size_t(g.ntp) * size_t(g.L) * size_t(g.L) > size_t(INT_MAX))
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "overlap-add seam buffer above 2^31 elements is not supported");
    // The seam pass addresses one image plane's patch results in bytes below 2^31.
    if (oaa && size_t(g.th) * size_t(g.tw) * size_t(g.L) * size_t(g.L) >= (size_t(1) << 29))
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "overlap-add results of one image above 2^29 elements are not supported");
    // The contraction indexes one bin's spectra with 32-bit offsets.
    if (size_t(p.cin) * size_t(g.coutp) > size_t(INT_MAX) || size_t(p.cin) * size_t(g.ntp) > size_t(INT_MAX) ||
        size_t(g.coutp) * size_t(g.ntp) > size_t(INT_MAX))
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "per-bin spectra above 2^31 elements are not supported");

    // Byte sizes with overflow checks.
    size_t xs, ys, wsb, tmp;
    if (!mul_ok(size_t(g.bins) * 8, size_t(round_up_block(p.cin)), &tmp) || !mul_ok(tmp, size_t(g.ntp), &xs) ||
        !mul_ok(size_t(g.bins) * 8, size_t(g.coutp), &tmp) || !mul_ok(tmp, size_t(g.ntp), &ys) ||
        !mul_ok(size_t(g.bins) * 8, size_t(p.cin), &tmp) || !mul_ok(tmp, size_t(g.coutp), &wsb))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "buffer sizes overflow size_t");
    // Kernels address x and y with 32-bit element offsets.
    size_t img_elems;
    if (!mul_ok(size_t(p.n) * size_t(p.h), size_t(p.w), &tmp) ||
        !mul_ok(tmp, size_t(p.cin > p.cout ? p.cin : p.cout), &img_elems))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "tensor sizes overflow size_t");
    // ... and with 32-bit byte offsets inside buffer descriptors.
    if (img_elems > size_t(INT_MAX) / 4)
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "input/output tensors above 2^29 elements are not supported");
    if (xs > size_t(UINT32_MAX) || ys > size_t(UINT32_MAX))
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "patch/output spectra above 4 GiB are not supported");

    // Architecture check.
    char archbuf[64] = {0};
    int cus = 256;   // MI355X
    if (device >= 0) {
        hipDeviceProp_t prop;
        hipError_t e = hipGetDeviceProperties(&prop, device);
        if (e != hipSuccess)
            return fail(FFTSPLIT_ERROR_DEVICE, std::string("hipGetDeviceProperties: ") + hipGetErrorString(e));
        std::snprintf(archbuf, sizeof(archbuf), "%s", prop.gcnArchName);
        if (prop.multiProcessorCount > 0) cus = prop.multiProcessorCount;
    } else {
        std::snprintf(archbuf, sizeof(archbuf), "%s", arch ? arch : "");
    }
    if (std::strncmp(archbuf, "gfx950", 6) != 0)
        return fail(FFTSPLIT_ERROR_ARCH, std::string("device architecture '") + archbuf + "' is not gfx950");

    fftsplit_plan_s* plan = new (std::nothrow) fftsplit_plan_s();
    if (!plan) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "out of host memory");
    plan->prob = p;
    plan->prob.tile = g.T;
    plan->device = device;
    plan->cus = cus;
    std::snprintf(plan->arch, sizeof(plan->arch), "%s", archbuf);
    plan->T = g.T;
    plan->L = g.L;
    plan->P = p.k / 2;
    plan->th = g.th;
    plan->tw = g.tw;
    plan->nt = g.nt;
    plan->ntp = g.ntp;
    plan->bins = g.bins;
    plan->coutp = g.coutp;
    plan->model_con_flops = g.con_flops;
    plan->model_xfer_bytes = g.xfer_bytes;
    plan->model_seconds = g.model_seconds;
    plan->oaa = oaa;
    plan->bias = (p.flags & FFTSPLIT_BIAS) != 0;
    plan->relu = (p.flags & FFTSPLIT_RELU) != 0;
    plan->pool = pool;
    plan->wspec_bytes = wsb;
    plan->xspec_off = 0;
    plan->xspec_bytes = xs;
    plan->yspec_off = round_up(xs, 256);
    plan->yspec_bytes = ys;
    plan->aux_off = round_up(plan->yspec_off + ys, 256);
    // Overlap-add keeps each patch's L x L inverse result for the seam pass.
    plan->aux_bytes = oaa ? size_t(p.cout) * size_t(g.ntp) * size_t(g.L) * size_t(g.L) * 4 : 0;
    plan->ws_bytes = plan->aux_off + plan->aux_bytes;

    // Contraction variant: 64x64 tiles (128x32 where the patches are padded
    // to 32 only), 16-channel stages (8-channel ones for few input channels
    // and many workgroups, below), three real products per complex
    // multiply-add (fastest measured on every layer shape);
    // FFTSPLIT_CONTRACT_TILE=[g3:|g4:]BMxBNxKC and FFTSPLIT_CONTRACT_PREFETCH
    // override.
    plan->con_bm = g.ntp % 64 == 0 ? 64 : 128;
    plan->con_bn = g.ntp % 64 == 0 ? 64 : 32;
    plan->con_kc = 16;
    plan->con_products = 3;
    // two stages ahead, through LDS (the tiles that have that variant)
    plan->con_prefetch = 2;
    // Few input channels and many workgroups (at most 8 stages of 16 per
    // workgroup, at least 8192 64x64 workgroups: the 224^2 and 112^2 VGG-16
    // layers): each workgroup's first stages, loaded before it can multiply,
    // are a large part of its time, and 8-channel stages three ahead (32 KB
    // of LDS, four workgroups per CU instead of three) hide more of them.
    if (plan->con_bm == 64 && p.cin <= 128 &&
        size_t(g.coutp / 64) * size_t(g.ntp / 64) * size_t(g.bins) >= 8192) {
        plan->con_kc = 8;
        plan->con_prefetch = 3;
    }
    const char* pf_env = std::getenv("FFTSPLIT_CONTRACT_PREFETCH");
    if (const char* v = std::getenv("FFTSPLIT_CONTRACT_TILE")) {
        if (*v) {
            plan->con_prefetch = 2;
            int prod = 4;
            const char* q = v;
            if (!std::strncmp(q, "g3:", 3)) { prod = 3; q += 3; }
            else if (!std::strncmp(q, "g4:", 3)) { q += 3; }
            int bm = 0, bn = 0, kc = 0, used = 0;
            if (std::sscanf(q, "%dx%dx%d%n", &bm, &bn, &kc, &used) != 3 || q[used] != '\0') {
                delete plan;
                return fail(FFTSPLIT_ERROR_INVALID_VALUE, "FFTSPLIT_CONTRACT_TILE must look like [g3:]BMxBNxKC");
            }
            if (!contract_variant_exists(bm, bn, kc, prod)) {
                delete plan;
                return fail(FFTSPLIT_ERROR_INVALID_VALUE, std::string("FFTSPLIT_CONTRACT_TILE=") + v +
                                                              " names no contraction kernel variant");
            }
            plan->con_bm = bm;
            plan->con_bn = bn;
            plan->con_kc = kc;
            plan->con_products = prod;
        }
    }
    if (pf_env) {
        const int pf = std::atoi(pf_env);
        if (pf >= 1 && pf <= 3) plan->con_prefetch = pf;
    }
    // the LDS-prefetch variants exist for the 3-product tiles with
    // 16-channel stages (64x64, 128x32, 128x64, 64x128; three stages ahead
    // for 64x64 only) and for 64x64 with 8-channel stages
    {
        const bool t64 = plan->con_bm == 64 && plan->con_bn == 64;
        const bool lds_variant =
            plan->con_products == 3 &&
            ((plan->con_kc == 16 && (t64 || (plan->con_bm == 128 && plan->con_bn == 32) ||
                                     (plan->con_bm == 128 && plan->con_bn == 64) ||
                                     (plan->con_bm == 64 && plan->con_bn == 128))) ||
             (plan->con_kc == 8 && t64));
        if (!lds_variant) plan->con_prefetch = 1;
        if (plan->con_prefetch == 3 && plan->con_bm != 64) plan->con_prefetch = 2;
    }
    if (g.coutp % plan->con_bm != 0 || g.ntp % plan->con_bn != 0) {
        const int bm = plan->con_bm, bn = plan->con_bn;
        delete plan;
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "contraction tile " + std::to_string(bm) + "x" + std::to_string(bn) +
                                                      " does not divide the padded problem");
    }

    choose_forward_band(*plan);
    choose_inverse_band(*plan);
    // The max-pool goes into the overlap-save inverse's store phase when no
    // pooling window straddles two tiles (even tile size) and, for the band
    // inverse, its slots pair up into pooled rows (even image height);
    // otherwise the unpooled output is staged in the workspace and pooled
    // by a separate pass.
    plan->pool_fused = pool && !oaa && g.L % 2 == 0 && g.T % 2 == 0 && (!plan->inv_band || p.h % 2 == 0);
    // Layers with at most 4 (L = 8) or 3 (L = 16) input channels, whose
    // patch spectra fit the inverse's registers: the channel sum moves into
    // the inverse (no contraction launch, output spectra never stored).
    // FFTSPLIT_FUSE_CIN=0 turns it off.
    plan->fuse_cin = plan->inv_band && p.cin <= (g.L == 8 ? 4 : (g.L == 16 ? 3 : 0));
    if (const char* e = std::getenv("FFTSPLIT_FUSE_CIN"))
        if (*e == '0') plan->fuse_cin = false;
    plan->pre_off = plan->ws_bytes;
    plan->pre_bytes = 0;
    if (pool && !plan->pool_fused) {
        plan->pre_off = round_up(plan->ws_bytes, 256);
        plan->pre_bytes = size_t(p.n) * p.cout * p.h * p.w * 4;
        plan->ws_bytes = plan->pre_off + plan->pre_bytes;
    }

    const char* log = std::getenv("FFTSPLIT_LOG");
    if (log && *log && *log != '0') {
        std::fprintf(stderr,
                     "[fftsplit] plan n=%d cin=%d %dx%d cout=%d k=%d -> T=%d L=%d tiles=%d(%d) bins=%d %s "
                     "model=%.1f us wspec=%zu ws=%zu\n",
                     p.n, p.cin, p.h, p.w, p.cout, p.k, g.T, g.L, g.nt, g.ntp, g.bins, oaa ? "oaa" : "os",
                     g.model_seconds * 1e6, wsb, plan->ws_bytes);
    }
    *out = plan;
    return FFTSPLIT_SUCCESS;
}

}  // namespace fftsplit

using namespace fftsplit;

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_plan(const fftsplit_problem_t* prob, int device, fftsplit_plan_t* out) {
    set_error("");
    if (device < 0) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "device ordinal must be >= 0");
    return build_plan(prob, device, nullptr, out);
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_plan_for_arch(const fftsplit_problem_t* prob, const char* arch,
                                                         fftsplit_plan_t* out) {
    set_error("");
    if (!arch) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "architecture string must be non-NULL");
    return build_plan(prob, -1, arch, out);
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_plan_info(fftsplit_plan_t plan, fftsplit_plan_info_t* out) {
    set_error("");
    if (!plan || !out) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "plan and output must be non-NULL");
    fftsplit_plan_info_t i{};
    i.tile = plan->T;
    i.nfft = plan->L;
    i.tiles_h = plan->th;
    i.tiles_w = plan->tw;
    i.tiles = plan->nt;
    i.tiles_padded = plan->ntp;
    i.bins = plan->bins;
    i.cout_padded = plan->coutp;
    i.flags = plan->prob.flags;
    i.wspec_bytes = plan->wspec_bytes;
    i.workspace_bytes = plan->ws_bytes;
    i.xspec_offset = plan->xspec_off;
    i.xspec_bytes = plan->xspec_bytes;
    i.yspec_offset = plan->yspec_off;
    i.yspec_bytes = plan->yspec_bytes;
    i.aux_offset = plan->aux_off;
    i.aux_bytes = plan->aux_bytes;
    i.contract_tile_m = plan->con_bm;
    i.contract_tile_n = plan->con_bn;
    i.contract_stage_k = plan->con_kc;
    i.contract_real_products = plan->con_products;
    i.direct_wspec_bytes = direct_wspec_bytes(*plan);
    i.spec_group = patch_group(plan->L);
    i.fused_channel_sum = plan->fuse_cin ? 1 : 0;
    i.contract_prefetch = plan->con_prefetch;
    i.forward_band = plan->fwd_band ? 1 : 0;
    i.forward_sweep = plan->fwd_band && plan->fwd_sweep ? 1 : 0;
    i.inverse_band = plan->inv_band ? 1 : 0;
    i.forward_stream = plan->fwd_band && plan->fwd_stream ? 1 : 0;
    i.model_contract_flops = plan->model_con_flops;
    i.model_transform_bytes = plan->model_xfer_bytes;
    i.model_seconds = plan->model_seconds;
    *out = i;
    return FFTSPLIT_SUCCESS;
}

FFTSPLIT_EXPORT void fftsplit_plan_destroy(fftsplit_plan_t plan) { delete plan; }

FFTSPLIT_EXPORT const char* fftsplit_status_string(fftsplit_status_t st) {
    switch (st) {
        case FFTSPLIT_SUCCESS: return "success";
        case FFTSPLIT_ERROR_INVALID_VALUE: return "invalid value";
        case FFTSPLIT_ERROR_NOT_SUPPORTED: return "not supported";
        case FFTSPLIT_ERROR_INSUFFICIENT_WORKSPACE: return "insufficient workspace";
        case FFTSPLIT_ERROR_DEVICE: return "device error";
        case FFTSPLIT_ERROR_ARCH: return "unsupported architecture";
    }
    return "unknown status";
}

FFTSPLIT_EXPORT const char* fftsplit_last_error(void) { return g_last_error.c_str(); }
