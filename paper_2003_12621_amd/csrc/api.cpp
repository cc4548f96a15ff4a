// Entry points that enqueue work: argument checks, device selection, kernel
// launch sequence and HIP-error mapping.
#include <cstdint>
#include <string>

#include "fftsplit_internal.hpp"
#include "launch_util.hpp"

using namespace fftsplit;

namespace {

// Timing events set by fftsplit_set_timing_events for this thread.
thread_local LaunchEvents t_events;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlap(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bn && b0 < a0 + an;
}

fftsplit_status_t check_plan(fftsplit_plan_t plan) {
    if (!plan) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "plan is NULL");
    if (plan->device < 0)
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "plan was created for an architecture name only and cannot run");
    return FFTSPLIT_SUCCESS;
}

fftsplit_status_t check_ptr(const void* p, const char* name) {
    if (!p) return fail(FFTSPLIT_ERROR_INVALID_VALUE, std::string(name) + " is NULL");
    if (!aligned16(p)) return fail(FFTSPLIT_ERROR_INVALID_VALUE, std::string(name) + " is not 16-byte aligned");
    return FFTSPLIT_SUCCESS;
}

fftsplit_status_t check_workspace(fftsplit_plan_t plan, const void* ws, size_t bytes) {
    if (fftsplit_status_t s = check_ptr(ws, "workspace")) return s;
    if (bytes < plan->ws_bytes)
        return fail(FFTSPLIT_ERROR_INSUFFICIENT_WORKSPACE,
                    "workspace has " + std::to_string(bytes) + " bytes, plan needs " + std::to_string(plan->ws_bytes));
    return FFTSPLIT_SUCCESS;
}

fftsplit_status_t check_bias(fftsplit_plan_t plan, const float* bias) {
    if (plan->bias) return check_ptr(bias, "bias");
    if (bias) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "bias given but the plan has no FFTSPLIT_BIAS flag");
    return FFTSPLIT_SUCCESS;
}

fftsplit_status_t launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(FFTSPLIT_ERROR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
    return FFTSPLIT_SUCCESS;
}

size_t x_bytes(fftsplit_plan_t p) { return size_t(p->prob.n) * p->prob.cin * p->prob.h * p->prob.w * 4; }
char* ws_at(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

size_t y_bytes(fftsplit_plan_t p) {
    const size_t plane = p->pool ? size_t(p->prob.h / 2) * (p->prob.w / 2) : size_t(p->prob.h) * p->prob.w;
    return size_t(p->prob.n) * p->prob.cout * plane * 4;
}

// The inverse stage into y: with FFTSPLIT_MAXPOOL either pooled in the
// inverse kernel itself or through the workspace's unpooled staging buffer
// and a pooling pass.
// xs/ws non-NULL: the fused variant (fuse_cin) that sums the channels itself.
hipError_t launch_inverse_to_y(fftsplit_plan_t plan, const float2* ys, const float* bias, float* y, void* workspace,
                               hipStream_t stream, const LaunchEvents& ev, const float2* xs = nullptr,
                               const float2* ws = nullptr) {
    void* aux = plan->aux_bytes ? ws_at(workspace, plan->aux_off) : nullptr;
    auto inverse = [&](float* out, const LaunchEvents& e) {
        return xs ? launch_inverse_fused(*plan, xs, ws, bias, out, stream, e)
                  : launch_inverse(*plan, ys, bias, out, aux, stream, e);
    };
    if (!plan->pool || plan->pool_fused) return inverse(y, ev);
    float* pre = reinterpret_cast<float*>(ws_at(workspace, plan->pre_off));
    LaunchEvents first;
    first.start = ev.start;
    const hipError_t e = inverse(pre, first);
    if (e != hipSuccess) return e;
    return launch_maxpool(pre, y, plan->prob.n, plan->prob.cout, plan->prob.h, plan->prob.w, stream, ev.stop);
}


}  // namespace

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_transform_weights(fftsplit_plan_t plan, const float* w, void* wspec,
                                                             hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(w, "w")) return s;
    if (fftsplit_status_t s = check_ptr(wspec, "wspec")) return s;
    const size_t wb = size_t(plan->prob.cout) * plan->prob.cin * plan->prob.k * plan->prob.k * 4;
    if (overlap(w, wb, wspec, plan->wspec_bytes)) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "w overlaps wspec");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(launch_weights(*plan, w, static_cast<float2*>(wspec), stream, t_events), "weight transform launch");
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_forward(fftsplit_plan_t plan, const float* x, void* workspace,
                                                   size_t workspace_bytes, hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(x, "x")) return s;
    if (fftsplit_status_t s = check_workspace(plan, workspace, workspace_bytes)) return s;
    if (overlap(x, x_bytes(plan), workspace, plan->ws_bytes))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "x overlaps the workspace");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(
        launch_forward(*plan, x, reinterpret_cast<float2*>(ws_at(workspace, plan->xspec_off)), stream, t_events),
        "forward patch transform launch");
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_contract(fftsplit_plan_t plan, const void* wspec, void* workspace,
                                                    size_t workspace_bytes, hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(wspec, "wspec")) return s;
    if (fftsplit_status_t s = check_workspace(plan, workspace, workspace_bytes)) return s;
    if (overlap(wspec, plan->wspec_bytes, workspace, plan->ws_bytes))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "wspec overlaps the workspace");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(launch_contract(*plan, reinterpret_cast<const float2*>(ws_at(workspace, plan->xspec_off)),
                                    static_cast<const float2*>(wspec),
                                    reinterpret_cast<float2*>(ws_at(workspace, plan->yspec_off)), stream, t_events),
                    "contraction launch");
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_inverse(fftsplit_plan_t plan, const float* bias, float* y,
                                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(y, "y")) return s;
    if (fftsplit_status_t s = check_bias(plan, bias)) return s;
    if (fftsplit_status_t s = check_workspace(plan, workspace, workspace_bytes)) return s;
    if (overlap(y, y_bytes(plan), workspace, plan->ws_bytes))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "y overlaps the workspace");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(launch_inverse_to_y(plan, reinterpret_cast<const float2*>(ws_at(workspace, plan->yspec_off)),
                                        bias, y, workspace, stream, t_events),
                    "inverse patch transform launch");
}

namespace fftsplit {

fftsplit_status_t check_conv2d_args(fftsplit_plan_t plan, const float* x, const void* wspec, const float* bias,
                                    const float* y) {
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(x, "x")) return s;
    if (fftsplit_status_t s = check_ptr(wspec, "wspec")) return s;
    if (fftsplit_status_t s = check_ptr(y, "y")) return s;
    if (fftsplit_status_t s = check_bias(plan, bias)) return s;
    if (overlap(x, x_bytes(plan), y, y_bytes(plan))) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "y overlaps x");
    if (overlap(wspec, plan->wspec_bytes, y, y_bytes(plan))) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "buffers overlap");
    return FFTSPLIT_SUCCESS;
}

fftsplit_status_t enqueue_conv2d(fftsplit_plan_t plan, const float* x, const void* wspec, const float* bias, float* y,
                                 void* workspace, hipStream_t stream) {
    float2* xs = reinterpret_cast<float2*>(ws_at(workspace, plan->xspec_off));
    float2* ys = reinterpret_cast<float2*>(ws_at(workspace, plan->yspec_off));
    LaunchEvents first, middle, last;
    first.start = t_events.start;
    last.stop = t_events.stop;
    if (fftsplit_status_t s = launched(launch_forward(*plan, x, xs, stream, first), "forward patch transform launch"))
        return s;
    if (plan->fuse_cin)
        return launched(launch_inverse_to_y(plan, ys, bias, y, workspace, stream, last, xs,
                                            static_cast<const float2*>(wspec)),
                        "inverse patch transform launch");
    if (fftsplit_status_t s = launched(launch_contract(*plan, xs, static_cast<const float2*>(wspec), ys, stream, middle),
                                       "contraction launch"))
        return s;
    return launched(launch_inverse_to_y(plan, ys, bias, y, workspace, stream, last), "inverse patch transform launch");
}

}  // namespace fftsplit

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_conv2d(fftsplit_plan_t plan, const float* x, const void* wspec,
                                                  const float* bias, float* y, void* workspace,
                                                  size_t workspace_bytes, hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_conv2d_args(plan, x, wspec, bias, y)) return s;
    if (fftsplit_status_t s = check_workspace(plan, workspace, workspace_bytes)) return s;
    if (overlap(x, x_bytes(plan), workspace, plan->ws_bytes) || overlap(y, y_bytes(plan), workspace, plan->ws_bytes) ||
        overlap(wspec, plan->wspec_bytes, workspace, plan->ws_bytes))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "buffers overlap");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return enqueue_conv2d(plan, x, wspec, bias, y, workspace, stream);
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_maxpool2x2(const float* x, float* y, int n, int c, int h, int w,
                                                      hipStream_t stream) {
    set_error("");
    if (n <= 0 || c <= 0 || h < 2 || w < 2) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "need n, c > 0 and h, w >= 2");
    if (fftsplit_status_t s = check_ptr(x, "x")) return s;
    if (fftsplit_status_t s = check_ptr(y, "y")) return s;
    const size_t xb = size_t(n) * c * h * w * 4, yb = size_t(n) * c * (h / 2) * (w / 2) * 4;
    if (overlap(x, xb, y, yb)) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "y overlaps x");
    return launched(launch_maxpool(x, y, n, c, h, w, stream), "max-pool launch");
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_direct_transform_weights(fftsplit_plan_t plan, const float* w, float* wd,
                                                                    hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(w, "w")) return s;
    if (fftsplit_status_t s = check_ptr(wd, "wd")) return s;
    const size_t wb = size_t(plan->prob.cout) * plan->prob.cin * plan->prob.k * plan->prob.k * 4;
    if (overlap(w, wb, wd, direct_wspec_bytes(*plan))) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "w overlaps wd");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(launch_direct_weights(*plan, w, wd, stream), "direct weight layout launch");
}

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_direct_conv2d(fftsplit_plan_t plan, const float* x, const float* wd,
                                                         const float* bias, float* y, hipStream_t stream) {
    set_error("");
    if (fftsplit_status_t s = check_plan(plan)) return s;
    if (fftsplit_status_t s = check_ptr(x, "x")) return s;
    if (fftsplit_status_t s = check_ptr(wd, "wd")) return s;
    if (fftsplit_status_t s = check_ptr(y, "y")) return s;
    if (fftsplit_status_t s = check_bias(plan, bias)) return s;
    if (overlap(x, x_bytes(plan), y, y_bytes(plan))) return fail(FFTSPLIT_ERROR_INVALID_VALUE, "y overlaps x");
    if (overlap(wd, direct_wspec_bytes(*plan), y, y_bytes(plan)))
        return fail(FFTSPLIT_ERROR_INVALID_VALUE, "y overlaps wd");
    if (x_bytes(plan) > 0x7fffffffu)
        return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "direct convolution: the input must be under 2 GiB");
    if (plan->pool) return fail(FFTSPLIT_ERROR_NOT_SUPPORTED, "direct convolution: FFTSPLIT_MAXPOOL is not supported");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    return launched(launch_direct(*plan, x, wd, bias, y, stream, t_events), "direct convolution launch");
}

namespace fftsplit {
LaunchEvents timing_events() { return t_events; }
}  // namespace fftsplit

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_set_timing_events(hipEvent_t start, hipEvent_t stop) {
    set_error("");
    t_events.start = start;
    t_events.stop = stop;
    return FFTSPLIT_SUCCESS;
}
