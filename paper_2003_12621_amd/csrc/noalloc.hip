// fftsplit_conv2d_noalloc: fftsplit_conv2d with the workspace taken from a
// static device array instead of a caller's buffer, for callers that cannot
// allocate device memory.
//
// The array is a file-scope __device__ variable: each device the library
// runs on holds its own copy, at its own address, from the first call on
// that device until the process ends.  Host code never uses the array's
// name as a device address (on the host it names a host-side stand-in):
// the device address is looked up once per device, with that device
// current, and kept in g_scratch_ptr.  Every call on a device shares that
// device's copy; nothing in it has to start at zero (each byte a kernel of
// the convolution reads was written earlier in the same call), and calls
// that overlap on one device race on it.
#include <mutex>
#include <string>

#include "fftsplit_internal.hpp"

static __device__ __align__(256) unsigned char scratch[FFTSPLIT_NOALLOC_MAX_WORKSPACE];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `device`'s copy of the scratch array; `device` must be
// the current device.
fftsplit_status_t scratch_address(int device, void** out) {
    if (device < 0 || device >= kMaxDevices)
        return fftsplit::fail(FFTSPLIT_ERROR_NOT_SUPPORTED,
                              "device ordinal " + std::to_string(device) + " is beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fftsplit::fail(FFTSPLIT_ERROR_DEVICE,
                                  std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return FFTSPLIT_SUCCESS;
}

}  // namespace

FFTSPLIT_EXPORT fftsplit_status_t fftsplit_conv2d_noalloc(fftsplit_plan_t plan, const float* x, const void* wspec,
                                                          const float* bias, float* y, hipStream_t stream) {
    using namespace fftsplit;
    set_error("");
    if (fftsplit_status_t s = check_conv2d_args(plan, x, wspec, bias, y)) return s;
    if (plan->ws_bytes > size_t(FFTSPLIT_NOALLOC_MAX_WORKSPACE))
        return fail(FFTSPLIT_ERROR_INSUFFICIENT_WORKSPACE,
                    "the plan needs a workspace of " + std::to_string(plan->ws_bytes) +
                        " bytes; the static scratch of fftsplit_conv2d_noalloc holds " +
                        std::to_string(size_t(FFTSPLIT_NOALLOC_MAX_WORKSPACE)) +
                        " (use fftsplit_conv2d with a caller workspace)");
    DeviceGuard g(plan->device);
    if (!g.ok()) return fail(FFTSPLIT_ERROR_DEVICE, "cannot select the plan's device");
    void* ws = nullptr;
    if (fftsplit_status_t s = scratch_address(plan->device, &ws)) return s;
    return enqueue_conv2d(plan, x, wspec, bias, y, ws, stream);
}
