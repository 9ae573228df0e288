// The projection entry point for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// allocation): logra_project_layers with its workspace in a static device
// array of the library instead of a caller buffer.
//
// `scratch` is a file-scope device array; every GPU the library runs on
// holds its own copy until the process ends.  In host code its name is only a
// host-side stand-in, never a device address: the address is looked up once
// per device (hipGetSymbolAddress, with that device current) on the entry
// point's first call there, kept per device, and only that address reaches
// the kernels.  The projection's kernels overwrite every workspace byte they
// read before reading it (the prep kernel clears the work counter and lists
// the tiles; partials and tile sums are written before they are summed), so
// nothing needs clearing between calls.  Calls that overlap on one GPU (other
// streams, other threads) share the array and race; the caller orders them.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"
#include "logra.h"

namespace {

constexpr size_t kScratchBytes = LOGRA_NOALLOC_WS_BYTES;
static_assert(kScratchBytes % 256 == 0, "the scratch size keeps the workspace's 256-byte carving");

__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void *g_scratch[kMaxDevices] = {};   // device address of `scratch` on each device, once looked up

// The current device's address of `scratch` (looked up on first use), or an
// error status.
int scratch_ptr(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return logra::hip_fail(e, "current device");
    if (dev < 0 || dev >= kMaxDevices) return logra::fail_unsupported("device index beyond 63");
    std::lock_guard<std::mutex> hold(g_lock);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) return logra::hip_fail(e, "scratch symbol address");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return LOGRA_OK;
}

}  // namespace

extern "C" int logra_project_layers_noalloc(const logra_layer_desc *layers, int n_layers, int in_dtype, int B,
                                            int T, const uint8_t *mask, int k_in, int k_out, int g_dtype,
                                            int64_t g_ld, void *stream) {
    if (B == 0 || T == 0)   // a no-op after the size checks; the scratch is not needed
        return logra::project_layers_checked(layers, n_layers, in_dtype, B, T, mask, k_in, k_out, g_dtype, g_ld,
                                             nullptr, 0, true, stream);
    void *ws = nullptr;
    const int rc = scratch_ptr(&ws);
    if (rc != LOGRA_OK) return rc;
    return logra::project_layers_checked(layers, n_layers, in_dtype, B, T, mask, k_in, k_out, g_dtype, g_ld, ws,
                                         kScratchBytes, true, stream);
}
