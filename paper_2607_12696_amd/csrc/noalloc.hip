// moe_verify_layer for callers that cannot allocate (code under HIP graph
// capture, serving loops, harnesses that forbid hipMalloc): the workspace is
// a fixed device array of this library, one per GPU, held until the process
// ends.  Every call on a GPU shares that GPU's array, so calls that overlap
// on one GPU (different streams, or different host threads without ordering)
// race; calls ordered on one stream do not.  The verify kernels need nothing
// in the workspace to start at zero, so nothing is cleared between calls.
#include "ecospec_moe.h"

#include <hip/hip_runtime.h>
#include <stdio.h>

#include <mutex>

#include "launch.hpp"

// The workspace of every moe_verify_layer_noalloc call on a GPU (each GPU
// holds its own copy of this array, at its own address).
static __device__ __align__(256) uint8_t scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace ecospec {

moe_status_t verify_impl(const void *x, const moe_weights_t *w, const moe_routing_t *r, void *y, void *workspace,
                         size_t workspace_bytes, void *stream, void *const *events);
void set_last_error(const char *msg);

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_lock;
void *g_scratch[kMaxDevices];  // device address of `scratch` on each device (null: not looked up yet)

// The current device's copy of `scratch`.  In host code the array's name only
// stands for the symbol; its device address comes from the runtime, once per
// device, with that device current.
hipError_t scratch_of_current_device(void **out)
{
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_lock);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (!ptr) return hipErrorInvalidSymbol;
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace
}  // namespace ecospec

extern "C" moe_status_t moe_verify_layer_noalloc(const void *x, const moe_weights_t *w, const moe_routing_t *r,
                                                 void *y, void *stream)
{
    size_t need = 0;
    const moe_status_t st = moe_verify_workspace_size(w, r ? r->T : 0, r ? r->k : 0, &need);
    if (st != MOE_OK) return st;
    if (need > (size_t)MOE_NOALLOC_SCRATCH_BYTES) {
        char msg[160];
        snprintf(msg, sizeof msg, "moe_verify_layer_noalloc: the call needs %zu bytes of workspace, above the %zu of the "
                 "library's fixed scratch", need, (size_t)MOE_NOALLOC_SCRATCH_BYTES);
        ecospec::set_last_error(msg);
        return MOE_ERR_WORKSPACE;
    }
    void *ws = nullptr;
    const hipError_t err = ecospec::scratch_of_current_device(&ws);
    if (err != hipSuccess) {
        ecospec::set_last_error(hipGetErrorString(err));
        return MOE_ERR_HIP;
    }
    return ecospec::verify_impl(x, w, r, y, ws, (size_t)MOE_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}
