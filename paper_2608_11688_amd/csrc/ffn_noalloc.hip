// apex_moe_ffn_noalloc: the expert FFN for callers that cannot allocate device memory.
//
// The workspace of apex_moe_ffn (the batch-1 intermediate h, or the grouped path's split
// partials, h and per-pair outputs) lives in a fixed device array of this file instead
// of a caller buffer.  Each GPU the library runs on holds its own copy of the array, at
// its own address, until the process ends.  In host code the array's name stands for
// nothing usable on the device, so the device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept; every kernel argument uses
// that address.  No call here allocates or frees memory.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ffn_internal.h"

namespace {

// Every kernel behind apex_moe_ffn writes each workspace byte it reads before reading it,
// so nothing here has to start at zero.
static __device__ __align__(256) unsigned char scratch[APEX_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void *g_scratch[kMaxDevices] = {};

// The device address of `scratch` on the current device, looked up on the first call on
// that device.
apex_status scratch_on_current_device(const char *fn, void **out) {
    int dev = -1;
    APEX_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: device %d is beyond the %d devices supported",
                          fn, dev, kMaxDevices);
    std::lock_guard<std::mutex> guard(g_lock);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return apex::fail(APEX_E_HIP, "%s: hipGetSymbolAddress of the workspace on device "
                              "%d failed: %s", fn, dev, hipGetErrorString(e));
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return APEX_OK;
}

}  // namespace

extern "C" apex_status apex_moe_ffn_noalloc(const float *x, int B, int d, int I, int E, int k,
                                            const int32_t *exec_idx, const float *exec_gate,
                                            const int32_t *slot_of_expert, const void *slots,
                                            int n_slots, int weights, float *y, int accumulate,
                                            hipStream_t stream) {
    const char *fn = "apex_moe_ffn_noalloc";
    APEX_REQUIRE(weights >= APEX_WEIGHTS_BF16 && weights <= APEX_WEIGHTS_FP32,
                 "%s: weights=%d is not an APEX_WEIGHTS_* value", fn, weights);
    if (weights == APEX_WEIGHTS_FP32 && B >= 2)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: 32-bit experts run at batch 1 only (B=%d)",
                          fn, B);
    if (B > 0 && B <= APEX_MAX_PAIRS && k >= 1 && d >= 1 && I >= 1) {
        const size_t need = apex_moe_ffn_workspace_bytes(B, d, I, k);
        if (need > APEX_NOALLOC_WORKSPACE_BYTES)
            return apex::fail(APEX_E_CAPACITY,
                              "%s: B=%d d=%d I=%d k=%d needs %zu workspace bytes, more than the "
                              "%zu this entry point holds; use apex_moe_ffn with a workspace",
                              fn, B, d, I, k, need, size_t(APEX_NOALLOC_WORKSPACE_BYTES));
    }
    void *ws = nullptr;
    apex_status st = scratch_on_current_device(fn, &ws);
    if (st != APEX_OK) return st;
    return apex::moe_ffn_checked(fn, apex::format_of(weights), x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                                 slots, n_slots, y, accumulate, ws, APEX_NOALLOC_WORKSPACE_BYTES,
                                 stream);
}
