// Expert movement between pinned host memory and the HBM slot pools.
//
// apex_expert_prefetch: plan the layer's cache for this step (apex_plan_residency),
// then issue one contiguous host-to-device copy per planned expert on the side
// stream (the DMA engines move them while the compute stream runs the attention
// window and the gate), and publish the new slot table to the compute stream with a
// one-wavefront kernel whose table travels in its kernel arguments, so the host may
// plan the next step at once without racing the device.
// apex_expert_fetch_misses: same mechanics for the correctness-preserving mode's
// missing routed experts, into a separate scratch pool.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "common.h"

namespace {

struct Table {
    int32_t slot[APEX_MAX_EXPERTS];
};

__global__ void publish_table_kernel(Table t, int E, int32_t *__restrict__ slot_of_expert,
                                     uint8_t *__restrict__ avail) {
    const int e = threadIdx.x;
    if (e < E) {
        slot_of_expert[e] = t.slot[e];
        if (avail) avail[e] = t.slot[e] >= 0 ? 1 : 0;
    }
}

// Makes `stream` wait for `ev` unless the event has already completed (or was never
// recorded): the wait would then be a no-op, and enqueueing a cross-stream wait costs the
// host more than a kernel launch.
apex_status wait_unless_done(hipStream_t stream, hipEvent_t ev) {
    if (!ev || hipEventQuery(ev) == hipSuccess) return APEX_OK;
    APEX_HIP(hipStreamWaitEvent(stream, ev, 0));
    return APEX_OK;
}

apex_status publish(const Table &t, int E, int32_t *slot_dev, uint8_t *avail_dev,
                    hipStream_t stream) {
    hipLaunchKernelGGL(publish_table_kernel, dim3(1), dim3(APEX_MAX_EXPERTS), 0, stream, t, E,
                       slot_dev, avail_dev);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace

extern "C" apex_status apex_expert_prefetch(
    const uint16_t *host_experts, uint16_t *slots, int E, int C, size_t expert_bytes,
    const int32_t *pf_idx, const int32_t *pf_count, int B, int k_max, int64_t step,
    int32_t *expert_of_slot, int64_t *last_used, int32_t *slot_of_expert_dev,
    uint8_t *avail_dev, hipStream_t side, hipStream_t compute, hipEvent_t readers_done,
    hipEvent_t ready, int32_t *copied_experts, int *n_copied) {
    const char *fn = "apex_expert_prefetch";
    APEX_REQUIRE(host_experts && slots && slot_of_expert_dev && ready,
                 "%s: NULL pointer or event", fn);
    APEX_REQUIRE(E >= 1 && E <= APEX_MAX_EXPERTS, "%s: E=%d out of [1, 64]", fn, E);
    APEX_REQUIRE(C >= 1 && C <= E, "%s: C=%d out of [1, E=%d]", fn, C, E);
    APEX_REQUIRE(expert_bytes > 0 && expert_bytes % 16 == 0,
                 "%s: expert_bytes=%zu must be a positive multiple of 16", fn, expert_bytes);
    std::vector<int32_t> ce(C), cs(C);
    int n = 0;
    apex_status st = apex_plan_residency(E, C, pf_idx, pf_count, B, k_max, step, expert_of_slot,
                                         last_used, ce.data(), cs.data(), &n);
    if (st != APEX_OK) return st;

    st = wait_unless_done(side, readers_done);
    if (st != APEX_OK) return st;
    const char *src = reinterpret_cast<const char *>(host_experts);
    char *dst = reinterpret_cast<char *>(slots);
    for (int i = 0; i < n; ++i)
        APEX_HIP(hipMemcpyAsync(dst + size_t(cs[i]) * expert_bytes,
                                src + size_t(ce[i]) * expert_bytes, expert_bytes,
                                hipMemcpyHostToDevice, side));
    APEX_HIP(hipEventRecord(ready, side));

    Table t;
    std::fill(t.slot, t.slot + APEX_MAX_EXPERTS, -1);
    for (int s = 0; s < C; ++s)
        if (expert_of_slot[s] >= 0) t.slot[expert_of_slot[s]] = s;
    st = publish(t, E, slot_of_expert_dev, avail_dev, compute);
    if (st != APEX_OK) return st;
    if (copied_experts)
        for (int i = 0; i < n; ++i) copied_experts[i] = ce[i];
    if (n_copied) *n_copied = n;
    return APEX_OK;
}

extern "C" apex_status apex_expert_fetch_misses(
    const uint16_t *host_experts, uint16_t *scratch, int n_scratch, int E, int C,
    size_t expert_bytes, const int32_t *route_idx, int B, int k, const int32_t *expert_of_slot,
    int32_t *miss_table_dev, hipStream_t side, hipStream_t compute, hipEvent_t scratch_free,
    hipEvent_t ready, int32_t *missing, int *n_missing) {
    const char *fn = "apex_expert_fetch_misses";
    APEX_REQUIRE(host_experts && scratch && expert_of_slot && miss_table_dev && ready && n_missing,
                 "%s: NULL pointer or event", fn);
    APEX_REQUIRE(E >= 1 && E <= APEX_MAX_EXPERTS, "%s: E=%d out of [1, 64]", fn, E);
    APEX_REQUIRE(C >= 1, "%s: C=%d must be >= 1", fn, C);
    APEX_REQUIRE(n_scratch >= 0, "%s: n_scratch=%d < 0", fn, n_scratch);
    APEX_REQUIRE(B >= 0 && k >= 1 && k <= E, "%s: B=%d k=%d", fn, B, k);
    APEX_REQUIRE(B == 0 || route_idx, "%s: NULL route_idx", fn);
    APEX_REQUIRE(expert_bytes > 0 && expert_bytes % 16 == 0,
                 "%s: expert_bytes=%zu must be a positive multiple of 16", fn, expert_bytes);
    bool resident[APEX_MAX_EXPERTS] = {false};
    for (int s = 0; s < C; ++s) {
        const int e = expert_of_slot[s];
        APEX_REQUIRE(e >= -1 && e < E, "%s: expert_of_slot[%d]=%d", fn, s, e);
        if (e >= 0) resident[e] = true;
    }
    bool wanted[APEX_MAX_EXPERTS] = {false};
    for (int i = 0; i < B * k; ++i) {
        const int e = route_idx[i];
        APEX_REQUIRE(e >= 0 && e < E, "%s: route_idx[%d]=%d", fn, i, e);
        if (!resident[e]) wanted[e] = true;
    }
    int list[APEX_MAX_EXPERTS];
    int n = 0;
    for (int e = 0; e < E; ++e)
        if (wanted[e]) list[n++] = e;
    if (n > n_scratch)
        return apex::fail(APEX_E_CAPACITY, "%s: %d missing experts > %d scratch slots", fn, n,
                          n_scratch);

    if (missing)
        for (int i = 0; i < n; ++i) missing[i] = list[i];
    *n_missing = n;
    if (n == 0) return APEX_OK;   // no second pass reads the table: nothing to enqueue
    apex_status st = wait_unless_done(side, scratch_free);
    if (st != APEX_OK) return st;
    const char *src = reinterpret_cast<const char *>(host_experts);
    char *dst = reinterpret_cast<char *>(scratch);
    for (int i = 0; i < n; ++i)
        APEX_HIP(hipMemcpyAsync(dst + size_t(i) * expert_bytes, src + size_t(list[i]) * expert_bytes,
                                expert_bytes, hipMemcpyHostToDevice, side));
    APEX_HIP(hipEventRecord(ready, side));

    Table t;
    std::fill(t.slot, t.slot + APEX_MAX_EXPERTS, -1);
    for (int i = 0; i < n; ++i) t.slot[list[i]] = i;
    return publish(t, E, miss_table_dev, nullptr, compute);
}
