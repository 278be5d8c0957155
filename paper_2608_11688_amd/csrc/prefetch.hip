// Expert movement between pinned host memory and the HBM slot pools.
//
// apex_expert_prefetch: plan the layer's cache for this step (apex_plan_residency),
// then move every planned expert with ONE copy-kernel launch on the side stream, which
// reads the pinned host copies over PCIe and writes the HBM slots while the compute
// stream runs the attention window and the gate, and publish the new slot table to the
// compute stream with a one-wavefront kernel whose table travels in its kernel
// arguments, so the host may plan the next step at once without racing the device.
// apex_expert_fetch_misses: same mechanics for the correctness-preserving mode's
// missing routed experts, into a separate scratch pool.
//
// Why a kernel and not one DMA-engine copy per expert: each engine copy carries a fixed
// cost of about 10 us on top of the transfer (a 3.15 MB expert takes 65-69 us against 55
// at the link's peak) and about 8 us of host time to issue, and the copies of a layer are
// on the critical path whenever the attention window cannot hide them.  One launch moves
// all of a layer's experts at 51-54 GB/s; its workgroups mostly wait on PCIe reads and
// take few compute-unit cycles from the kernels running beside them.
//
// The grid is 24 workgroups, whatever the number of experts: the link is full from about
// 24 (fewer lose bandwidth: 16 reach 39-44 GB/s), while every read the copy keeps queued
// on the link delays the PCIe reads of other work (dispatch packets, kernel arguments,
// completion signals).  Three experts on 96 workgroups took a chain of three small
// kernels on another stream from 12 to 65 us; on 24 it takes 16.  Experts of 32 MB and
// more take 48: over milliseconds of copying that delay is hidden, and the rate rises
// from 56.3 to 57.5 GB/s (256 MB; the DMA engine reaches 57.0).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "prefetch_internal.h"

namespace {

struct Table {
    int32_t slot[APEX_MAX_EXPERTS];
};

// Expert list of one copy launch: workgroup row y moves expert `from[y]` of the host
// array into slot `to[y]` of the pool.
struct CopyPlan {
    int32_t from[APEX_MAX_EXPERTS];
    int32_t to[APEX_MAX_EXPERTS];
};

constexpr int kCopyThreads = 256;       // one 16-byte word per thread per chunk
constexpr int kCopyGroups = 24;         // workgroups per launch
constexpr int kCopyGroupsLarge = 48;    //   for experts of kLargeExpert bytes and more
constexpr size_t kLargeExpert = size_t(32) << 20;

// The n experts of a launch are cut into chunks of kCopyThreads 16-byte words, numbered
// expert by expert (chunks_per_expert each, the last one ragged); workgroup g moves
// chunks g, g + grid, g + 2 * grid, ...  n16 = expert bytes / 16.
__global__ __launch_bounds__(kCopyThreads) void expert_copy_kernel(
    const uint4 *__restrict__ src, uint4 *__restrict__ dst, uint32_t n16,
    uint32_t chunks_per_expert, uint32_t chunks, CopyPlan plan) {
    for (uint32_t c = blockIdx.x; c < chunks; c += gridDim.x) {
        const uint32_t i = c / chunks_per_expert;
        const uint32_t j = (c - i * chunks_per_expert) * kCopyThreads + threadIdx.x;
        if (j < n16) dst[size_t(plan.to[i]) * n16 + j] = src[size_t(plan.from[i]) * n16 + j];
    }
}

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

}  // namespace

apex_status apex::pinned_device_view(const char *fn, const void *host, size_t bytes,
                               const uint4 **dev) {
    APEX_REQUIRE(reinterpret_cast<uintptr_t>(host) % 16 == 0,
                 "%s: host_experts %p is not 16-byte aligned", fn, host);
    hipPointerAttribute_t first{}, last{};
    const char *end = static_cast<const char *>(host) + (bytes - 1);
    const bool ok = hipPointerGetAttributes(&first, host) == hipSuccess &&
                    hipPointerGetAttributes(&last, end) == hipSuccess;
    (void)hipGetLastError();   // a refused query must not surface in a later call
    APEX_REQUIRE(ok && first.type == hipMemoryTypeHost && first.devicePointer &&
                     last.type == hipMemoryTypeHost &&
                     static_cast<const char *>(last.devicePointer) ==
                         static_cast<const char *>(first.devicePointer) + (bytes - 1),
                 "%s: host_experts (%zu bytes at %p) must be pinned host memory "
                 "(hipHostMalloc or equivalent)", fn, bytes, host);
    *dev = static_cast<const uint4 *>(first.devicePointer);
    return APEX_OK;
}

namespace {

// n >= 1 experts of expert_bytes (a multiple of 16, at most 16 * UINT32_MAX; checked by
// the entry points).
apex_status copy_experts(const uint4 *src, void *pool, size_t expert_bytes, const CopyPlan &plan,
                         int n, hipStream_t stream) {
    const uint32_t n16 = uint32_t(expert_bytes / 16);
    const uint32_t per = (n16 + kCopyThreads - 1) / kCopyThreads;
    const uint32_t chunks = per * uint32_t(n);
    const uint32_t groups = expert_bytes >= kLargeExpert ? kCopyGroupsLarge : kCopyGroups;
    const uint32_t grid = std::min<uint32_t>(groups, chunks);
    hipLaunchKernelGGL(expert_copy_kernel, dim3(grid), dim3(kCopyThreads), 0, stream, src,
                       static_cast<uint4 *>(pool), n16, per, chunks, plan);
    APEX_HIP(hipGetLastError());
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

apex_status apex::expert_prefetch(
    const uint4 *src, uint16_t *slots, int E, int C, size_t expert_bytes, const int32_t *pf_idx,
    const int32_t *pf_count, int B, int k_max, int64_t step, int32_t *expert_of_slot,
    int64_t *last_used, int32_t *slot_of_expert_dev, uint8_t *avail_dev, hipStream_t side,
    hipStream_t compute, hipStream_t compute_if_none, hipEvent_t readers_done, hipEvent_t ready,
    int32_t *copied_experts, int *n_copied, bool publish_unchanged) {
    int32_t ce[APEX_MAX_EXPERTS], cs[APEX_MAX_EXPERTS];
    int n = 0;
    apex_status st = apex_plan_residency(E, C, pf_idx, pf_count, B, k_max, step, expert_of_slot,
                                         last_used, ce, cs, &n);
    if (st != APEX_OK) return st;

    st = wait_unless_done(side, readers_done);
    if (st != APEX_OK) return st;
    if (n > 0) {
        CopyPlan plan;
        for (int i = 0; i < n; ++i) {
            plan.from[i] = ce[i];
            plan.to[i] = cs[i];
        }
        st = copy_experts(src, slots, expert_bytes, plan, n, side);
        if (st != APEX_OK) return st;
    }
    if (ready) APEX_HIP(hipEventRecord(ready, side));

    // a plan without copies leaves the table as it was: its device copy needs no rewrite
    // unless the caller cannot vouch that the device copy is current
    if (n > 0 || publish_unchanged) {
        Table t;
        std::fill(t.slot, t.slot + APEX_MAX_EXPERTS, -1);
        for (int s = 0; s < C; ++s)
            if (expert_of_slot[s] >= 0) t.slot[expert_of_slot[s]] = s;
        st = publish(t, E, slot_of_expert_dev, avail_dev, n > 0 ? compute : compute_if_none);
        if (st != APEX_OK) return st;
    }
    if (copied_experts)
        for (int i = 0; i < n; ++i) copied_experts[i] = ce[i];
    if (n_copied) *n_copied = n;
    return APEX_OK;
}

extern "C" apex_status apex_expert_prefetch(
    const uint16_t *host_experts, uint16_t *slots, int E, int C, size_t expert_bytes,
    const int32_t *pf_idx, const int32_t *pf_count, int B, int k_max, int64_t step,
    int32_t *expert_of_slot, int64_t *last_used, int32_t *slot_of_expert_dev,
    uint8_t *avail_dev, hipStream_t side, hipStream_t compute, hipEvent_t readers_done,
    hipEvent_t ready, int32_t *copied_experts, int *n_copied) {
    const char *fn = "apex_expert_prefetch";
    APEX_REQUIRE(host_experts && slots && slot_of_expert_dev, "%s: NULL pointer", fn);
    APEX_REQUIRE(E >= 1 && E <= APEX_MAX_EXPERTS, "%s: E=%d out of [1, 64]", fn, E);
    APEX_REQUIRE(C >= 1 && C <= E, "%s: C=%d out of [1, E=%d]", fn, C, E);
    APEX_REQUIRE(expert_bytes > 0 && expert_bytes % 16 == 0 && expert_bytes / 16 <= UINT32_MAX,
                 "%s: expert_bytes=%zu must be a positive multiple of 16 below 64 GiB", fn,
                 expert_bytes);
    const uint4 *src = nullptr;
    apex_status st = apex::pinned_device_view(fn, host_experts, size_t(E) * expert_bytes, &src);
    if (st != APEX_OK) return st;
    return apex::expert_prefetch(src, slots, E, C, expert_bytes, pf_idx, pf_count, B, k_max,
                                 step, expert_of_slot, last_used, slot_of_expert_dev, avail_dev,
                                 side, compute, compute, readers_done, ready, copied_experts,
                                 n_copied, true);
}

apex_status apex::fetch_misses(const uint16_t *host_experts, const uint4 *src, uint16_t *scratch,
                              int n_scratch, int E, int C, size_t expert_bytes, const int32_t *route_idx, int B, int k,
                              const int32_t *expert_of_slot, int32_t *miss_table_dev,
                              hipStream_t side, hipStream_t compute, hipEvent_t scratch_free,
                              hipEvent_t ready, int32_t *missing, int *n_missing) {
    const char *fn = "apex_expert_fetch_misses";
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
    apex_status st = APEX_OK;
    if (!src) {
        st = apex::pinned_device_view(fn, host_experts, size_t(E) * expert_bytes, &src);
        if (st != APEX_OK) return st;
    }
    if (missing)
        for (int i = 0; i < n; ++i) missing[i] = list[i];
    *n_missing = n;
    if (n == 0) return APEX_OK;   // no second pass reads the table: nothing to enqueue
    st = wait_unless_done(side, scratch_free);
    if (st != APEX_OK) return st;
    CopyPlan plan;
    for (int i = 0; i < n; ++i) {
        plan.from[i] = list[i];
        plan.to[i] = i;
    }
    st = copy_experts(src, scratch, expert_bytes, plan, n, side);
    if (st != APEX_OK) return st;
    if (ready) APEX_HIP(hipEventRecord(ready, side));

    Table t;
    std::fill(t.slot, t.slot + APEX_MAX_EXPERTS, -1);
    for (int i = 0; i < n; ++i) t.slot[list[i]] = i;
    return publish(t, E, miss_table_dev, nullptr, compute);
}

extern "C" apex_status apex_expert_fetch_misses(
    const uint16_t *host_experts, uint16_t *scratch, int n_scratch, int E, int C,
    size_t expert_bytes, const int32_t *route_idx, int B, int k, const int32_t *expert_of_slot,
    int32_t *miss_table_dev, hipStream_t side, hipStream_t compute, hipEvent_t scratch_free,
    hipEvent_t ready, int32_t *missing, int *n_missing) {
    const char *fn = "apex_expert_fetch_misses";
    APEX_REQUIRE(host_experts && scratch && expert_of_slot && miss_table_dev && n_missing,
                 "%s: NULL pointer", fn);
    APEX_REQUIRE(E >= 1 && E <= APEX_MAX_EXPERTS, "%s: E=%d out of [1, 64]", fn, E);
    APEX_REQUIRE(C >= 1, "%s: C=%d must be >= 1", fn, C);
    APEX_REQUIRE(n_scratch >= 0, "%s: n_scratch=%d < 0", fn, n_scratch);
    APEX_REQUIRE(B >= 0 && k >= 1 && k <= E, "%s: B=%d k=%d", fn, B, k);
    APEX_REQUIRE(B == 0 || route_idx, "%s: NULL route_idx", fn);
    APEX_REQUIRE(expert_bytes > 0 && expert_bytes % 16 == 0 && expert_bytes / 16 <= UINT32_MAX,
                 "%s: expert_bytes=%zu must be a positive multiple of 16 below 64 GiB", fn,
                 expert_bytes);
    return apex::fetch_misses(host_experts, nullptr, scratch, n_scratch, E, C, expert_bytes,
                              route_idx, B, k, expert_of_slot, miss_table_dev, side, compute,
                              scratch_free, ready, missing, n_missing);
}
