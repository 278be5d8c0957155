// Expert-copy pieces shared by the prefetch entry points and the decode driver.
#pragma once

#include <hip/hip_runtime.h>

#include "apex.h"

namespace apex {

// The device address of `bytes` bytes of pinned host memory at `host` (16-byte aligned),
// which the copy kernel reads.  Pageable memory, device memory and ranges whose last byte
// leaves pinned memory are refused with APEX_E_INVAL naming `fn`: a kernel cannot read them.
apex_status pinned_device_view(const char *fn, const void *host, size_t bytes, const uint4 **dev);

// apex_expert_prefetch after argument checks, reading the experts at the device view
// `src`, with two differences: the slot table goes to `compute` when any expert is copied
// and to `compute_if_none` otherwise; and with publish_unchanged false a plan without
// copies publishes nothing (the caller keeps the device table equal to the host table,
// which such a plan does not change).
apex_status expert_prefetch(const uint4 *src, uint16_t *slots, int E, int C, size_t expert_bytes,
                            const int32_t *pf_idx, const int32_t *pf_count, int B, int k_max,
                            int64_t step, int32_t *expert_of_slot, int64_t *last_used,
                            int32_t *slot_of_expert_dev, uint8_t *avail_dev, hipStream_t side,
                            hipStream_t compute, hipStream_t compute_if_none,
                            hipEvent_t readers_done, hipEvent_t ready, int32_t *copied_experts,
                            int *n_copied, bool publish_unchanged);

// apex_expert_fetch_misses after argument checks, reading the experts at the device view
// `src` (the decode driver keeps one per layer, so no pointer query per call); with src
// NULL the view of host_experts is looked up (and pageable memory refused) after the
// capacity check.
apex_status fetch_misses(const uint16_t *host_experts, const uint4 *src, uint16_t *scratch,
                         int n_scratch, int E, int C, size_t expert_bytes, const int32_t *route_idx, int B, int k,
                         const int32_t *expert_of_slot, int32_t *miss_table_dev,
                         hipStream_t side, hipStream_t compute, hipEvent_t scratch_free,
                         hipEvent_t ready, int32_t *missing, int *n_missing);

}  // namespace apex
