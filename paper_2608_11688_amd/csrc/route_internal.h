// Router launches with an optional host-visible completion flag, for the decode driver.
#pragma once

#include <hip/hip_runtime.h>

#include "apex.h"

namespace apex {

// apex_prefetch_route / apex_gate_topk; in addition, when `done` is not NULL, each token
// b's workgroup writes done[b] = seq once its outputs (including those in host memory)
// are visible to the system.  `done` is [B] int32 in pinned host memory.
apex_status prefetch_route(const float *h_pre, const uint16_t *w_pf, const float *b_pf, int B,
                           int d, int E, int k, int k_max, int policy, float tau,
                           int static_delta, const float *cdf_w, const float *cdf_theta,
                           int32_t *pf_idx, int32_t *pf_count, float *pf_prob, int32_t *done,
                           int32_t seq, hipStream_t stream);
apex_status gate_topk(const float *h_post, const uint16_t *w_g, const float *b_g, int B, int d,
                      int E, int k, int mode, const uint8_t *avail, int avail_stride,
                      int32_t *route_idx, float *route_gate, int32_t *exec_idx, float *exec_gate,
                      float *gate_prob, int32_t *done, int32_t seq, hipStream_t stream);

}  // namespace apex
