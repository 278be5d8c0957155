// Launchers of the two expert-FFN paths behind apex_moe_ffn.  Arguments are checked by
// the entry point before either is called; both enqueue on `stream` and return
// APEX_E_HIP if a launch fails.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "common.h"

namespace apex {

// Expert weight formats of a slot pool.
enum class WeightFormat { kBf16, kE4M3, kMxfp4, kF32 };

// The format of an apex_weights code (checked to be in range by the caller).
inline WeightFormat format_of(int weights) {
    return weights == APEX_WEIGHTS_FP8_E4M3 ? WeightFormat::kE4M3
           : weights == APEX_WEIGHTS_MXFP4  ? WeightFormat::kMxfp4
           : weights == APEX_WEIGHTS_FP32   ? WeightFormat::kF32
                                            : WeightFormat::kBf16;
}

// One token: up_b1 then down_b1.  `h` is k x I fp32 scratch.
size_t ffn_b1_workspace(int d, int I, int k);
apex_status ffn_b1(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                   const float *exec_gate, const int32_t *slot_of_expert, const uint16_t *slots,
                   int n_slots, float *h, float *y, int accumulate, hipStream_t stream);

// The same over apex_pack_expert_fp8 slots (d and I multiples of 16).
apex_status ffn_b1_fp8(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                       const float *exec_gate, const int32_t *slot_of_expert,
                       const uint8_t *slots, int n_slots, float *h, float *y, int accumulate,
                       hipStream_t stream);

// The same over apex_pack_expert_mxfp4 slots (d and I multiples of 32).
apex_status ffn_b1_mxfp4(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                         const float *exec_gate, const int32_t *slot_of_expert,
                         const uint8_t *slots, int n_slots, float *h, float *y, int accumulate,
                         hipStream_t stream);

// The same over apex_pack_expert_fp32 slots (d and I multiples of 4).
apex_status ffn_b1_fp32(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                        const float *exec_gate, const int32_t *slot_of_expert,
                        const float *slots, int n_slots, float *h, float *y, int accumulate,
                        hipStream_t stream);

// Two or more tokens: grouped GEMMs on the matrix cores, over slots of format fmt.  `workspace` is 256-byte aligned and holds ffn_grouped_workspace(B, d, I, k)
// bytes.
size_t ffn_grouped_workspace(int B, int d, int I, int k);
// The grouped path's launch plan: out = {token tiles per pass, gate/up K splits, down K
// splits}.
void ffn_grouped_plan(int B, int d, int I, int E, int k, int n_slots, WeightFormat fmt,
                      int32_t out[3]);
apex_status ffn_grouped(const float *x, int B, int d, int I, int E, int k,
                        const int32_t *exec_idx, const float *exec_gate,
                        const int32_t *slot_of_expert, const void *slots, int n_slots,
                        WeightFormat fmt, float *y, int accumulate, void *workspace,
                        hipStream_t stream);

// apex_moe_ffn in format fmt with its argument checks, `fn` naming the entry point in
// error messages (moe_ffn.cpp).
apex_status moe_ffn_checked(const char *fn, WeightFormat fmt, const float *x, int B, int d,
                            int I, int E, int k, const int32_t *exec_idx, const float *exec_gate,
                            const int32_t *slot_of_expert, const void *slots, int n_slots,
                            float *y, int accumulate, void *workspace, size_t workspace_bytes,
                            hipStream_t stream);

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace apex
