// apex_moe_ffn, apex_moe_ffn_fp8, apex_moe_ffn_mxfp4 and apex_moe_ffn_fp32: argument
// checks and the choice between the batch-1 paths (ffn_b1*.hip) and the grouped
// matrix-core path (ffn_gemm.hip; not for 32-bit experts).
#include <hip/hip_runtime.h>

#include "ffn_internal.h"

extern "C" size_t apex_moe_ffn_workspace_bytes(int B, int d, int I, int k) {
    if (B <= 0 || k <= 0 || I <= 0 || d <= 0) return 256;
    return B == 1 ? apex::ffn_b1_workspace(d, I, k) : apex::ffn_grouped_workspace(B, d, I, k);
}

extern "C" apex_status apex_moe_ffn_plan(int B, int d, int I, int E, int k, int n_slots,
                                         int weights, int32_t *plan) {
    APEX_REQUIRE(plan, "apex_moe_ffn_plan: NULL pointer");
    APEX_REQUIRE(weights >= APEX_WEIGHTS_BF16 && weights <= APEX_WEIGHTS_FP32,
                 "apex_moe_ffn_plan: weights=%d is not an APEX_WEIGHTS_* value", weights);
    APEX_REQUIRE(B >= 0 && d >= 1 && I >= 1 && E >= 1 && k >= 1 && k <= E && n_slots >= 1,
                 "apex_moe_ffn_plan: B=%d d=%d I=%d E=%d k=%d n_slots=%d out of range", B, d, I,
                 E, k, n_slots);
    plan[0] = plan[1] = plan[2] = 0;
    if (B < 2) return APEX_OK;
    if (weights == APEX_WEIGHTS_FP32)
        return apex::fail(APEX_E_UNSUPPORTED,
                          "apex_moe_ffn_plan: 32-bit experts run at batch 1 only (B=%d)", B);
    apex::ffn_grouped_plan(B, d, I, E, k, n_slots, apex::format_of(weights), plan);
    return APEX_OK;
}

apex_status apex::moe_ffn_checked(const char *fn, apex::WeightFormat fmt, const float *x, int B,
                                  int d, int I, int E, int k,
                    const int32_t *exec_idx, const float *exec_gate,
                    const int32_t *slot_of_expert, const void *slots, int n_slots, float *y,
                    int accumulate, void *workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    // one 16-byte load holds 4 fp32, 8 bf16 or 16 E4M3 weights; MXFP4 rows are whole
    // 32-value blocks
    const int mult = fmt == apex::WeightFormat::kF32    ? 4
                     : fmt == apex::WeightFormat::kBf16 ? 8
                     : fmt == apex::WeightFormat::kE4M3 ? 16
                                                        : 32;
    APEX_REQUIRE(B >= 0, "%s: B=%d must be >= 0", fn, B);
    APEX_REQUIRE(E >= 1, "%s: E=%d must be >= 1", fn, E);
    if (E > APEX_MAX_EXPERTS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: E=%d exceeds %d", fn, E, APEX_MAX_EXPERTS);
    APEX_REQUIRE(k >= 1 && k <= E, "%s: k=%d out of [1, E=%d]", fn, k, E);
    APEX_REQUIRE(d >= mult && d % mult == 0, "%s: d=%d must be a positive multiple of %d", fn,
                 d, mult);
    APEX_REQUIRE(I >= mult && I % mult == 0, "%s: I=%d must be a positive multiple of %d", fn,
                 I, mult);
    APEX_REQUIRE(n_slots >= 1, "%s: n_slots=%d must be >= 1", fn, n_slots);
    if (size_t(B) * k > APEX_MAX_PAIRS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: B*k=%d exceeds %d", fn, B * k, APEX_MAX_PAIRS);
    if (B == 0) return APEX_OK;
    if (fmt == apex::WeightFormat::kF32 && B >= 2)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: 32-bit experts run at batch 1 only (B=%d)",
                          fn, B);
    APEX_REQUIRE(x && exec_idx && exec_gate && slot_of_expert && slots && y && workspace,
                 "%s: NULL pointer", fn);
    APEX_REQUIRE(apex::aligned16(x) && apex::aligned16(slots) && apex::aligned16(workspace) &&
                     apex::aligned16(y),
                 "%s: x, slots, y and workspace must be 16-byte aligned", fn);
    const size_t need = apex_moe_ffn_workspace_bytes(B, d, I, k);
    if (workspace_bytes < need)
        return apex::fail(APEX_E_CAPACITY, "%s: workspace %zu < %zu bytes", fn, workspace_bytes,
                          need);
    if (B == 1) {
        float *h = static_cast<float *>(workspace);
        const uint8_t *codes = static_cast<const uint8_t *>(slots);
        if (fmt == apex::WeightFormat::kE4M3)
            return apex::ffn_b1_fp8(x, d, I, E, k, exec_idx, exec_gate, slot_of_expert, codes,
                                    n_slots, h, y, accumulate, stream);
        if (fmt == apex::WeightFormat::kMxfp4)
            return apex::ffn_b1_mxfp4(x, d, I, E, k, exec_idx, exec_gate, slot_of_expert, codes,
                                      n_slots, h, y, accumulate, stream);
        if (fmt == apex::WeightFormat::kF32)
            return apex::ffn_b1_fp32(x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                                     static_cast<const float *>(slots), n_slots, h, y,
                                     accumulate, stream);
        return apex::ffn_b1(x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                            static_cast<const uint16_t *>(slots), n_slots, h, y, accumulate,
                            stream);
    }
    return apex::ffn_grouped(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots,
                             n_slots, fmt, y, accumulate, workspace, stream);
}

extern "C" apex_status apex_moe_ffn(const float *x, int B, int d, int I, int E, int k,
                                    const int32_t *exec_idx, const float *exec_gate,
                                    const int32_t *slot_of_expert, const uint16_t *slots,
                                    int n_slots, float *y, int accumulate, void *workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
    return apex::moe_ffn_checked("apex_moe_ffn", apex::WeightFormat::kBf16, x, B, d, I, E, k, exec_idx,
                   exec_gate, slot_of_expert, slots, n_slots, y, accumulate, workspace,
                   workspace_bytes, stream);
}

extern "C" apex_status apex_moe_ffn_fp8(const float *x, int B, int d, int I, int E, int k,
                                        const int32_t *exec_idx, const float *exec_gate,
                                        const int32_t *slot_of_expert, const void *slots,
                                        int n_slots, float *y, int accumulate, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
    return apex::moe_ffn_checked("apex_moe_ffn_fp8", apex::WeightFormat::kE4M3, x, B, d, I, E, k, exec_idx,
                   exec_gate, slot_of_expert, slots, n_slots, y, accumulate, workspace,
                   workspace_bytes, stream);
}

extern "C" apex_status apex_moe_ffn_mxfp4(const float *x, int B, int d, int I, int E, int k,
                                          const int32_t *exec_idx, const float *exec_gate,
                                          const int32_t *slot_of_expert, const void *slots,
                                          int n_slots, float *y, int accumulate,
                                          void *workspace, size_t workspace_bytes,
                                          hipStream_t stream) {
    return apex::moe_ffn_checked("apex_moe_ffn_mxfp4", apex::WeightFormat::kMxfp4, x, B, d, I, E, k,
                   exec_idx, exec_gate, slot_of_expert, slots, n_slots, y, accumulate,
                   workspace, workspace_bytes, stream);
}

extern "C" apex_status apex_moe_ffn_fp32(const float *x, int B, int d, int I, int E, int k,
                                         const int32_t *exec_idx, const float *exec_gate,
                                         const int32_t *slot_of_expert, const void *slots,
                                         int n_slots, float *y, int accumulate, void *workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
    return apex::moe_ffn_checked("apex_moe_ffn_fp32", apex::WeightFormat::kF32, x, B, d, I, E,
                                 k, exec_idx, exec_gate, slot_of_expert, slots, n_slots, y,
                                 accumulate, workspace, workspace_bytes, stream);
}
