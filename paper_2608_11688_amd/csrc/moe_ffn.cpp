// apex_moe_ffn: argument checks and the choice between the batch-1 path (ffn_b1.hip)
// and the grouped matrix-core path (ffn_gemm.hip).
#include <hip/hip_runtime.h>

#include "ffn_internal.h"

extern "C" size_t apex_moe_ffn_workspace_bytes(int B, int d, int I, int k) {
    if (B <= 0 || k <= 0 || I <= 0 || d <= 0) return 256;
    return B == 1 ? apex::ffn_b1_workspace(d, I, k) : apex::ffn_grouped_workspace(B, d, I, k);
}

extern "C" apex_status apex_moe_ffn(const float *x, int B, int d, int I, int E, int k,
                                    const int32_t *exec_idx, const float *exec_gate,
                                    const int32_t *slot_of_expert, const uint16_t *slots,
                                    int n_slots, float *y, int accumulate, void *workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
    const char *fn = "apex_moe_ffn";
    APEX_REQUIRE(B >= 0, "%s: B=%d must be >= 0", fn, B);
    APEX_REQUIRE(E >= 1, "%s: E=%d must be >= 1", fn, E);
    if (E > APEX_MAX_EXPERTS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: E=%d exceeds %d", fn, E, APEX_MAX_EXPERTS);
    APEX_REQUIRE(k >= 1 && k <= E, "%s: k=%d out of [1, E=%d]", fn, k, E);
    APEX_REQUIRE(d >= 8 && d % 8 == 0, "%s: d=%d must be a positive multiple of 8", fn, d);
    APEX_REQUIRE(I >= 8 && I % 8 == 0, "%s: I=%d must be a positive multiple of 8", fn, I);
    APEX_REQUIRE(n_slots >= 1, "%s: n_slots=%d must be >= 1", fn, n_slots);
    if (size_t(B) * k > APEX_MAX_PAIRS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: B*k=%d exceeds %d", fn, B * k, APEX_MAX_PAIRS);
    if (B == 0) return APEX_OK;
    APEX_REQUIRE(x && exec_idx && exec_gate && slot_of_expert && slots && y && workspace,
                 "%s: NULL pointer", fn);
    APEX_REQUIRE(apex::aligned16(x) && apex::aligned16(slots) && apex::aligned16(workspace) &&
                     apex::aligned16(y),
                 "%s: x, slots, y and workspace must be 16-byte aligned", fn);
    const size_t need = apex_moe_ffn_workspace_bytes(B, d, I, k);
    if (workspace_bytes < need)
        return apex::fail(APEX_E_CAPACITY, "%s: workspace %zu < %zu bytes", fn, workspace_bytes,
                          need);
    if (B == 1)
        return apex::ffn_b1(x, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots, n_slots,
                            static_cast<float *>(workspace), y, accumulate, stream);
    return apex::ffn_grouped(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert, slots,
                             n_slots, y, accumulate, workspace, stream);
}
