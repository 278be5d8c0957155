// Packing of experts with 32-bit weights (apex_expert_bytes_fp32, apex_pack_expert_fp32):
// the bf16 experts widened exactly to fp32, in the bf16 slot's order.  Host code only.
//
// Slot layout (12*d*I bytes):
//   [I rows of (W1[i, :], d floats | W3[i, :], d floats)]
//   [W2, d rows of I floats]
#include <cstring>

#include "common.h"

namespace {

float bf16_value(uint16_t bits) {
    const uint32_t u = uint32_t(bits) << 16;
    float f;
    std::memcpy(&f, &u, sizeof f);
    return f;
}

}  // namespace

extern "C" size_t apex_expert_bytes_fp32(int d, int I) {
    if (d <= 0 || I <= 0) return 0;
    return size_t(12) * size_t(d) * size_t(I);
}

extern "C" apex_status apex_pack_expert_fp32(const uint16_t *w1, const uint16_t *w3,
                                             const uint16_t *w2, int d, int I, void *out) {
    APEX_REQUIRE(w1 && w3 && w2 && out, "apex_pack_expert_fp32: NULL pointer");
    APEX_REQUIRE(d > 0 && I > 0 && d % 4 == 0 && I % 4 == 0,
                 "apex_pack_expert_fp32: d=%d and I=%d must be positive multiples of 4", d, I);
    float *o = static_cast<float *>(out);
    for (size_t i = 0; i < size_t(I); ++i) {
        float *row = o + i * 2 * size_t(d);
        for (size_t c = 0; c < size_t(d); ++c) {
            row[c] = bf16_value(w1[i * d + c]);
            row[d + c] = bf16_value(w3[i * d + c]);
        }
    }
    float *o2 = o + size_t(2) * I * d;
    for (size_t n = 0; n < size_t(d) * I; ++n) o2[n] = bf16_value(w2[n]);
    return APEX_OK;
}
