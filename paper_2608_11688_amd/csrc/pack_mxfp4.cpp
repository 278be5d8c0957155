// Packing of experts with 4-bit MXFP4 weights (apex_expert_bytes_mxfp4,
// apex_pack_expert_mxfp4).  Host code only.
//
// Slot layout (d and I multiples of 32; 3*d*I/2 + 3*d*I/32 bytes):
//   [I rows of (W1[i, :] codes, d/2 bytes | W3[i, :] codes, d/2 bytes)]
//   [W2 codes, d rows of I/2 bytes]
//   [scale bytes: W1 (I rows of d/32), W3 (I rows of d/32), W2 (d rows of I/32)]
// Codes are FP4 E2M1 (sign, 2 exponent bits with bias 1, 1 mantissa bit), two per byte,
// element 2j of a row in the low nibble of byte j.  Each block of 32 consecutive values
// of a row shares the scale 2^X, stored as the byte X + 127, with X = floor(log2 of the
// block's largest magnitude) - 2; elements are v / 2^X rounded to the nearest E2M1 value
// (ties to the even code, magnitudes above 6 clamped to 6, sign bit for v < 0).  A block
// of zeros gets X = -127 and codes 0.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "common.h"

namespace {

double bf16_value(uint16_t bits) {
    const uint32_t u = uint32_t(bits) << 16;
    float f;
    std::memcpy(&f, &u, sizeof f);
    return f;
}

// Nearest E2M1 code of a value already divided by its block scale.
uint8_t e2m1_code(double v) {
    static const double mag[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};
    const uint8_t sign = v < 0 ? 0x8 : 0x0;
    const double a = std::fmin(std::fabs(v), 6.0);
    int c = 0;
    while (c < 7 && mag[c + 1] <= a) ++c;          // mag[c] <= a < mag[c + 1] (or c = 7)
    if (c < 7) {
        const double below = a - mag[c], above = mag[c + 1] - a;
        if (above < below || (above == below && (c + 1) % 2 == 0)) ++c;
    }
    return sign | uint8_t(c);
}

// `rows` rows of `cols` bf16 values (row r at src + r * stride) into packed codes (row r
// at codes + r * code_stride bytes) and scale bytes (row r at scales + r * cols / 32).
void quantize(const uint16_t *src, size_t rows, size_t cols, size_t stride, uint8_t *codes,
              size_t code_stride, uint8_t *scales) {
    for (size_t r = 0; r < rows; ++r) {
        const uint16_t *in = src + r * stride;
        uint8_t *out = codes + r * code_stride;
        for (size_t b = 0; b < cols / 32; ++b) {
            double v[32], peak = 0.0;
            for (int c = 0; c < 32; ++c) {
                v[c] = bf16_value(in[32 * b + c]);
                peak = std::fmax(peak, std::fabs(v[c]));
            }
            int X = -127;
            if (peak > 0.0) {
                int e;
                std::frexp(peak, &e);                  // peak in [2^(e-1), 2^e)
                X = std::min(127, std::max(-127, e - 1 - 2));
            }
            scales[r * (cols / 32) + b] = uint8_t(X + 127);
            for (int c = 0; c < 32; c += 2) {
                const uint8_t lo = e2m1_code(std::ldexp(v[c], -X));
                const uint8_t hi = e2m1_code(std::ldexp(v[c + 1], -X));
                out[16 * b + c / 2] = uint8_t(lo | (hi << 4));
            }
        }
    }
}

}  // namespace

extern "C" size_t apex_expert_bytes_mxfp4(int d, int I) {
    if (d <= 0 || I <= 0) return 0;
    const size_t dI = size_t(d) * size_t(I);
    return 3 * dI / 2 + 3 * dI / 32;
}

extern "C" apex_status apex_pack_expert_mxfp4(const uint16_t *w1, const uint16_t *w3,
                                              const uint16_t *w2, int d, int I, void *out) {
    APEX_REQUIRE(w1 && w3 && w2 && out, "apex_pack_expert_mxfp4: NULL pointer");
    APEX_REQUIRE(d > 0 && I > 0 && d % 32 == 0 && I % 32 == 0,
                 "apex_pack_expert_mxfp4: d=%d I=%d must be positive multiples of 32", d, I);
    const size_t D = size_t(d), N = size_t(I);
    uint8_t *codes = static_cast<uint8_t *>(out);
    uint8_t *scales = codes + 3 * N * D / 2;
    quantize(w1, N, D, D, codes, D, scales);
    quantize(w3, N, D, D, codes + D / 2, D, scales + N * D / 32);
    quantize(w2, D, N, N, codes + N * D, N / 2, scales + 2 * N * D / 32);
    return APEX_OK;
}
