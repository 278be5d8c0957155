// Packing of experts with 8-bit E4M3 weights and one fp32 scale per output row
// (apex_expert_bytes_fp8, apex_pack_expert_fp8).  Host code only.
//
// Slot layout (fp8 slots are 3*d*I + 4*(2*I + d) bytes, 16-byte aligned sections):
//   [I rows of (W1[i, :] codes, d bytes | W3[i, :] codes, d bytes)]
//   [W2 codes, d rows of I bytes]
//   [fp32 scales: W1 rows (I), W3 rows (I), W2 rows (d)]
// Each row r of a matrix W is stored as codes q = E4M3(W[r, :] / s_r) with
// s_r = fp32(max |W[r, :]| / 448), rounded to the nearest code with ties to the even
// code; W[r, :] is then s_r * q.  All-zero rows get s_r = 0.
#include <cmath>
#include <cstring>
#include <vector>

#include "common.h"

namespace {

double bf16_value(uint16_t bits) {
    const uint32_t u = uint32_t(bits) << 16;
    float f;
    std::memcpy(&f, &u, sizeof f);
    return f;
}

// Nearest E4M3 code of x, ties to even, sign bit for x < 0; |x| above 448 saturates.
uint8_t e4m3_code(double x) {
    const uint8_t sign = x < 0 ? 0x80 : 0x00;
    const double a = std::fabs(x);
    if (!(a < 448.0)) return sign | 0x7E;
    // round-half-even of a non-negative value to an integer
    const auto rne = [](double v) {
        const double f = std::floor(v);
        const double r = v - f;
        if (r > 0.5) return f + 1.0;
        if (r < 0.5) return f;
        return std::fmod(f, 2.0) == 0.0 ? f : f + 1.0;
    };
    if (a < 0.015625) {                           // subnormal range: m/8 * 2^-6, m <= 8
        const int m = int(rne(a * 512.0));       // m == 8 is the smallest normal, code 0x08
        return sign | uint8_t(m);
    }
    int ex;
    const double f = std::frexp(a, &ex);          // a = f * 2^ex, f in [0.5, 1)
    int e = ex - 1;                               // a in [2^e, 2^(e+1))
    int m = int(rne((2.0 * f - 1.0) * 8.0));
    if (m == 8) {
        m = 0;
        ++e;
    }
    int code = ((e + 7) << 3) | m;
    if (code > 0x7E) code = 0x7E;
    return sign | uint8_t(code);
}

// codes and scale of `rows` rows of `cols` bf16 values, row r at src + r * stride
void quantize(const uint16_t *src, size_t rows, size_t cols, size_t stride, uint8_t *codes,
              size_t code_stride, float *scales) {
    std::vector<double> row(cols);
    for (size_t r = 0; r < rows; ++r) {
        double peak = 0.0;
        for (size_t c = 0; c < cols; ++c) {
            row[c] = bf16_value(src[r * stride + c]);
            peak = std::fmax(peak, std::fabs(row[c]));
        }
        const float s = float(peak / 448.0);
        scales[r] = s;
        uint8_t *out = codes + r * code_stride;
        if (s == 0.f) {
            std::memset(out, 0, cols);
            continue;
        }
        for (size_t c = 0; c < cols; ++c) out[c] = e4m3_code(row[c] / double(s));
    }
}

}  // namespace

extern "C" size_t apex_expert_bytes_fp8(int d, int I) {
    if (d <= 0 || I <= 0) return 0;
    return size_t(3) * size_t(d) * size_t(I) + sizeof(float) * (size_t(2) * I + size_t(d));
}

extern "C" apex_status apex_pack_expert_fp8(const uint16_t *w1, const uint16_t *w3,
                                            const uint16_t *w2, int d, int I, void *out) {
    APEX_REQUIRE(w1 && w3 && w2 && out, "apex_pack_expert_fp8: NULL pointer");
    APEX_REQUIRE(d > 0 && I > 0 && d % 8 == 0 && I % 8 == 0,
                 "apex_pack_expert_fp8: d=%d I=%d must be positive multiples of 8", d, I);
    const size_t D = size_t(d), N = size_t(I);
    uint8_t *codes = static_cast<uint8_t *>(out);
    float *scales = reinterpret_cast<float *>(codes + 3 * N * D);
    quantize(w1, N, D, D, codes, 2 * D, scales);
    quantize(w3, N, D, D, codes + D, 2 * D, scales + N);
    quantize(w2, D, N, N, codes + 2 * N * D, N, scales + 2 * N);
    return APEX_OK;
}
