// Device helpers shared by the expert-FFN kernels: bf16 unpacking, 8-wide (bf16) and
// 16-wide (E4M3) dot products against fp32 activations, a wavefront sum and SiLU.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace apex {
namespace ffn {

constexpr int kWave = 64;

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float dot8(uint4 w, float4 a, float4 b, float acc) {
    acc = fmaf(bf_lo(w.x), a.x, acc);
    acc = fmaf(bf_hi(w.x), a.y, acc);
    acc = fmaf(bf_lo(w.y), a.z, acc);
    acc = fmaf(bf_hi(w.y), a.w, acc);
    acc = fmaf(bf_lo(w.z), b.x, acc);
    acc = fmaf(bf_hi(w.z), b.y, acc);
    acc = fmaf(bf_lo(w.w), b.z, acc);
    acc = fmaf(bf_hi(w.w), b.w, acc);
    return acc;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float silu(float u) { return u / (1.f + expf(-u)); }

// 16 E4M3 codes (the little-endian bytes of w) times x[0..3] (16 fp32 values); the
// hardware conversion is exact, the products accumulate in fp32.
__device__ __forceinline__ float dot16_e4m3(uint4 w, const float4 (&x)[4], float acc) {
    const uint32_t word[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(int(word[q]), false);   // bytes 0, 1
        const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(int(word[q]), true);    // bytes 2, 3
        acc = fmaf(lo[0], x[q].x, acc);
        acc = fmaf(lo[1], x[q].y, acc);
        acc = fmaf(hi[0], x[q].z, acc);
        acc = fmaf(hi[1], x[q].w, acc);
    }
    return acc;
}

}  // namespace ffn
}  // namespace apex
