// Device helpers shared by the expert-FFN kernels: bf16 unpacking, 8-wide (bf16) and
// 16-wide (E4M3, MXFP4) dot products against fp32 activations, a wavefront sum and SiLU.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace apex {
namespace ffn {

constexpr int kWave = 64;

// Loads of data a kernel reads exactly once, whole cache lines at a time (the expert
// weight codes): marked non-temporal, so the stream does not push the activations that
// every wavefront re-reads (x, h) out of L2 and the Infinity Cache.  Mixtral-shaped
// batch-1 call: 119.8 -> 109.7 us.  Scales are not loaded this way: a line of them
// serves several loads (MXFP4 block scales of consecutive K blocks, an E4M3 row scale
// read by every unrolled step), and marked non-temporal it is fetched again for each.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 ld_stream(const uint4 *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 ld_stream(const uint2 *p) {
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(p));
    return make_uint2(v.x, v.y);
}

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

// The fp32 value 2^(b - 127) of an MX scale byte b (b = 0 is the subnormal 2^-127).
__device__ __forceinline__ float mx_scale(uint32_t b) {
    return __uint_as_float(b ? b << 23 : 0x00400000u);
}

// 16 FP4 E2M1 codes (two per byte of w, the low nibble first) times x[0..3] (16 fp32
// values), each code widened and multiplied by its block scale exactly in hardware.
__device__ __forceinline__ float dot16_mxfp4(uint2 w, float scale, const float4 (&x)[4],
                                             float acc) {
    const uint32_t word[2] = {w.x, w.y};
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const auto p0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word[q], scale, 0);
        const auto p1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word[q], scale, 1);
        const auto p2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word[q], scale, 2);
        const auto p3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word[q], scale, 3);
        const float4 a = x[2 * q], b = x[2 * q + 1];
        acc = fmaf(p0[0], a.x, acc);
        acc = fmaf(p0[1], a.y, acc);
        acc = fmaf(p1[0], a.z, acc);
        acc = fmaf(p1[1], a.w, acc);
        acc = fmaf(p2[0], b.x, acc);
        acc = fmaf(p2[1], b.y, acc);
        acc = fmaf(p3[0], b.z, acc);
        acc = fmaf(p3[1], b.w, acc);
    }
    return acc;
}

}  // namespace ffn
}  // namespace apex
