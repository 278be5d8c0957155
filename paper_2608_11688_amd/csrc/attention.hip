// Decode attention of one layer (apex_attention_decode): the block whose run time the
// expert prefetch overlaps.
//
// Four launches per call:
//   attn_qkv    grid (ceil(R / 4), B), R = (H + 2G) * hd: one wavefront per row of W_qkv,
//               all loads of the row issued before the multiplies.  Query rows go to the
//               workspace (fp32); key and value rows are rounded to bf16 and stored at
//               position pos of the caches.
//   attn_split  grid (S, G, B): positions 0..pos split S ways; a workgroup takes one
//               split of one key/value head for the H / G query heads that share it.
//               The lanes of one position hold 8 dimensions each (hd / 8 lanes per
//               position); every position slot keeps a running maximum, normaliser and
//               weighted sum of values per query head (online softmax), and the slots
//               are merged with the log-sum-exp rule, across the wavefront by shuffles
//               and across wavefronts in LDS.  Output per (token, head, split):
//               hd weighted sums, the maximum and the normaliser.
//   attn_merge  grid (H, B): the splits of one head merged (log-sum-exp rule) into the
//               attention vector, all of its loads issued at once.
//   attn_out    grid (ceil(d / 4), B): one wavefront per row of W_o.
// fp32 arithmetic on bf16 weights and caches; no atomics, so results are deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "common.h"
#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::dot8;
using apex::ffn::kWave;
using apex::ffn::wave_sum;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxGroup = 8;       // query heads per key/value head
constexpr int kOutRows = kWaves;   // W_o rows per attn_out workgroup (one per wavefront)
constexpr int kMaxSplits = kThreads;   // position splits (one merge thread each)

__device__ __forceinline__ uint16_t bf16_bits(float v) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

template <int NPL>
__global__ __launch_bounds__(kThreads) void attn_qkv(
    const float *__restrict__ h, const uint16_t *__restrict__ w_qkv, int d, int H, int G,
    int hd, uint16_t *__restrict__ k_cache, uint16_t *__restrict__ v_cache, int ctx_max,
    int pos, float *__restrict__ q) {
    const int b = blockIdx.y;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int R = (H + 2 * G) * hd;
    const int r = blockIdx.x * kWaves + wave;
    if (r >= R) return;
    const int nch = d / 8;
    const uint4 *row = reinterpret_cast<const uint4 *>(w_qkv + size_t(r) * d);
    const float4 *x4 = reinterpret_cast<const float4 *>(h + size_t(b) * d);
    float acc = 0.f;
    for (int c0 = 0; c0 < nch; c0 += NPL * kWave) {
        uint4 w[NPL];
        float4 a[NPL], bb[NPL];
#pragma unroll
        for (int n = 0; n < NPL; ++n) {
            const int c = min(c0 + lane + n * kWave, nch - 1);
            w[n] = row[c];
            a[n] = x4[2 * c];
            bb[n] = x4[2 * c + 1];
        }
#pragma unroll
        for (int n = 0; n < NPL; ++n)
            if (c0 + lane + n * kWave < nch) acc = dot8(w[n], a[n], bb[n], acc);
    }
    const float v = wave_sum(acc);
    if (lane != 0) return;
    const int qrows = H * hd;
    if (r < qrows) {
        q[size_t(b) * qrows + r] = v;
        return;
    }
    const int kv = r - qrows;
    const bool is_v = kv >= G * hd;
    const int gr = is_v ? kv - G * hd : kv;
    const int g = gr / hd, dim = gr % hd;
    uint16_t *cache = is_v ? v_cache : k_cache;
    cache[((size_t(b) * G + g) * ctx_max + pos) * hd + dim] = bf16_bits(v);
}

// (m, l, acc) of one query head merged with another's (log-sum-exp rule); an empty state
// has m = -inf and l = 0.
__device__ __forceinline__ void merge_state(float &m, float &l, float (&acc)[8], float m2,
                                            float l2, const float (&acc2)[8]) {
    const float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;
    const float c1 = expf(m - mn), c2 = expf(m2 - mn);
    l = l * c1 + l2 * c2;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = acc[t] * c1 + acc2[t] * c2;
    m = mn;
}

template <int HD, int GR>
__global__ __launch_bounds__(kThreads) void attn_split(
    const float *__restrict__ q, const uint16_t *__restrict__ k_cache,
    const uint16_t *__restrict__ v_cache, int H, int G, int ctx_max, int n_pos, float scale,
    float *__restrict__ part) {
    constexpr int LPP = HD / 8;              // lanes per position
    constexpr int PPW = kWave / LPP;         // position slots per wavefront
    constexpr int SLOTS = kWaves * PPW;
    __shared__ float red_m[kWaves][GR], red_l[kWaves][GR];
    __shared__ float red_acc[kWaves][GR][HD];
    const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z, S = gridDim.x;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int sub = lane % LPP, slot = wave * PPW + lane / LPP;
    const int dim0 = 8 * sub;
    const int j_lo = int((long long)s * n_pos / S), j_hi = int((long long)(s + 1) * n_pos / S);

    float qv[GR][8];
#pragma unroll
    for (int i = 0; i < GR; ++i) {
        const float *qi = q + (size_t(b) * H + g * GR + i) * HD + dim0;
#pragma unroll
        for (int t = 0; t < 8; ++t) qv[i][t] = qi[t] * scale;
    }
    float m[GR], l[GR], acc[GR][8];
#pragma unroll
    for (int i = 0; i < GR; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t) acc[i][t] = 0.f;
    }
    const size_t head_base = (size_t(b) * G + g) * ctx_max;
    for (int j = j_lo + slot; j < j_hi; j += SLOTS) {
        const uint4 kw = *reinterpret_cast<const uint4 *>(k_cache + (head_base + j) * HD + dim0);
        const uint4 vw = *reinterpret_cast<const uint4 *>(v_cache + (head_base + j) * HD + dim0);
        float kf[8], vf[8];
        const uint32_t kk[4] = {kw.x, kw.y, kw.z, kw.w}, vv[4] = {vw.x, vw.y, vw.z, vw.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            kf[2 * t] = __uint_as_float(kk[t] << 16);
            kf[2 * t + 1] = __uint_as_float(kk[t] & 0xffff0000u);
            vf[2 * t] = __uint_as_float(vv[t] << 16);
            vf[2 * t + 1] = __uint_as_float(vv[t] & 0xffff0000u);
        }
#pragma unroll
        for (int i = 0; i < GR; ++i) {
            float sc = 0.f;
#pragma unroll
            for (int t = 0; t < 8; ++t) sc = fmaf(qv[i][t], kf[t], sc);
#pragma unroll
            for (int o = 1; o < LPP; o <<= 1) sc += __shfl_xor(sc, o, kWave);
            const float mn = fmaxf(m[i], sc);
            const float c = expf(m[i] - mn), p = expf(sc - mn);
            l[i] = l[i] * c + p;
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[i][t] = fmaf(p, vf[t], acc[i][t] * c);
            m[i] = mn;
        }
    }
    // merge the position slots of the wavefront (lanes with the same sub hold the same dims)
#pragma unroll
    for (int o = LPP; o < kWave; o <<= 1) {
#pragma unroll
        for (int i = 0; i < GR; ++i) {
            const float m2 = __shfl_xor(m[i], o, kWave), l2 = __shfl_xor(l[i], o, kWave);
            float a2[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) a2[t] = __shfl_xor(acc[i][t], o, kWave);
            merge_state(m[i], l[i], acc[i], m2, l2, a2);
        }
    }
    if (lane < LPP) {
#pragma unroll
        for (int i = 0; i < GR; ++i) {
            if (lane == 0) {
                red_m[wave][i] = m[i];
                red_l[wave][i] = l[i];
            }
#pragma unroll
            for (int t = 0; t < 8; ++t) red_acc[wave][i][dim0 + t] = acc[i][t];
        }
    }
    __syncthreads();
    // wavefronts in order; thread (head i, dim) writes the split's result
    for (int idx = threadIdx.x; idx < GR * HD; idx += kThreads) {
        const int i = idx / HD, dim = idx % HD;
        float mm = -INFINITY, ll = 0.f, aa = 0.f;
        for (int w = 0; w < kWaves; ++w) {
            const float m2 = red_m[w][i];
            const float mn = fmaxf(mm, m2);
            if (mn == -INFINITY) continue;
            const float c1 = expf(mm - mn), c2 = expf(m2 - mn);
            ll = ll * c1 + red_l[w][i] * c2;
            aa = aa * c1 + red_acc[w][i][dim] * c2;
            mm = mn;
        }
        float *out = part + ((size_t(b) * H + g * GR + i) * S + s) * (HD + 2);
        out[dim] = aa;
        if (dim == 0) {
            out[HD] = mm;
            out[HD + 1] = ll;
        }
    }
}

// attn_merge: grid (H, B).  The splits of one query head merged by the log-sum-exp
// rule: every thread loads its share of the splits' values at once (S * hd / 256 of
// them), then the partial sums meet in LDS.  a [B, H * hd] out.
__global__ __launch_bounds__(kThreads) void attn_merge(const float *__restrict__ part, int S,
                                                       int H, int hd, float *__restrict__ a) {
    __shared__ float w[kMaxSplits];
    __shared__ float red[kWaves];
    __shared__ float num[kThreads];
    const int head = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
    const int wave = t / kWave, lane = t % kWave;
    const float *p = part + (size_t(b) * H + head) * S * (hd + 2);
    // maximum over the splits
    float m = t < S ? p[size_t(t) * (hd + 2) + hd] : -INFINITY;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
    if (lane == 0) red[wave] = m;
    __syncthreads();
    const float M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    // split weights exp(m_s - M) and the normaliser
    float den = 0.f;
    if (t < S) {
        const float ms = p[size_t(t) * (hd + 2) + hd];
        const float ws = ms == -INFINITY ? 0.f : expf(ms - M);
        w[t] = ws;
        den = ws * p[size_t(t) * (hd + 2) + hd + 1];
    }
    den = wave_sum(den);
    if (lane == 0) red[wave] = den;
    __syncthreads();
    const float D = red[0] + red[1] + red[2] + red[3];
    // weighted sums: thread t takes dimension t % hd of splits t / hd, t / hd + 256 / hd, ...
    const int dim = t % hd, s0 = t / hd, step = kThreads / hd;
    float acc = 0.f;
#pragma unroll 8
    for (int s = s0; s < S; s += step) acc = fmaf(w[s], p[size_t(s) * (hd + 2) + dim], acc);
    num[t] = acc;
    __syncthreads();
    if (t < hd) {
        float sum = 0.f;
        for (int g = 0; g < step; ++g) sum += num[g * hd + t];
        a[(size_t(b) * H + head) * hd + t] = sum / D;
    }
}

// attn_out: grid (ceil(d / 4), B): o[b, r] = W_o[r] . a[b], one row per wavefront, a[b]
// staged in LDS.
__global__ __launch_bounds__(kThreads) void attn_out(const float *__restrict__ a,
                                                     const uint16_t *__restrict__ w_o, int d,
                                                     int H, int hd, float *__restrict__ o) {
    extern __shared__ float a_lds[];           // [H * hd]
    const int b = blockIdx.y;
    const int qrows = H * hd;
    for (int idx = threadIdx.x; idx < qrows / 4; idx += kThreads)
        reinterpret_cast<float4 *>(a_lds)[idx] =
            reinterpret_cast<const float4 *>(a + size_t(b) * qrows)[idx];
    __syncthreads();
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = qrows / 8;
    for (int r = blockIdx.x * kOutRows + wave; r < min(d, (blockIdx.x + 1) * kOutRows);
         r += kWaves) {
        const uint4 *row = reinterpret_cast<const uint4 *>(w_o + size_t(r) * qrows);
        float acc = 0.f;
        for (int c = lane; c < nch; c += kWave) {
            const float4 x0 = *reinterpret_cast<const float4 *>(&a_lds[8 * c]);
            const float4 x1 = *reinterpret_cast<const float4 *>(&a_lds[8 * c + 4]);
            acc = dot8(row[c], x0, x1, acc);
        }
        acc = wave_sum(acc);
        if (lane == 0) o[size_t(b) * d + r] = acc;
    }
}

// splits of the position range: enough workgroups for the chip, at least 16 positions each
int pick_splits(int n_pos, int B, int G) {
    const int want = (256 + B * G - 1) / (B * G);
    const int most = (n_pos + 15) / 16;
    return std::max(1, std::min(want, most));
}

}  // namespace

extern "C" size_t apex_attention_workspace_bytes(int B, int H, int G, int hd, int ctx_max) {
    if (B <= 0 || H <= 0 || G <= 0 || hd <= 0 || ctx_max <= 0) return 256;
    const size_t qb = apex::align_up(size_t(B) * H * hd * sizeof(float), 256);   // q, a
    const size_t pb = size_t(B) * H * kMaxSplits * (hd + 2) * sizeof(float);
    return 2 * qb + apex::align_up(pb, 256);
}

extern "C" apex_status apex_attention_decode(const float *h, const uint16_t *w_qkv,
                                             const uint16_t *w_o, int B, int d, int H, int G,
                                             int hd, uint16_t *k_cache, uint16_t *v_cache,
                                             int ctx_max, int pos, float *o, void *workspace,
                                             size_t workspace_bytes, hipStream_t stream) {
    const char *fn = "apex_attention_decode";
    APEX_REQUIRE(B >= 0, "%s: B=%d must be >= 0", fn, B);
    APEX_REQUIRE(d >= 8 && d % 8 == 0, "%s: d=%d must be a positive multiple of 8", fn, d);
    APEX_REQUIRE(hd == 64 || hd == 128, "%s: head size %d must be 64 or 128", fn, hd);
    APEX_REQUIRE(H >= 1 && G >= 1 && H % G == 0 && H / G <= kMaxGroup,
                 "%s: H=%d must be a multiple of G=%d with at most %d query heads per group",
                 fn, H, G, kMaxGroup);
    APEX_REQUIRE(H / G <= 4 || H / G == 8, "%s: %d query heads per group is not supported",
                 fn, H / G);
    APEX_REQUIRE(ctx_max >= 1 && pos >= 0 && pos < ctx_max, "%s: pos=%d out of [0, %d)", fn,
                 pos, ctx_max);
    if (B == 0) return APEX_OK;
    APEX_REQUIRE(h && w_qkv && w_o && k_cache && v_cache && o && workspace, "%s: NULL pointer",
                 fn);
    APEX_REQUIRE(apex::aligned16(h) && apex::aligned16(w_qkv) && apex::aligned16(w_o) &&
                     apex::aligned16(k_cache) && apex::aligned16(v_cache) &&
                     apex::aligned16(workspace),
                 "%s: inputs, caches and workspace must be 16-byte aligned", fn);
    const size_t need = apex_attention_workspace_bytes(B, H, G, hd, ctx_max);
    if (workspace_bytes < need)
        return apex::fail(APEX_E_CAPACITY, "%s: workspace %zu < %zu bytes", fn, workspace_bytes,
                          need);
    const int n_pos = pos + 1;
    const int S = std::min(pick_splits(n_pos, B, G), kMaxSplits);
    const size_t qb = apex::align_up(size_t(B) * H * hd * sizeof(float), 256);
    float *q = static_cast<float *>(workspace);
    float *a = reinterpret_cast<float *>(static_cast<char *>(workspace) + qb);
    float *part = reinterpret_cast<float *>(static_cast<char *>(workspace) + 2 * qb);

    const int R = (H + 2 * G) * hd;
    const int nch = d / 8;
    const dim3 gq((R + kWaves - 1) / kWaves, B);
    if (nch <= kWave)
        hipLaunchKernelGGL((attn_qkv<1>), gq, dim3(kThreads), 0, stream, h, w_qkv, d, H, G, hd,
                           k_cache, v_cache, ctx_max, pos, q);
    else if (nch <= 2 * kWave)
        hipLaunchKernelGGL((attn_qkv<2>), gq, dim3(kThreads), 0, stream, h, w_qkv, d, H, G, hd,
                           k_cache, v_cache, ctx_max, pos, q);
    else
        hipLaunchKernelGGL((attn_qkv<4>), gq, dim3(kThreads), 0, stream, h, w_qkv, d, H, G, hd,
                           k_cache, v_cache, ctx_max, pos, q);
    APEX_HIP(hipGetLastError());

    const dim3 gs(S, G, B);
    const float scale = 1.f / std::sqrt(float(hd));
    const int GR = H / G;
#define APEX_SPLIT(HD_, GR_)                                                                   \
    hipLaunchKernelGGL((attn_split<HD_, GR_>), gs, dim3(kThreads), 0, stream, q, k_cache,       \
                       v_cache, H, G, ctx_max, n_pos, scale, part)
#define APEX_SPLIT_HD(HD_)                                                                     \
    switch (GR) {                                                                              \
        case 1: APEX_SPLIT(HD_, 1); break;                                                     \
        case 2: APEX_SPLIT(HD_, 2); break;                                                     \
        case 3: APEX_SPLIT(HD_, 3); break;                                                     \
        case 4: APEX_SPLIT(HD_, 4); break;                                                     \
        default: APEX_SPLIT(HD_, 8); break;                                                    \
    }
    if (hd == 64) {
        APEX_SPLIT_HD(64)
    } else {
        APEX_SPLIT_HD(128)
    }
#undef APEX_SPLIT_HD
#undef APEX_SPLIT
    APEX_HIP(hipGetLastError());
    hipLaunchKernelGGL(attn_merge, dim3(H, B), dim3(kThreads), 0, stream, part, S, H, hd, a);
    APEX_HIP(hipGetLastError());
    const dim3 go((d + kOutRows - 1) / kOutRows, B);
    hipLaunchKernelGGL(attn_out, go, dim3(kThreads), size_t(H) * hd * sizeof(float), stream, a,
                       w_o, d, H, hd, o);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}
