// Gated SwiGLU experts over HBM cache slots (apex_moe_ffn).
//
// Two launches per call, both HBM-bound streams of bf16 weights:
//   ffn_gate_up  grid (I tiles, active experts): each wavefront owns RW rows i of one
//                expert and computes h[p, i] = silu(W1[i] . x_b) * (W3[i] . x_b) for every
//                token b routed to that expert (pair p), reading each weight once;
//   ffn_down     grid (d tiles): each wavefront owns RD output rows j and accumulates
//                g_p * (W2_e[j] . h[p]) over the (expert, token) pairs in (expert, token)
//                order into LDS, then writes y once - no atomics, deterministic.
// Weights are read with 16-byte loads; lanes of a wavefront cover consecutive 16-byte
// chunks of a row, so every wavefront load is a contiguous 1 KB burst.
// Every workgroup derives the expert grouping of the batch itself (at most B*k <= 1024
// pairs, a few hundred LDS operations) instead of paying a separate launch.
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.h"

namespace {

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kWavesPerGroup = kThreads / kWave;
constexpr int kInvalidKey = 0x7fffffff;

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

// Pairs p = b*k + j of the batch whose expert has a slot in this pass, sorted by
// (expert, p), and the active experts in ascending id order with their ranges.
struct Groups {
    int n_items;
    int n_act;
    unsigned int mask[2];
    int act_e[APEX_MAX_EXPERTS];
    int act_start[APEX_MAX_EXPERTS + 1];
    int key[APEX_MAX_PAIRS];
    int item[APEX_MAX_PAIRS];
};

__device__ void build_groups(Groups &G, const int32_t *__restrict__ exec_idx,
                             const int32_t *__restrict__ slot_of_expert, int P, int E,
                             int n_slots) {
    const int tid = threadIdx.x;
    if (tid == 0) {
        G.n_items = 0;
        G.mask[0] = G.mask[1] = 0u;
    }
    __syncthreads();
    for (int p = tid; p < P; p += kThreads) {
        const int e = exec_idx[p];
        bool ok = e >= 0 && e < E;
        if (ok) {
            const int s = slot_of_expert[e];
            ok = s >= 0 && s < n_slots;
        }
        G.key[p] = ok ? ((e << 16) | p) : kInvalidKey;
        if (ok) {
            atomicAdd(&G.n_items, 1);
            atomicOr(&G.mask[e >> 5], 1u << (e & 31));
        }
    }
    __syncthreads();
    for (int p = tid; p < P; p += kThreads) {
        const int kp = G.key[p];
        if (kp == kInvalidKey) continue;
        int pos = 0;
        for (int q = 0; q < P; ++q) pos += G.key[q] < kp ? 1 : 0;
        G.item[pos] = p;
    }
    if (tid < APEX_MAX_EXPERTS) {
        const int e = tid;
        const unsigned long long m =
            (static_cast<unsigned long long>(G.mask[1]) << 32) | G.mask[0];
        if ((m >> e) & 1ull) {
            const int a = __popcll(m & ((1ull << e) - 1ull));
            int start = 0;
            for (int q = 0; q < P; ++q) start += G.key[q] < (e << 16) ? 1 : 0;
            G.act_e[a] = e;
            G.act_start[a] = start;
        }
        if (tid == 0) {
            G.n_act = __popcll(m);
            G.act_start[G.n_act] = G.n_items;
        }
    }
    __syncthreads();
}

template <int RW, int NT>
__global__ __launch_bounds__(kThreads) void ffn_gate_up(
    const float *__restrict__ x, int d, int I, int E, int k, int P,
    const int32_t *__restrict__ exec_idx, const int32_t *__restrict__ slot_of_expert,
    const uint16_t *__restrict__ slots, int n_slots, size_t slot_elems, float *__restrict__ h) {
    __shared__ Groups G;
    build_groups(G, exec_idx, slot_of_expert, P, E, n_slots);
    const int a = blockIdx.y;
    if (a >= G.n_act) return;
    const int e = G.act_e[a];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i0 = (blockIdx.x * kWavesPerGroup + wave) * RW;
    if (i0 >= I) return;
    const uint16_t *Wrows = slots + size_t(slot_of_expert[e]) * slot_elems;
    const int beg = G.act_start[a], end = G.act_start[a + 1];
    const int nch = d / 8;
    const size_t row_stride = size_t(2) * d;

    for (int t0 = beg; t0 < end; t0 += NT) {
        int pair[NT];
        const float4 *xr[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            pair[t] = (t0 + t < end) ? G.item[t0 + t] : -1;
            const int bb = pair[t] >= 0 ? pair[t] / k : 0;
            xr[t] = reinterpret_cast<const float4 *>(x + size_t(bb) * d);
        }
        float u[RW][NT], v[RW][NT];
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t) u[r][t] = v[r][t] = 0.f;

        for (int c = lane; c < nch; c += kWave) {
            uint4 w1[RW], w3[RW];
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const int i = (i0 + r < I) ? i0 + r : I - 1;
                const uint4 *row = reinterpret_cast<const uint4 *>(Wrows + size_t(i) * row_stride);
                w1[r] = row[c];
                w3[r] = row[nch + c];
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                if (pair[t] < 0) continue;
                const float4 xa = xr[t][2 * c], xb = xr[t][2 * c + 1];
#pragma unroll
                for (int r = 0; r < RW; ++r) {
                    u[r][t] = dot8(w1[r], xa, xb, u[r][t]);
                    v[r][t] = dot8(w3[r], xa, xb, v[r][t]);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const float su = wave_sum(u[r][t]);
                const float sv = wave_sum(v[r][t]);
                if (lane == 0 && pair[t] >= 0 && i0 + r < I)
                    h[size_t(pair[t]) * I + i0 + r] = silu(su) * sv;
            }
    }
}

template <int RD, int UI>
__global__ __launch_bounds__(kThreads) void ffn_down(
    int B, int d, int I, int E, int k, int P, const int32_t *__restrict__ exec_idx,
    const float *__restrict__ exec_gate, const int32_t *__restrict__ slot_of_expert,
    const uint16_t *__restrict__ slots, int n_slots, size_t slot_elems,
    const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    __shared__ Groups G;
    extern __shared__ float yacc[];   // [B][kWavesPerGroup * RD]
    constexpr int kRows = kWavesPerGroup * RD;
    build_groups(G, exec_idx, slot_of_expert, P, E, n_slots);
    for (int i = threadIdx.x; i < B * kRows; i += kThreads) yacc[i] = 0.f;
    __syncthreads();

    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int j0 = blockIdx.x * kRows + wave * RD;
    const int nch = I / 8;
    const size_t w2_off = size_t(2) * I * d;
    if (j0 < d) {
        for (int it0 = 0; it0 < G.n_items; it0 += UI) {
            int pair[UI];
            const uint4 *wrow[UI];
            const float4 *hr[UI];
#pragma unroll
            for (int u = 0; u < UI; ++u) {
                pair[u] = (it0 + u < G.n_items) ? G.item[it0 + u] : -1;
                const int p = pair[u] >= 0 ? pair[u] : G.item[it0];
                const int e = exec_idx[p];
                wrow[u] = reinterpret_cast<const uint4 *>(
                    slots + size_t(slot_of_expert[e]) * slot_elems + w2_off);
                hr[u] = reinterpret_cast<const float4 *>(h + size_t(p) * I);
            }
            float acc[UI][RD];
#pragma unroll
            for (int u = 0; u < UI; ++u)
#pragma unroll
                for (int r = 0; r < RD; ++r) acc[u][r] = 0.f;
            for (int c = lane; c < nch; c += kWave) {
#pragma unroll
                for (int u = 0; u < UI; ++u) {
                    if (pair[u] < 0) continue;
                    const float4 ha = hr[u][2 * c], hb = hr[u][2 * c + 1];
#pragma unroll
                    for (int r = 0; r < RD; ++r) {
                        const int j = (j0 + r < d) ? j0 + r : d - 1;
                        acc[u][r] = dot8(wrow[u][size_t(j) * nch + c], ha, hb, acc[u][r]);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < UI; ++u)
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const float s = wave_sum(acc[u][r]);
                    if (lane == 0 && pair[u] >= 0 && j0 + r < d) {
                        const int bb = pair[u] / k;
                        yacc[bb * kRows + wave * RD + r] += exec_gate[pair[u]] * s;
                    }
                }
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < B * kRows; i += kThreads) {
        const int bb = i / kRows, rr = i % kRows;
        const int j = blockIdx.x * kRows + rr;
        if (j < d) {
            float *dst = y + size_t(bb) * d + j;
            *dst = (accumulate ? *dst : 0.f) + yacc[i];
        }
    }
}

// ---------------------------------------------------------------------------------
// Batch-1 path.  One token, so no grouping: position j of exec_idx is expert j's pair.
//
// up_b1: grid (I / (WAVES * RW), k).  A wavefront owns RW rows of the expert at
// position blockIdx.y and issues every 16-byte load of those rows (W1 and W3, NPL
// chunks per lane) before the first multiply, so each lane keeps 2 * RW * NPL loads in
// flight.  Writes h[j, i] = silu(W1[i] . x) * (W3[i] . x) * gate_j: the gate is folded
// in here so the down projection is one long dot product per output row.
template <int NPL, int RW, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_b1(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const uint16_t *__restrict__ slots, int n_slots,
    size_t slot_elems, float *__restrict__ h) {
    const int j = blockIdx.y;
    const int e = exec_idx[j];
    const float g = exec_gate[j];
    if (e < 0 || e >= E) return;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i0 = (blockIdx.x * WAVES + wave) * RW;
    if (i0 >= I) return;
    const int nch = d / 8;
    const uint4 *W = reinterpret_cast<const uint4 *>(slots + size_t(s) * slot_elems);
    const float4 *x4 = reinterpret_cast<const float4 *>(x);

    float u[RW], v[RW];   // lane partial sums over every block of the row
#pragma unroll
    for (int r = 0; r < RW; ++r) u[r] = v[r] = 0.f;
    for (int cb = 0; cb < nch; cb += NPL * kWave) {
        uint4 w1[RW][NPL], w3[RW][NPL];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint4 *row = W + size_t(i) * 2 * nch;
#pragma unroll
            for (int n = 0; n < NPL; ++n) {
                const int c = cb + lane + n * kWave;
                if (c < nch) {
                    w1[r][n] = row[c];
                    w3[r][n] = row[nch + c];
                }
            }
        }
        float4 xa[NPL], xb[NPL];
#pragma unroll
        for (int n = 0; n < NPL; ++n) {
            const int c = cb + lane + n * kWave;
            if (c < nch) {
                xa[n] = x4[2 * c];
                xb[n] = x4[2 * c + 1];
            }
        }
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
            for (int n = 0; n < NPL; ++n) {
                const int c = cb + lane + n * kWave;
                if (c < nch) {
                    u[r] = dot8(w1[r][n], xa[n], xb[n], u[r]);
                    v[r] = dot8(w3[r][n], xa[n], xb[n], v[r]);
                }
            }
    }
    float hv = 0.f;
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const float su = wave_sum(u[r]);
        const float sv = wave_sum(v[r]);
        if (lane == r) hv = silu(su) * sv * g;
    }
    if (lane < RW && i0 + lane < I) h[size_t(j) * I + i0 + lane] = hv;
}

// down_b1: grid d / (WAVES * RD).  A wavefront owns RD output rows; the gated h of
// all valid positions is one vector of length (#valid) * I, so each row is a single dot
// product over the concatenated W2 rows of the executed experts.  Lanes step through
// (position, chunk) pairs UNR at a time with all loads issued before the multiplies.
template <int RD, int WAVES, int UNR>
__global__ __launch_bounds__(WAVES *kWave) void down_b1(
    int d, int I, int E, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, const uint16_t *__restrict__ slots, int n_slots,
    size_t slot_elems, const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ const uint4 *meta_w2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 8;
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            meta_pos[idx] = lane;
            meta_w2[idx] = reinterpret_cast<const uint4 *>(slots + size_t(s) * slot_elems +
                                                           size_t(2) * I * d);
        }
        if (lane == 0) n_valid = __popcll(m);
    }
    __syncthreads();
    const int j0 = (blockIdx.x * WAVES + wave) * RD;
    if (j0 >= d) return;
    const int total = n_valid * nch;
    float acc[RD];
#pragma unroll
    for (int r = 0; r < RD; ++r) acc[r] = 0.f;
    // lane's first (position, chunk): t = lane
    int item = 0, c = lane;
    while (c >= nch && item < n_valid) { c -= nch; ++item; }
    for (int t0 = lane; t0 < total; t0 += UNR * kWave) {
        uint4 w[UNR][RD];
        float4 ha[UNR], hb[UNR];
        bool on[UNR];
        int it = item, cc = c;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            on[u] = t0 + u * kWave < total;
            if (on[u]) {
                const uint4 *w2 = meta_w2[it];
                const float4 *hr = reinterpret_cast<const float4 *>(h + size_t(meta_pos[it]) * I);
                ha[u] = hr[2 * cc];
                hb[u] = hr[2 * cc + 1];
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const int jr = (j0 + r < d) ? j0 + r : d - 1;
                    w[u][r] = w2[size_t(jr) * nch + cc];
                }
            }
            cc += kWave;
            while (cc >= nch) { cc -= nch; ++it; }
        }
        item = it;
        c = cc;
#pragma unroll
        for (int u = 0; u < UNR; ++u)
            if (on[u])
#pragma unroll
                for (int r = 0; r < RD; ++r) acc[r] = dot8(w[u][r], ha[u], hb[u], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < RD; ++r) {
        const float s = wave_sum(acc[r]);
        if (lane == r && j0 + r < d) y[j0 + r] = (accumulate ? y[j0 + r] : 0.f) + s;
    }
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

extern "C" size_t apex_moe_ffn_workspace_bytes(int B, int k, int I) {
    if (B <= 0 || k <= 0 || I <= 0) return 256;
    return align_up(size_t(B) * k * I * sizeof(float), 256);
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
    const size_t need = apex_moe_ffn_workspace_bytes(B, k, I);
    if (workspace_bytes < need)
        return apex::fail(APEX_E_CAPACITY, "%s: workspace %zu < %zu bytes", fn, workspace_bytes,
                          need);
    // y rows are read back when accumulating
    const int P = B * k;
    const size_t slot_elems = size_t(3) * d * I;
    float *h = static_cast<float *>(workspace);
    const int max_act = P < E ? P : E;

    if (B == 1) {
        // h holds gated rows per position; tile shapes measured on MI355X (streaming rate
        // of the two launches against the plain read rate at the same sizes)
        const int npl = (d + 511) / 512;
        if (d <= 2048) {
            const dim3 gu(I / 4 + (I % 4 != 0), k);
            if (npl <= 1)
                hipLaunchKernelGGL((up_b1<1, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                                   exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h);
            else if (npl == 2)
                hipLaunchKernelGGL((up_b1<2, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                                   exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h);
            else if (npl == 3)
                hipLaunchKernelGGL((up_b1<3, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                                   exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h);
            else
                hipLaunchKernelGGL((up_b1<4, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                                   exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h);
            APEX_HIP(hipGetLastError());
            hipLaunchKernelGGL((down_b1<1, 1, 8>), dim3(d), dim3(64), 0, stream, d, I, E, k,
                               exec_idx, slot_of_expert, slots, n_slots, slot_elems, h, y,
                               accumulate);
        } else {
            const dim3 gu(I / 8 + (I % 8 != 0), k);
            hipLaunchKernelGGL((up_b1<4, 2, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                               exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h);
            APEX_HIP(hipGetLastError());
            hipLaunchKernelGGL((down_b1<4, 4, 8>), dim3(d / 16 + (d % 16 != 0)), dim3(256), 0,
                               stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                               slot_elems, h, y, accumulate);
        }
        APEX_HIP(hipGetLastError());
        return APEX_OK;
    }

    constexpr int RW = 4;
    const dim3 g1((I + kWavesPerGroup * RW - 1) / (kWavesPerGroup * RW), max_act);
    if (B == 1)
        hipLaunchKernelGGL((ffn_gate_up<RW, 1>), g1, dim3(kThreads), 0, stream, x, d, I, E, k, P,
                           exec_idx, slot_of_expert, slots, n_slots, slot_elems, h);
    else
        hipLaunchKernelGGL((ffn_gate_up<RW, 4>), g1, dim3(kThreads), 0, stream, x, d, I, E, k, P,
                           exec_idx, slot_of_expert, slots, n_slots, slot_elems, h);
    APEX_HIP(hipGetLastError());

    constexpr int RD = 1, UI = 8;
    const int rows = kWavesPerGroup * RD;
    const dim3 g2((d + rows - 1) / rows);
    const size_t smem = size_t(B) * rows * sizeof(float);
    hipLaunchKernelGGL((ffn_down<RD, UI>), g2, dim3(kThreads), smem, stream, B, d, I, E, k, P,
                       exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_elems, h, y,
                       accumulate);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}
