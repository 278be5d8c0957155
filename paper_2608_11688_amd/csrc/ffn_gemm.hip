// Expert FFN for two or more tokens (apex_moe_ffn, batch >= 2): a grouped GEMM on the
// matrix cores.
//
// group_pairs converts x to bf16 and builds one table of the (token, position) pairs
// sorted by expert; up_gemm and down_gemm stage 64-row weight tiles and 16*MT token rows
// through LDS and issue v_mfma_f32_16x16x32_bf16 on them; combine_pairs sums the gated
// per-pair outputs of every token in pair order.  Every executed expert's weights are
// read once per call whatever the number of tokens routed to it, and no atomics are
// used, so results are deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::kWave;
using apex::ffn::silu;

// ---------------------------------------------------------------------------------
// Batched path (B >= 2): grouped GEMMs on the matrix cores.
//
// group_pairs (one workgroup) writes the (expert, token) grouping once per call; the
// GEMM kernels take tokens as the M dimension (tiles of 16, padded), weight rows as N
// and the hidden / intermediate dimension as K, with v_mfma_f32_16x16x32_bf16
// (activations rounded to bf16, fp32 accumulation).  Every expert's weights are read
// once per call whatever the number of tokens routed to it.  Per-pair outputs go to
// the workspace and a combine kernel applies the gates in a fixed order.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

struct GroupTable {          // lives at the start of the workspace
    int n_act;
    int n_items;
    int act_e[APEX_MAX_EXPERTS];
    int act_start[APEX_MAX_EXPERTS + 1];
    int item[APEX_MAX_PAIRS];   // pair indices sorted by (expert, pair)
};

constexpr int kGroupThreads = 1024;

// Every workgroup rounds a slice of the activations to bf16 (xb [B, d], 8 values per
// thread per step) for the matrix cores; workgroup 0 also builds the grouping.
__global__ __launch_bounds__(kGroupThreads) void group_pairs(
    const int32_t *__restrict__ exec_idx, const int32_t *__restrict__ slot_of_expert, int P, int E,
    int n_slots, GroupTable *__restrict__ G, const float *__restrict__ x, int B, int d,
    __bf16 *__restrict__ xb) {
    const size_t n8 = size_t(B) * d / 8;
    for (size_t i = size_t(blockIdx.x) * kGroupThreads + threadIdx.x; i < n8;
         i += size_t(gridDim.x) * kGroupThreads) {
        const float4 p = reinterpret_cast<const float4 *>(x)[2 * i];
        const float4 q = reinterpret_cast<const float4 *>(x)[2 * i + 1];
        bf16x8 v;
        v[0] = (__bf16)p.x; v[1] = (__bf16)p.y; v[2] = (__bf16)p.z; v[3] = (__bf16)p.w;
        v[4] = (__bf16)q.x; v[5] = (__bf16)q.y; v[6] = (__bf16)q.z; v[7] = (__bf16)q.w;
        reinterpret_cast<bf16x8 *>(xb)[i] = v;
    }
    if (blockIdx.x != 0) return;
    constexpr int kW = kGroupThreads / kWave;
    __shared__ int cnt[kW][APEX_MAX_EXPERTS];
    __shared__ int wave_off[kW][APEX_MAX_EXPERTS];
    __shared__ int start[APEX_MAX_EXPERTS + 1];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    for (int base = 0; base < P; base += kGroupThreads) {
        // pairs [base, base + 1024) this round; P <= 1024 so there is one round
        const int p = base + threadIdx.x;
        int e = -1;
        if (p < P) {
            const int x = exec_idx[p];
            if (x >= 0 && x < E) {
                const int s = slot_of_expert[x];
                if (s >= 0 && s < n_slots) e = x;
            }
        }
        int local = 0;
        for (int ex = 0; ex < E; ++ex) {
            const unsigned long long m = __ballot(e == ex);
            if (e == ex) local = __popcll(m & ((1ull << lane) - 1ull));
            if (lane == 0) cnt[wave][ex] = __popcll(m);
        }
        __syncthreads();
        if (threadIdx.x < E) {
            int run = 0;
            for (int w = 0; w < kW; ++w) {
                wave_off[w][threadIdx.x] = run;
                run += cnt[w][threadIdx.x];
            }
            cnt[0][threadIdx.x] = run;   // total per expert (cnt[0] already consumed)
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int run = 0, n_act = 0;
            for (int ex = 0; ex < E; ++ex) {
                start[ex] = run;
                if (cnt[0][ex] > 0) {
                    G->act_e[n_act] = ex;
                    G->act_start[n_act] = run;
                    ++n_act;
                }
                run += cnt[0][ex];
            }
            start[E] = run;
            G->act_start[n_act] = run;
            G->n_act = n_act;
            G->n_items = run;
        }
        __syncthreads();
        if (e >= 0) G->item[start[e] + wave_off[wave][e] + local] = p;
    }
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Grouped-GEMM mainloop shared by the gate/up and down projections.
// A workgroup (4 wavefronts) owns a tile of 64 weight rows of NW weight matrices and up
// to 16*MT tokens.  K advances in blocks of 128: every thread loads 16-byte pieces so
// that each group of 16 threads reads 256 contiguous bytes of one weight row (whole
// cache lines), the block goes to LDS, and while the matrix cores work on it the next
// block is already loading into registers.  Wavefront w multiplies its 16 rows with
// every token tile: v_mfma_f32_16x16x32_bf16, tokens as M, weight rows as N.
constexpr int kKB = 128;
constexpr int kLdsRow = kKB + 8;   // +16 B per row: the 16 rows of a fragment read hit distinct banks

// One K block of the tile into registers.  Every address is valid (rows and K are
// clamped); pieces outside the tile are zeroed after the load instead of branching,
// so all 4*NW + MT loads issue back to back.
// Component-wise select: a select of the whole vector struct is lowered through
// private memory by the compiler.
__device__ __forceinline__ uint4 keep_if(uint4 v, bool c) {
    return make_uint4(c ? v.x : 0u, c ? v.y : 0u, c ? v.z : 0u, c ? v.w : 0u);
}

template <int NW, int MT>
__device__ __forceinline__ void gemm_load(uint4 (&wreg)[NW][4], uint4 (&xreg)[MT],
                                          const uint16_t *const (&wbase)[NW], size_t wstride,
                                          int rows_valid, int K, const uint16_t *const (&xrow)[MT],
                                          const bool (&xok)[MT], int k0, int r0, int seg) {
    const int kk = k0 + 8 * seg;
    const bool in = kk < K;
    const int kc = in ? kk : K - 8;
#pragma unroll
    for (int m = 0; m < NW; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int row = r0 + 16 * j;
            const int rc = row < rows_valid ? row : rows_valid - 1;
            const uint4 v = *reinterpret_cast<const uint4 *>(wbase[m] + size_t(rc) * wstride + kc);
            wreg[m][j] = keep_if(v, in && row < rows_valid);
        }
#pragma unroll
    for (int j = 0; j < MT; ++j) {
        const uint4 v = *reinterpret_cast<const uint4 *>(xrow[j] + kc);
        xreg[j] = keep_if(v, in && xok[j]);
    }
}

template <int NW, int MT>
__device__ __forceinline__ void gemm_mainloop(const uint16_t *const (&wbase)[NW], size_t wstride,
                                              int rows_valid, int K,
                                              const uint16_t *const (&xrow)[MT],
                                              const bool (&xok)[MT], int n_tiles,
                                              uint16_t (*Ws)[64][kLdsRow],
                                              uint16_t (*Xs)[kLdsRow], floatx4 (&acc)[NW][MT]) {
    const int t = threadIdx.x, wave = t / kWave, lane = t % kWave;
    const int seg = t & 15, r0 = t >> 4;
    uint4 wreg[NW][4], xreg[MT];
#pragma unroll
    for (int m = 0; m < NW; ++m)
#pragma unroll
        for (int tt = 0; tt < MT; ++tt) acc[m][tt] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int nb = (K + kKB - 1) / kKB;
    // Workgroups start at different K blocks: tiles that run side by side then read
    // different offsets of their rows instead of all hitting the same DRAM channels.
    const int rot = int((blockIdx.x * 7u + blockIdx.y * 13u) % unsigned(nb));
    const auto kblk = [nb, rot](int b) { const int q = b + rot; return (q >= nb ? q - nb : q) * kKB; };
    gemm_load<NW, MT>(wreg, xreg, wbase, wstride, rows_valid, K, xrow, xok, kblk(0), r0, seg);
    for (int b = 0; b < nb; ++b) {
        __syncthreads();   // the previous block's fragments have been read
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                *reinterpret_cast<uint4 *>(&Ws[m][r0 + 16 * j][8 * seg]) = wreg[m][j];
#pragma unroll
        for (int j = 0; j < MT; ++j) *reinterpret_cast<uint4 *>(&Xs[r0 + 16 * j][8 * seg]) = xreg[j];
        __syncthreads();
        if (b + 1 < nb)
            gemm_load<NW, MT>(wreg, xreg, wbase, wstride, rows_valid, K, xrow, xok,
                              kblk(b + 1), r0, seg);
#pragma unroll
        for (int q = 0; q < kKB / 32; ++q) {
            const int kc = 32 * q + 8 * (lane >> 4);
            uint4 wop[NW];
#pragma unroll
            for (int m = 0; m < NW; ++m)
                wop[m] = *reinterpret_cast<const uint4 *>(&Ws[m][16 * wave + (lane & 15)][kc]);
#pragma unroll
            for (int tt = 0; tt < MT; ++tt) {
                if (tt >= n_tiles) continue;
                const uint4 xop = *reinterpret_cast<const uint4 *>(&Xs[16 * tt + (lane & 15)][kc]);
#pragma unroll
                for (int m = 0; m < NW; ++m)
                    acc[m][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        as_bf16x8(xop), as_bf16x8(wop[m]), acc[m][tt], 0, 0, 0);
            }
        }
    }
}

// up_gemm: grid (ceil(I / 64), max active experts): 64 rows of W1 and W3 of one expert,
// every token of the expert (16*MT per pass).
// hb[pair, i] = bf16(silu(W1[i] . x_b) * (W3[i] . x_b)), ungated.
template <int MT>
__global__ __launch_bounds__(256) void up_gemm(
    const __bf16 *__restrict__ xb, int d, int I, int k, const GroupTable *__restrict__ G,
    const int32_t *__restrict__ slot_of_expert, const uint16_t *__restrict__ slots,
    size_t slot_elems, __bf16 *__restrict__ hb) {
    __shared__ uint16_t Ws[2][64][kLdsRow];
    __shared__ uint16_t Xs[16 * MT][kLdsRow];
    const int a = blockIdx.y;
    if (a >= G->n_act) return;
    const int i0 = blockIdx.x * 64;
    if (i0 >= I) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int e = G->act_e[a];
    const int beg = G->act_start[a], n_e = G->act_start[a + 1] - beg;
    const uint16_t *W = slots + size_t(slot_of_expert[e]) * slot_elems + size_t(i0) * 2 * d;
    const uint16_t *const wbase[2] = {W, W + d};
    const uint16_t *xs = reinterpret_cast<const uint16_t *>(xb);
    for (int t0 = 0; t0 < n_e; t0 += 16 * MT) {
        const uint16_t *xrow[MT];
        bool xok[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int tok = t0 + (threadIdx.x >> 4) + 16 * j;
            xok[j] = tok < n_e;
            xrow[j] = xs + size_t(G->item[beg + (xok[j] ? tok : 0)] / k) * d;
        }
        const int n_tiles = min(MT, (n_e - t0 + 15) / 16);
        floatx4 acc[2][MT];
        gemm_mainloop<2, MT>(wbase, size_t(2) * d, I - i0, d, xrow, xok, n_tiles, Ws, Xs, acc);
        const int i = i0 + 16 * wave + (lane & 15);
#pragma unroll
        for (int tt = 0; tt < MT; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tok = t0 + 16 * tt + 4 * (lane >> 4) + r;
                if (tt < n_tiles && tok < n_e && i < I)
                    hb[size_t(G->item[beg + tok]) * I + i] =
                        (__bf16)(silu(acc[0][tt][r]) * acc[1][tt][r]);
            }
    }
}

// down_gemm: grid (ceil(d / 64), max active experts): 64 rows j of W2 of one expert.
// ypair[pair, j] = W2[j] . h[pair] for every token of the expert.
template <int MT>
__global__ __launch_bounds__(256) void down_gemm(
    int d, int I, const GroupTable *__restrict__ G, const int32_t *__restrict__ slot_of_expert,
    const uint16_t *__restrict__ slots, size_t slot_elems, const __bf16 *__restrict__ hb,
    float *__restrict__ ypair) {
    __shared__ uint16_t Ws[1][64][kLdsRow];
    __shared__ uint16_t Xs[16 * MT][kLdsRow];
    const int a = blockIdx.y;
    if (a >= G->n_act) return;
    const int j0 = blockIdx.x * 64;
    if (j0 >= d) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int e = G->act_e[a];
    const int beg = G->act_start[a], n_e = G->act_start[a + 1] - beg;
    const uint16_t *const wbase[1] = {slots + size_t(slot_of_expert[e]) * slot_elems +
                                      size_t(2) * I * d + size_t(j0) * I};
    const uint16_t *hs = reinterpret_cast<const uint16_t *>(hb);
    for (int t0 = 0; t0 < n_e; t0 += 16 * MT) {
        const uint16_t *hrow[MT];
        bool hok[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int tok = t0 + (threadIdx.x >> 4) + 16 * j;
            hok[j] = tok < n_e;
            hrow[j] = hs + size_t(G->item[beg + (hok[j] ? tok : 0)]) * I;
        }
        const int n_tiles = min(MT, (n_e - t0 + 15) / 16);
        floatx4 acc[1][MT];
        gemm_mainloop<1, MT>(wbase, size_t(I), d - j0, I, hrow, hok, n_tiles, Ws, Xs, acc);
        const int j = j0 + 16 * wave + (lane & 15);
#pragma unroll
        for (int tt = 0; tt < MT; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tok = t0 + 16 * tt + 4 * (lane >> 4) + r;
                if (tt < n_tiles && tok < n_e && j < d)
                    ypair[size_t(G->item[beg + tok]) * d + j] = acc[0][tt][r];
            }
        __syncthreads();   // LDS is reused by the next pass
    }
}

// combine: y[b, j] (+)= sum over positions p of token b, in position order, of
// gate[p] * ypair[p, j] for the pairs this pass executed.
__global__ __launch_bounds__(256) void combine_pairs(
    int B, int d, int E, int k, const int32_t *__restrict__ exec_idx,
    const float *__restrict__ exec_gate, const int32_t *__restrict__ slot_of_expert, int n_slots,
    const float *__restrict__ ypair, float *__restrict__ y, int accumulate) {
    const int b = blockIdx.y;
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (b >= B || j >= d) return;
    float s = 0.f;
    for (int q = 0; q < k; ++q) {
        const int p = b * k + q;
        const int e = exec_idx[p];
        if (e < 0 || e >= E) continue;
        const int sl = slot_of_expert[e];
        if (sl < 0 || sl >= n_slots) continue;
        s += exec_gate[p] * ypair[size_t(p) * d + j];
    }
    float *dst = y + size_t(b) * d + j;
    *dst = (accumulate ? *dst : 0.f) + s;
}

}  // namespace

namespace apex {

// [GroupTable][h: B*k x I bf16][per-pair outputs: B*k x d fp32][x: B x d bf16]
size_t ffn_grouped_workspace(int B, int d, int I, int k) {
    const size_t P = size_t(B) * k;
    return align_up(sizeof(GroupTable), 256) + align_up(P * I * 2, 256) +
           align_up(P * d * sizeof(float), 256) + align_up(size_t(B) * d * 2, 256);
}

apex_status ffn_grouped(const float *x, int B, int d, int I, int E, int k,
                        const int32_t *exec_idx, const float *exec_gate,
                        const int32_t *slot_of_expert, const uint16_t *slots, int n_slots,
                        float *y, int accumulate, void *workspace, hipStream_t stream) {
    const int P = B * k;
    const size_t slot_elems = size_t(3) * d * I;
    const int max_act = P < E ? P : E;
    char *wsb = static_cast<char *>(workspace);
    GroupTable *G = reinterpret_cast<GroupTable *>(wsb);
    __bf16 *hb = reinterpret_cast<__bf16 *>(wsb + align_up(sizeof(GroupTable), 256));
    char *after_h = reinterpret_cast<char *>(hb) + align_up(size_t(P) * I * 2, 256);
    float *ypair = reinterpret_cast<float *>(after_h);
    __bf16 *xb = reinterpret_cast<__bf16 *>(after_h + align_up(size_t(P) * d * sizeof(float), 256));
    const size_t n8 = size_t(B) * d / 8;
    const unsigned conv_blocks = unsigned(std::min<size_t>(64, (n8 + kGroupThreads - 1) / kGroupThreads));
    hipLaunchKernelGGL(group_pairs, dim3(conv_blocks), dim3(kGroupThreads), 0, stream,
                       exec_idx, slot_of_expert, P, E, n_slots, G, x, B, d, xb);
    APEX_HIP(hipGetLastError());
    const dim3 gu((I + 63) / 64, max_act), gd((d + 63) / 64, max_act);
    // token tiles per pass: enough for the whole batch on one expert up to 64 tokens
    if (B >= 48) {
        hipLaunchKernelGGL((up_gemm<4>), gu, dim3(256), 0, stream, xb, d, I, k, G,
                           slot_of_expert, slots, slot_elems, hb);
        APEX_HIP(hipGetLastError());
        hipLaunchKernelGGL((down_gemm<4>), gd, dim3(256), 0, stream, d, I, G,
                           slot_of_expert, slots, slot_elems, hb, ypair);
    } else if (B >= 24) {
        hipLaunchKernelGGL((up_gemm<2>), gu, dim3(256), 0, stream, xb, d, I, k, G,
                           slot_of_expert, slots, slot_elems, hb);
        APEX_HIP(hipGetLastError());
        hipLaunchKernelGGL((down_gemm<2>), gd, dim3(256), 0, stream, d, I, G,
                           slot_of_expert, slots, slot_elems, hb, ypair);
    } else {
        hipLaunchKernelGGL((up_gemm<1>), gu, dim3(256), 0, stream, xb, d, I, k, G,
                           slot_of_expert, slots, slot_elems, hb);
        APEX_HIP(hipGetLastError());
        hipLaunchKernelGGL((down_gemm<1>), gd, dim3(256), 0, stream, d, I, G,
                           slot_of_expert, slots, slot_elems, hb, ypair);
    }
    APEX_HIP(hipGetLastError());
    hipLaunchKernelGGL(combine_pairs, dim3((d + 255) / 256, B), dim3(256), 0, stream, B, d, E,
                       k, exec_idx, exec_gate, slot_of_expert, n_slots, ypair, y, accumulate);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
