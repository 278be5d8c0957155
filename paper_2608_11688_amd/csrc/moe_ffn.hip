// Gated SwiGLU experts over HBM cache slots (apex_moe_ffn).
//
// Both paths stream each executed expert's bf16 weights from HBM once per call and
// need no atomics, so results are deterministic:
//
// Batch 1 (up_b1, down_b1): one token, k experts. up_b1 reads W1/W3 rows of an expert
//   with all row loads issued before any arithmetic and writes h[j, i]; down_b1 owns one
//   output row of y and sums g_j * (W2_j[row] . h[j]) over the k experts in one
//   flattened dot, so the k experts share a single launch.
// Batch >= 2 (group_pairs, up_gemm, down_gemm, combine_pairs): a grouped GEMM on the
//   matrix cores. group_pairs converts x to bf16 and builds one table of the pairs
//   sorted by expert; up_gemm and down_gemm stage 64-row weight tiles and 16*MT token
//   rows through LDS and issue v_mfma_f32_16x16x32_bf16 on them; combine_pairs sums
//   the gated per-pair outputs of every token in pair order.
// Weights are read with 16-byte loads that cover consecutive 16-byte chunks of a row.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "common.h"

namespace {

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

constexpr int kMfmaMinBatch = 2;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

// workspace: [GroupTable][h: B*k x I fp32 (bf16 on the batched path)]
//            then, for B >= 2: [per-pair outputs: B*k x d fp32][bf16 activations: B x d]
extern "C" size_t apex_moe_ffn_workspace_bytes(int B, int d, int I, int k) {
    if (B <= 0 || k <= 0 || I <= 0 || d <= 0) return 256;
    const size_t P = size_t(B) * k;
    size_t n = align_up(sizeof(GroupTable), 256) + align_up(P * I * sizeof(float), 256);
    if (B >= kMfmaMinBatch)
        n += align_up(P * d * sizeof(float), 256) + align_up(size_t(B) * d * 2, 256);
    return n;
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
    // y rows are read back when accumulating
    const int P = B * k;
    const size_t slot_elems = size_t(3) * d * I;
    char *wsb = static_cast<char *>(workspace);
    GroupTable *G = reinterpret_cast<GroupTable *>(wsb);
    float *h = reinterpret_cast<float *>(wsb + align_up(sizeof(GroupTable), 256));
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

    // B >= 2: grouped GEMM on the matrix cores
    char *after_h = wsb + align_up(sizeof(GroupTable), 256) +
                    align_up(size_t(P) * I * sizeof(float), 256);
    float *ypair = reinterpret_cast<float *>(after_h);
    __bf16 *xb = reinterpret_cast<__bf16 *>(after_h + align_up(size_t(P) * d * sizeof(float), 256));
    __bf16 *hb = reinterpret_cast<__bf16 *>(h);
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


