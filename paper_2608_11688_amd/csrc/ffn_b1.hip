// Expert FFN for one token (apex_moe_ffn, batch 1): gated SwiGLU experts over HBM
// cache slots, two launches that each stream their weights once.
//
// up_b1 / up_sk read the W1/W3 rows of every executed expert with all loads of a row
// issued before any arithmetic and write h[j, i] = silu(W1[i] . x) * (W3[i] . x) * gate_j;
// down_b1 owns output rows of y and sums W2_j[row] . h[j] over the k experts as one
// flattened dot product, so the k experts share a single launch and y is written once
// without atomics.  Loads are 16 bytes wide over consecutive chunks of a row.
#include <hip/hip_runtime.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::dot8;
using apex::ffn::kWave;
using apex::ffn::ld_stream;
using apex::ffn::silu;
using apex::ffn::wave_sum;

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
                    w1[r][n] = ld_stream(row + c);
                    w3[r][n] = ld_stream(row + nch + c);
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

// up_sk: the same h with each row's length split over a workgroup.  Grid
// (I / R, k); the WAVES * 64 lanes cover the d / 8 chunks of a row one chunk each, so a
// lane loads its 32 bytes of x once and then only weights: the 2R chunks of the R W1/W3
// row pairs, all issued before the multiplies.  Each wavefront reduces its partial sums,
// and the WAVES partials of a row are added in LDS in wavefront order (deterministic).
template <int R, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_sk(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const uint16_t *__restrict__ slots, int n_slots,
    size_t slot_elems, float *__restrict__ h) {
    __shared__ float pu[WAVES][R], pv[WAVES][R];
    const int j = blockIdx.y;
    const int e = exec_idx[j];
    const float g = exec_gate[j];
    // uniform over the workgroup: the whole workgroup leaves before the barrier
    if (e < 0 || e >= E) return;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = d / 8;
    const int c = threadIdx.x;
    const bool on = c < nch;
    const int i0 = blockIdx.x * R;
    const uint4 *W = reinterpret_cast<const uint4 *>(slots + size_t(s) * slot_elems);
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    uint4 w1[R], w3[R];
    float4 xa, xb;
    if (on) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint4 *row = W + size_t(i) * 2 * nch;
            w1[r] = ld_stream(row + c);
            w3[r] = ld_stream(row + nch + c);
        }
        xa = x4[2 * c];
        xb = x4[2 * c + 1];
    }
    float u[R], v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        u[r] = on ? dot8(w1[r], xa, xb, 0.f) : 0.f;
        v[r] = on ? dot8(w3[r], xa, xb, 0.f) : 0.f;
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float su = wave_sum(u[r]);
        const float sv = wave_sum(v[r]);
        if (lane == 0) {
            pu[wave][r] = su;
            pv[wave][r] = sv;
        }
    }
    __syncthreads();
    if (threadIdx.x < R && i0 + int(threadIdx.x) < I) {
        const int r = threadIdx.x;
        float su = 0.f, sv = 0.f;
#pragma unroll
        for (int q = 0; q < WAVES; ++q) {
            su += pu[q][r];
            sv += pv[q][r];
        }
        h[size_t(j) * I + i0 + r] = silu(su) * sv * g;
    }
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
    // W2 of valid position idx starts at chunk meta_w2[idx] of the slot pool (offsets, not
    // pointers, so that the loads stay global loads and do not wait on LDS traffic)
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ size_t meta_w2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 8;
    const uint4 *pool = reinterpret_cast<const uint4 *>(slots);
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            meta_pos[idx] = lane;
            meta_w2[idx] = (size_t(s) * slot_elems + size_t(2) * I * d) / 8;
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
                const uint4 *w2 = pool + meta_w2[it];
                const float4 *hr = reinterpret_cast<const float4 *>(h + size_t(meta_pos[it]) * I);
                ha[u] = hr[2 * cc];
                hb[u] = hr[2 * cc + 1];
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const int jr = (j0 + r < d) ? j0 + r : d - 1;
                    w[u][r] = ld_stream(w2 + size_t(jr) * nch + cc);
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

}  // namespace

namespace apex {

size_t ffn_b1_workspace(int d, int I, int k) {
    (void)d;
    return align_up(size_t(k) * I * sizeof(float), 256);
}

apex_status ffn_b1(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                   const float *exec_gate, const int32_t *slot_of_expert, const uint16_t *slots,
                   int n_slots, float *h, float *y, int accumulate, hipStream_t stream) {
    const size_t slot_elems = size_t(3) * d * I;
    // h holds gated rows per position; tile shapes measured on MI355X (streaming rate
    // of the two launches against the plain read rate at the same sizes)
    using UpKernel = decltype(&up_b1<1, 1, 4>);
    UpKernel up;
    dim3 gu, bu;
    if (d > 512 && d <= 4096) {
        // a row pair per workgroup of 2, 4 or 8 wavefronts (one 16-byte chunk of the row
        // per lane), or two row pairs where one would mean more than 16384 workgroups.
        // Up projection against one row pair per wavefront (up_b1), us: Granite-1B 5.45 ->
        // 5.36, Granite-3B 6.79 -> 6.58, OLMoE 13.5 -> 12.5, DeepSeek-16B 14.3 -> 13.3,
        // Phi-7B 8.0 -> 7.1, Mixtral 76.7 -> 74.0 (two row pairs); at d = 256 up_b1 is
        // faster (2.6 against 2.8)
        const bool two = size_t(I) * k > 16384;
        const int waves = d <= 1024 ? 2 : d <= 2048 ? 4 : 8;
        if (waves == 2) up = two ? up_sk<2, 2> : up_sk<1, 2>;
        else if (waves == 4) up = two ? up_sk<2, 4> : up_sk<1, 4>;
        else up = two ? up_sk<2, 8> : up_sk<1, 8>;
        gu = dim3(two ? I / 2 + (I % 2 != 0) : I, k);
        bu = dim3(waves * kWave);
    } else {
        // one row pair per wavefront: four wavefronts per workgroup for rows of up to 512
        // values (one chunk per lane), two for rows longer than 4096 (four chunks per lane)
        const bool shortrow = d <= 512;
        up = shortrow ? up_b1<1, 1, 4> : up_b1<4, 1, 2>;
        gu = shortrow ? dim3(I / 4 + (I % 4 != 0), k) : dim3(I / 2 + (I % 2 != 0), k);
        bu = dim3(shortrow ? 256 : 128);
    }
    hipLaunchKernelGGL(up, gu, bu, 0, stream, x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                       slots, n_slots, slot_elems, h);
    APEX_HIP(hipGetLastError());
    if (d <= 2048) {
        hipLaunchKernelGGL((down_b1<1, 1, 8>), dim3(d), dim3(64), 0, stream, d, I, E, k,
                           exec_idx, slot_of_expert, slots, n_slots, slot_elems, h, y,
                           accumulate);
    } else if (size_t(k) * I >= 8192) {
        // more than 2048 output rows, each a dot product of at least 8192 values: four
        // rows per wavefront (h loaded once for the four), two wavefronts per workgroup,
        // four chunks of every row in flight per lane.  Down projection alone at the
        // Mixtral shape (k I = 28672), against down_b1<2,4,8>: 40.6-40.8 -> 38.1 us, the
        // call 109.1-110.4 -> 106.4-107.3 us; two or four wavefronts per workgroup, or
        // four rows with 2, 3 or 6 chunks in flight, 38.6-40.3 us; six or eight rows
        // 42.3-55.2 us.
        hipLaunchKernelGGL((down_b1<4, 2, 4>), dim3(d / 8 + (d % 8 != 0)), dim3(128), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_elems, h, y, accumulate);
    } else {
        // more than 2048 output rows over short dot products: two rows per wavefront
        // (at the Phi-7B shape, k I = 1664, four rows per wavefront take 5.6 us against
        // 5.0 us)
        hipLaunchKernelGGL((down_b1<2, 4, 8>), dim3(d / 8 + (d % 8 != 0)), dim3(256), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_elems, h, y, accumulate);
    }
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
