// Expert FFN for one token over apex_pack_expert_fp8 slots (apex_moe_ffn_fp8, batch 1):
// the two launches of ffn_b1.hip with E4M3 weights and fp32 row scales.
#include <hip/hip_runtime.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::dot16_e4m3;
using apex::ffn::kWave;
using apex::ffn::ld_stream;
using apex::ffn::silu;
using apex::ffn::wave_sum;

// ---------------------------------------------------------------------------------
// E4M3 codes with fp32 row scales (apex_pack_expert_fp8 layout).
// A 16-byte load holds 16 weights; NPL counts 16-byte chunks per lane (1024 values of
// a row per pass of a wavefront).  up_b1_e4m3 multiplies each row's dot products by
// the row's scale; down_b1_e4m3 multiplies every (expert, chunk) partial by that
// expert's W2 row scale before it joins the row's sum.
template <int NPL, int RW, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_b1_e4m3(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const uint8_t *__restrict__ slots, int n_slots,
    size_t slot_bytes, float *__restrict__ h) {
    const int j = blockIdx.y;
    const int e = exec_idx[j];
    const float g = exec_gate[j];
    if (e < 0 || e >= E) return;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i0 = (blockIdx.x * WAVES + wave) * RW;
    if (i0 >= I) return;
    const int nch = d / 16;
    const uint8_t *slot = slots + size_t(s) * slot_bytes;
    const uint4 *W = reinterpret_cast<const uint4 *>(slot);                // rows of 2 * nch chunks
    const float *scale = reinterpret_cast<const float *>(slot + size_t(3) * I * d);
    const float4 *x4 = reinterpret_cast<const float4 *>(x);

    float u[RW], v[RW];
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
        float4 xs[NPL][4];
#pragma unroll
        for (int n = 0; n < NPL; ++n) {
            const int c = cb + lane + n * kWave;
            if (c < nch)
#pragma unroll
                for (int q = 0; q < 4; ++q) xs[n][q] = x4[4 * c + q];
        }
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
            for (int n = 0; n < NPL; ++n) {
                const int c = cb + lane + n * kWave;
                if (c < nch) {
                    u[r] = dot16_e4m3(w1[r][n], xs[n], u[r]);
                    v[r] = dot16_e4m3(w3[r][n], xs[n], v[r]);
                }
            }
    }
    float hv = 0.f;
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const int i = (i0 + r < I) ? i0 + r : I - 1;
        const float su = wave_sum(u[r]) * scale[i];
        const float sv = wave_sum(v[r]) * scale[I + i];
        if (lane == r) hv = silu(su) * sv * g;
    }
    if (lane < RW && i0 + lane < I) h[size_t(j) * I + i0 + lane] = hv;
}

// up_sk_e4m3: the same h with each row's length split over a workgroup, grid
// (I / R, k).  The WAVES * 64 lanes cover the d / 16 chunks of a row one chunk each: a
// lane loads its 64 bytes of x once, then the 2R chunks of the R W1/W3 row pairs, all
// before the multiplies.  The wavefronts' partial sums meet in LDS and are added in
// wavefront order before the row scales are applied.
template <int R, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_sk_e4m3(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const uint8_t *__restrict__ slots, int n_slots,
    size_t slot_bytes, float *__restrict__ h) {
    __shared__ float pu[WAVES][R], pv[WAVES][R];
    const int j = blockIdx.y;
    const int e = exec_idx[j];
    const float g = exec_gate[j];
    // uniform over the workgroup: the whole workgroup leaves before the barrier
    if (e < 0 || e >= E) return;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = d / 16;
    const int c = threadIdx.x;
    const bool on = c < nch;
    const int i0 = blockIdx.x * R;
    const uint8_t *slot = slots + size_t(s) * slot_bytes;
    const uint4 *W = reinterpret_cast<const uint4 *>(slot);
    const float *scale = reinterpret_cast<const float *>(slot + size_t(3) * I * d);
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    uint4 w1[R], w3[R];
    float4 xs[4];
    if (on) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint4 *row = W + size_t(i) * 2 * nch;
            w1[r] = ld_stream(row + c);
            w3[r] = ld_stream(row + nch + c);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) xs[q] = x4[4 * c + q];
    }
    float u[R], v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        u[r] = on ? dot16_e4m3(w1[r], xs, 0.f) : 0.f;
        v[r] = on ? dot16_e4m3(w3[r], xs, 0.f) : 0.f;
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
        const int i = i0 + threadIdx.x;
        float su = 0.f, sv = 0.f;
#pragma unroll
        for (int q = 0; q < WAVES; ++q) {
            su += pu[q][threadIdx.x];
            sv += pv[q][threadIdx.x];
        }
        h[size_t(j) * I + i] = silu(su * scale[i]) * (sv * scale[I + i]) * g;
    }
}

template <int RD, int WAVES, int UNR>
__global__ __launch_bounds__(WAVES *kWave) void down_b1_e4m3(
    int d, int I, int E, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, const uint8_t *__restrict__ slots, int n_slots,
    size_t slot_bytes, const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    // offsets into the slot pool (16-byte chunks for W2, floats for its row scales), not
    // pointers, so that the loads stay global loads and do not wait on LDS traffic
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ size_t meta_w2[APEX_MAX_EXPERTS];
    __shared__ size_t meta_s2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 16;
    const uint4 *pool = reinterpret_cast<const uint4 *>(slots);
    const float *pool_f = reinterpret_cast<const float *>(slots);
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            const size_t base = size_t(s) * slot_bytes;
            meta_pos[idx] = lane;
            meta_w2[idx] = (base + size_t(2) * I * d) / 16;
            meta_s2[idx] = (base + size_t(3) * I * d) / 4 + 2 * size_t(I);
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
    int item = 0, c = lane;
    while (c >= nch && item < n_valid) { c -= nch; ++item; }
    for (int t0 = lane; t0 < total; t0 += UNR * kWave) {
        uint4 w[UNR][RD];
        float sc[UNR][RD];
        float4 hx[UNR][4];
        bool on[UNR];
        int it = item, cc = c;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            on[u] = t0 + u * kWave < total;
            if (on[u]) {
                const uint4 *w2 = pool + meta_w2[it];
                const float *s2 = pool_f + meta_s2[it];
                const float4 *hr = reinterpret_cast<const float4 *>(h + size_t(meta_pos[it]) * I);
#pragma unroll
                for (int q = 0; q < 4; ++q) hx[u][q] = hr[4 * cc + q];
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const int jr = (j0 + r < d) ? j0 + r : d - 1;
                    w[u][r] = ld_stream(w2 + size_t(jr) * nch + cc);
                    sc[u][r] = s2[jr];
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
                for (int r = 0; r < RD; ++r)
                    acc[r] = fmaf(sc[u][r], dot16_e4m3(w[u][r], hx[u], 0.f), acc[r]);
    }
#pragma unroll
    for (int r = 0; r < RD; ++r) {
        const float s = wave_sum(acc[r]);
        if (lane == r && j0 + r < d) y[j0 + r] = (accumulate ? y[j0 + r] : 0.f) + s;
    }
}

}  // namespace

namespace apex {

apex_status ffn_b1_fp8(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                       const float *exec_gate, const int32_t *slot_of_expert,
                       const uint8_t *slots, int n_slots, float *h, float *y, int accumulate,
                       hipStream_t stream) {
    const size_t slot_bytes = apex_expert_bytes_fp8(d, I);
    // tile shapes measured on MI355X (timing probe, the calls of one workload cycling over
    // a 1.5 GB pool)
    using UpKernel = decltype(&up_b1_e4m3<1, 1, 4>);
    UpKernel up;
    dim3 gu, bu;
    if (d > 1024 && d <= 4096) {
        // a workgroup of 2 or 4 wavefronts per R row pairs, one 16-byte chunk of the row
        // per lane; R grows with the number of row pairs.  Up projection against one or
        // two row pairs per wavefront (up_b1_e4m3), us: Granite-3B 6.13 -> 5.58, OLMoE
        // 9.44 -> 8.48, Phi-7B 7.27 -> 5.87, Mixtral 51.3 -> 41.3 (R = 4; R = 8 43.0); at
        // d = 1024 up_b1_e4m3 is faster (4.76 against 5.02)
        const size_t pairs = size_t(I) * k;
        const int rows = pairs > 16384 ? 4 : pairs > 2048 ? 2 : 1;
        if (d <= 2048)
            up = rows == 4 ? up_sk_e4m3<4, 2> : rows == 2 ? up_sk_e4m3<2, 2> : up_sk_e4m3<1, 2>;
        else
            up = rows == 4 ? up_sk_e4m3<4, 4> : rows == 2 ? up_sk_e4m3<2, 4> : up_sk_e4m3<1, 4>;
        gu = dim3(I / rows + (I % rows != 0), k);
        bu = dim3((d <= 2048 ? 2 : 4) * kWave);
    } else if (d <= 1024) {
        up = up_b1_e4m3<1, 1, 4>;   // one row pair per wavefront, the whole row in one pass
        gu = dim3(I / 4 + (I % 4 != 0), k);
        bu = dim3(256);
    } else {
        up = up_b1_e4m3<4, 2, 4>;   // two row pairs per wavefront, 4096 values per pass
        gu = dim3(I / 8 + (I % 8 != 0), k);
        bu = dim3(256);
    }
    hipLaunchKernelGGL(up, gu, bu, 0, stream, x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                       slots, n_slots, slot_bytes, h);
    APEX_HIP(hipGetLastError());
    if (d <= 1024) {
        hipLaunchKernelGGL((down_b1_e4m3<1, 1, 4>), dim3(d), dim3(64), 0, stream, d, I, E, k,
                           exec_idx, slot_of_expert, slots, n_slots, slot_bytes, h, y, accumulate);
    } else if (d <= 2048) {
        // two output rows per wavefront (against one: OLMoE 7.33 -> 6.92 us, Granite-3B 4.67
        // -> 4.54)
        hipLaunchKernelGGL((down_b1_e4m3<2, 4, 4>), dim3(d / 8 + (d % 8 != 0)), dim3(256), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_bytes, h, y, accumulate);
    } else {
        hipLaunchKernelGGL((down_b1_e4m3<4, 4, 4>), dim3(d / 16 + (d % 16 != 0)), dim3(256), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_bytes, h, y, accumulate);
    }
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
