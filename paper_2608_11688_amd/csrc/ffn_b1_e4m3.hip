// Expert FFN for one token over apex_pack_expert_fp8 slots (apex_moe_ffn_fp8, batch 1):
// the two launches of ffn_b1.hip with E4M3 weights and fp32 row scales.
#include <hip/hip_runtime.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::dot16_e4m3;
using apex::ffn::kWave;
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
                    w1[r][n] = row[c];
                    w3[r][n] = row[nch + c];
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
                    w[u][r] = w2[size_t(jr) * nch + cc];
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
    const int npl = (d + 1023) / 1024;   // 16-byte chunks per lane for a whole row
    if (d <= 2048) {
        const dim3 gu(I / 4 + (I % 4 != 0), k);
        if (npl <= 1)
            hipLaunchKernelGGL((up_b1_e4m3<1, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                               exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_bytes, h);
        else
            hipLaunchKernelGGL((up_b1_e4m3<2, 1, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                               exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_bytes, h);
        APEX_HIP(hipGetLastError());
        hipLaunchKernelGGL((down_b1_e4m3<1, 1, 4>), dim3(d), dim3(64), 0, stream, d, I, E, k,
                           exec_idx, slot_of_expert, slots, n_slots, slot_bytes, h, y, accumulate);
    } else {
        const dim3 gu(I / 8 + (I % 8 != 0), k);
        hipLaunchKernelGGL((up_b1_e4m3<4, 2, 4>), gu, dim3(256), 0, stream, x, d, I, E, k,
                           exec_idx, exec_gate, slot_of_expert, slots, n_slots, slot_bytes, h);
        APEX_HIP(hipGetLastError());
        hipLaunchKernelGGL((down_b1_e4m3<4, 4, 4>), dim3(d / 16 + (d % 16 != 0)), dim3(256), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_bytes, h, y, accumulate);
    }
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
