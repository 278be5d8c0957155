// Expert FFN for one token over apex_pack_expert_fp32 slots (apex_moe_ffn_fp32, batch 1):
// the two launches of ffn_b1.hip with 32-bit weights, four per 16-byte load.
//
// up_sk_f32 / up_b1_f32 write h[j, i] = silu(W1[i] . x) * (W3[i] . x) * gate_j for every
// executed expert; down_f32 owns output rows of y and sums W2_j[row] . h[j] over the
// executed experts as one flattened dot product.  Weight loads are non-temporal (a call
// reads each weight once).
#include <hip/hip_runtime.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::kWave;
using apex::ffn::ld_stream;
using apex::ffn::silu;
using apex::ffn::wave_sum;

__device__ __forceinline__ float dot4(uint4 w, float4 x, float acc) {
    acc = fmaf(__uint_as_float(w.x), x.x, acc);
    acc = fmaf(__uint_as_float(w.y), x.y, acc);
    acc = fmaf(__uint_as_float(w.z), x.z, acc);
    acc = fmaf(__uint_as_float(w.w), x.w, acc);
    return acc;
}

// up_sk_f32: grid (I / R, k).  The WAVES * 64 lanes cover the d / 4 chunks of a row one
// chunk each: a lane loads its 16 bytes of x once, then the 2R chunks of the R W1/W3 row
// pairs, all before the multiplies; the wavefronts' partial sums meet in LDS and are
// added in wavefront order.
template <int R, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_sk_f32(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const float *__restrict__ slots, int n_slots,
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
    const int nch = d / 4;
    const int c = threadIdx.x;
    const bool on = c < nch;
    const int i0 = blockIdx.x * R;
    const uint4 *W = reinterpret_cast<const uint4 *>(slots + size_t(s) * slot_elems);
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    uint4 w1[R], w3[R];
    float4 xs;
    if (on) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint4 *row = W + size_t(i) * 2 * nch;
            w1[r] = ld_stream(row + c);
            w3[r] = ld_stream(row + nch + c);
        }
        xs = x4[c];
    }
    float u[R], v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        u[r] = on ? dot4(w1[r], xs, 0.f) : 0.f;
        v[r] = on ? dot4(w3[r], xs, 0.f) : 0.f;
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
        float su = 0.f, sv = 0.f;
#pragma unroll
        for (int q = 0; q < WAVES; ++q) {
            su += pu[q][threadIdx.x];
            sv += pv[q][threadIdx.x];
        }
        h[size_t(j) * I + i0 + threadIdx.x] = silu(su) * sv * g;
    }
}

// up_b1_f32: rows longer than 4096 values.  Grid (I / WAVES, k); a wavefront owns one row
// pair and steps through it NPL chunks per lane at a time, every load of a step issued
// before its multiplies.
template <int NPL, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_b1_f32(
    const float *__restrict__ x, int d, int I, int E, int k,
    const int32_t *__restrict__ exec_idx, const float *__restrict__ exec_gate,
    const int32_t *__restrict__ slot_of_expert, const float *__restrict__ slots, int n_slots,
    size_t slot_elems, float *__restrict__ h) {
    const int j = blockIdx.y;
    const int e = exec_idx[j];
    const float g = exec_gate[j];
    if (e < 0 || e >= E) return;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int i = blockIdx.x * WAVES + wave;
    if (i >= I) return;
    const int nch = d / 4;
    const uint4 *row =
        reinterpret_cast<const uint4 *>(slots + size_t(s) * slot_elems) + size_t(i) * 2 * nch;
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    float u = 0.f, v = 0.f;
    for (int cb = 0; cb < nch; cb += NPL * kWave) {
        uint4 w1[NPL], w3[NPL];
        float4 xs[NPL];
#pragma unroll
        for (int n = 0; n < NPL; ++n) {
            const int c = cb + lane + n * kWave;
            if (c < nch) {
                w1[n] = ld_stream(row + c);
                w3[n] = ld_stream(row + nch + c);
                xs[n] = x4[c];
            }
        }
#pragma unroll
        for (int n = 0; n < NPL; ++n)
            if (cb + lane + n * kWave < nch) {
                u = dot4(w1[n], xs[n], u);
                v = dot4(w3[n], xs[n], v);
            }
    }
    const float su = wave_sum(u), sv = wave_sum(v);
    if (lane == 0) h[size_t(j) * I + i] = silu(su) * sv * g;
}

// down_f32: grid d / (WAVES * RD).  A wavefront owns RD output rows; the gated h of all
// valid positions is one vector of length (#valid) * I, so each row is one dot product
// over the concatenated W2 rows of the executed experts.  Lanes step through (position,
// chunk) pairs UNR at a time with all loads issued before the multiplies.
template <int RD, int WAVES, int UNR>
__global__ __launch_bounds__(WAVES *kWave) void down_f32(
    int d, int I, int E, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, const float *__restrict__ slots, int n_slots,
    size_t slot_elems, const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    // W2 of valid position idx starts at chunk meta_w2[idx] of the slot pool
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ size_t meta_w2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 4;
    const uint4 *pool = reinterpret_cast<const uint4 *>(slots);
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            meta_pos[idx] = lane;
            meta_w2[idx] = (size_t(s) * slot_elems + size_t(2) * I * d) / 4;
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
    while (c >= nch && item < n_valid) {
        c -= nch;
        ++item;
    }
    for (int t0 = lane; t0 < total; t0 += UNR * kWave) {
        uint4 w[UNR][RD];
        float4 hx[UNR];
        bool on[UNR];
        int it = item, cc = c;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            on[u] = t0 + u * kWave < total;
            if (on[u]) {
                const uint4 *w2 = pool + meta_w2[it];
                hx[u] = reinterpret_cast<const float4 *>(h + size_t(meta_pos[it]) * I)[cc];
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const int jr = (j0 + r < d) ? j0 + r : d - 1;
                    w[u][r] = ld_stream(w2 + size_t(jr) * nch + cc);
                }
            }
            cc += kWave;
            while (cc >= nch) {
                cc -= nch;
                ++it;
            }
        }
        item = it;
        c = cc;
#pragma unroll
        for (int u = 0; u < UNR; ++u)
            if (on[u])
#pragma unroll
                for (int r = 0; r < RD; ++r) acc[r] = dot4(w[u][r], hx[u], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < RD; ++r) {
        const float s = wave_sum(acc[r]);
        if (lane == r && j0 + r < d) y[j0 + r] = (accumulate ? y[j0 + r] : 0.f) + s;
    }
}

}  // namespace

namespace apex {

apex_status ffn_b1_fp32(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                        const float *exec_gate, const int32_t *slot_of_expert,
                        const float *slots, int n_slots, float *h, float *y, int accumulate,
                        hipStream_t stream) {
    const size_t slot_elems = size_t(3) * d * I;
    using UpKernel = decltype(&up_sk_f32<1, 1>);
    UpKernel up;
    dim3 gu, bu;
    if (d <= 4096) {
        // a row pair per workgroup (two where one would mean more than 16384
        // workgroups), the fewest wavefronts whose lanes cover the row one chunk each
        const bool two = size_t(I) * k > 16384;
        const int waves = d <= 256 ? 1 : d <= 512 ? 2 : d <= 1024 ? 4 : d <= 2048 ? 8 : 16;
        if (waves == 1) up = two ? up_sk_f32<2, 1> : up_sk_f32<1, 1>;
        else if (waves == 2) up = two ? up_sk_f32<2, 2> : up_sk_f32<1, 2>;
        else if (waves == 4) up = two ? up_sk_f32<2, 4> : up_sk_f32<1, 4>;
        else if (waves == 8) up = two ? up_sk_f32<2, 8> : up_sk_f32<1, 8>;
        else up = two ? up_sk_f32<2, 16> : up_sk_f32<1, 16>;
        gu = dim3(two ? I / 2 + (I % 2 != 0) : I, k);
        bu = dim3(waves * kWave);
    } else {
        up = up_b1_f32<4, 2>;
        gu = dim3(I / 2 + (I % 2 != 0), k);
        bu = dim3(2 * kWave);
    }
    hipLaunchKernelGGL(up, gu, bu, 0, stream, x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                       slots, n_slots, slot_elems, h);
    APEX_HIP(hipGetLastError());
    if (d <= 2048)
        hipLaunchKernelGGL((down_f32<1, 1, 8>), dim3(d), dim3(kWave), 0, stream, d, I, E, k,
                           exec_idx, slot_of_expert, slots, n_slots, slot_elems, h, y,
                           accumulate);
    else
        hipLaunchKernelGGL((down_f32<2, 4, 8>), dim3(d / 8 + (d % 8 != 0)), dim3(4 * kWave), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_elems, h, y, accumulate);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
