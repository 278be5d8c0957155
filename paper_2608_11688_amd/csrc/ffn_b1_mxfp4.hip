// Expert FFN for one token over apex_pack_expert_mxfp4 slots (apex_moe_ffn_mxfp4, batch
// 1): the two launches of ffn_b1.hip with 4-bit E2M1 weights and a power-of-two scale
// per block of 32 values.  A lane's unit is 16 codes (8 bytes, half a block) and the
// scale byte of its block; codes are widened and scaled exactly by the hardware
// conversion, and the products accumulate in fp32.
#include <hip/hip_runtime.h>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::dot16_mxfp4;
using apex::ffn::kWave;
using apex::ffn::ld_stream;
using apex::ffn::mx_scale;
using apex::ffn::silu;
using apex::ffn::wave_sum;

// up_b1_mxfp4: grid (I / (WAVES * RW), k).  A wavefront owns RW rows of the expert at
// position blockIdx.y; NPL counts 16-code units per lane (1024 values of a row per pass
// of a wavefront).  All loads of a pass are issued before the first multiply.
template <int NPL, int RW, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_b1_mxfp4(
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
    const int nch = d / 16;                       // units per row of W1 (and of W3)
    const int nsb = d / 32;                       // scale bytes per row
    const uint8_t *slot = slots + size_t(s) * slot_bytes;
    const uint2 *W = reinterpret_cast<const uint2 *>(slot);     // rows of 2 * nch units
    const uint8_t *sc1 = slot + size_t(3) * I * d / 2;          // W1 scales [I][d/32]
    const uint8_t *sc3 = sc1 + size_t(I) * nsb;                 // W3 scales
    const float4 *x4 = reinterpret_cast<const float4 *>(x);

    float u[RW], v[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) u[r] = v[r] = 0.f;
    for (int cb = 0; cb < nch; cb += NPL * kWave) {
        uint2 w1[RW][NPL], w3[RW][NPL];
        uint32_t b1[RW][NPL], b3[RW][NPL];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint2 *row = W + size_t(i) * 2 * nch;
#pragma unroll
            for (int n = 0; n < NPL; ++n) {
                const int c = cb + lane + n * kWave;
                if (c < nch) {
                    w1[r][n] = ld_stream(row + c);
                    w3[r][n] = ld_stream(row + nch + c);
                    b1[r][n] = sc1[size_t(i) * nsb + c / 2];
                    b3[r][n] = sc3[size_t(i) * nsb + c / 2];
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
                    u[r] = dot16_mxfp4(w1[r][n], mx_scale(b1[r][n]), xs[n], u[r]);
                    v[r] = dot16_mxfp4(w3[r][n], mx_scale(b3[r][n]), xs[n], v[r]);
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

// up_sk_mxfp4: the same h with each row's length split over a workgroup, grid
// (I / R, k).  The WAVES * 64 lanes cover the d / 16 units of a row one unit each: a
// lane loads its 64 bytes of x once, then for each of the R W1/W3 row pairs two 8-byte
// units and their two scale bytes, all before the multiplies.  The wavefronts' partial
// sums meet in LDS and are added in wavefront order.
template <int R, int WAVES>
__global__ __launch_bounds__(WAVES *kWave) void up_sk_mxfp4(
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
    const int nch = d / 16;                       // units per row of W1 (and of W3)
    const int nsb = d / 32;                       // scale bytes per row
    const int c = threadIdx.x;
    const bool on = c < nch;
    const int i0 = blockIdx.x * R;
    const uint8_t *slot = slots + size_t(s) * slot_bytes;
    const uint2 *W = reinterpret_cast<const uint2 *>(slot);     // rows of 2 * nch units
    const uint8_t *sc1 = slot + size_t(3) * I * d / 2;          // W1 scales [I][d/32]
    const uint8_t *sc3 = sc1 + size_t(I) * nsb;                 // W3 scales
    const float4 *x4 = reinterpret_cast<const float4 *>(x);
    uint2 w1[R], w3[R];
    uint32_t b1[R], b3[R];
    float4 xs[4];
    if (on) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int i = (i0 + r < I) ? i0 + r : I - 1;
            const uint2 *row = W + size_t(i) * 2 * nch;
            w1[r] = ld_stream(row + c);
            w3[r] = ld_stream(row + nch + c);
            b1[r] = sc1[size_t(i) * nsb + c / 2];
            b3[r] = sc3[size_t(i) * nsb + c / 2];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) xs[q] = x4[4 * c + q];
    }
    float u[R], v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        u[r] = on ? dot16_mxfp4(w1[r], mx_scale(b1[r]), xs, 0.f) : 0.f;
        v[r] = on ? dot16_mxfp4(w3[r], mx_scale(b3[r]), xs, 0.f) : 0.f;
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

// down_b1_mxfp4: grid d / (WAVES * RD).  A wavefront owns RD output rows; lanes step
// through (valid position, unit) pairs UNR at a time, as down_b1 does.
template <int RD, int WAVES, int UNR>
__global__ __launch_bounds__(WAVES *kWave) void down_b1_mxfp4(
    int d, int I, int E, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, const uint8_t *__restrict__ slots, int n_slots,
    size_t slot_bytes, const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    // offsets into the slot pool (8-byte units of W2 codes, bytes of its scales)
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ size_t meta_w2[APEX_MAX_EXPERTS];
    __shared__ size_t meta_s2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 16, nsb = I / 32;
    const uint2 *pool = reinterpret_cast<const uint2 *>(slots);
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            const size_t base = size_t(s) * slot_bytes;
            meta_pos[idx] = lane;
            meta_w2[idx] = (base + size_t(I) * d) / 8;
            meta_s2[idx] = base + size_t(3) * I * d / 2 + size_t(2) * I * (d / 32);
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
        uint2 w[UNR][RD];
        uint32_t sb[UNR][RD];
        float4 hx[UNR][4];
        bool on[UNR];
        int it = item, cc = c;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            on[u] = t0 + u * kWave < total;
            if (on[u]) {
                const uint2 *w2 = pool + meta_w2[it];
                const uint8_t *s2 = slots + meta_s2[it];
                const float4 *hr = reinterpret_cast<const float4 *>(h + size_t(meta_pos[it]) * I);
#pragma unroll
                for (int q = 0; q < 4; ++q) hx[u][q] = hr[4 * cc + q];
#pragma unroll
                for (int r = 0; r < RD; ++r) {
                    const int jr = (j0 + r < d) ? j0 + r : d - 1;
                    w[u][r] = ld_stream(w2 + size_t(jr) * nch + cc);
                    sb[u][r] = s2[size_t(jr) * nsb + cc / 2];
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
                    acc[r] = dot16_mxfp4(w[u][r], mx_scale(sb[u][r]), hx[u], acc[r]);
    }
#pragma unroll
    for (int r = 0; r < RD; ++r) {
        const float s = wave_sum(acc[r]);
        if (lane == r && j0 + r < d) y[j0 + r] = (accumulate ? y[j0 + r] : 0.f) + s;
    }
}

// down_rows_mxfp4: the down projection for long flattened rows (more than 1024 units of
// 16 codes over the executed experts, Mixtral: 1792).  The WAVES * 64 lanes hold CPL
// units of the gated h of every valid position in registers, loaded once, so that every
// later load is codes and their scale bytes; the workgroup then streams RW output rows,
// G rows per step, one partial sum per row and lane.  Each row's wavefront partials
// meet in LDS and are added in wavefront order.  Grid d / RW; n_valid * I / 16 must not
// exceed WAVES * 64 * CPL (the dispatch checks k * I / 16).
template <int RW, int G, int WAVES, int CPL>
__global__ __launch_bounds__(WAVES *kWave) void down_rows_mxfp4(
    int d, int I, int E, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, const uint8_t *__restrict__ slots, int n_slots,
    size_t slot_bytes, const float *__restrict__ h, float *__restrict__ y, int accumulate) {
    __shared__ int meta_pos[APEX_MAX_EXPERTS];
    __shared__ size_t meta_w2[APEX_MAX_EXPERTS];
    __shared__ size_t meta_s2[APEX_MAX_EXPERTS];
    __shared__ int n_valid;
    __shared__ float part[WAVES][RW];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = I / 16, nsb = I / 32;
    const uint2 *pool = reinterpret_cast<const uint2 *>(slots);
    if (wave == 0) {
        const int e = lane < k ? exec_idx[lane] : -1;
        const int s = (e >= 0 && e < E) ? slot_of_expert[e] : -1;
        const bool ok = s >= 0 && s < n_slots;
        const unsigned long long m = __ballot(ok);
        if (ok) {
            const int idx = __popcll(m & ((1ull << lane) - 1ull));
            const size_t base = size_t(s) * slot_bytes;
            meta_pos[idx] = lane;
            meta_w2[idx] = (base + size_t(I) * d) / 8;
            meta_s2[idx] = base + size_t(3) * I * d / 2 + size_t(2) * I * (d / 32);
        }
        if (lane == 0) n_valid = __popcll(m);
    }
    __syncthreads();
    const int total = n_valid * nch;
    const int row0 = blockIdx.x * RW;
    // this lane's units: flattened index t -> (valid position, unit of its W2 row)
    size_t woff[CPL], soff[CPL];
    int hoff[CPL];
    bool on[CPL];
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
        const int t = threadIdx.x + u * WAVES * kWave;
        on[u] = t < total;
        const int it = on[u] ? t / nch : 0, cc = on[u] ? t - it * nch : 0;
        woff[u] = meta_w2[it] + cc;
        soff[u] = meta_s2[it] + cc / 2;
        hoff[u] = meta_pos[it] * I + 16 * cc;
    }
    float acc[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r] = 0.f;
    float4 hx[CPL][4];
#pragma unroll
    for (int rb = 0; rb < RW; rb += G) {
        uint2 w[G][CPL];
        uint32_t sb[G][CPL];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int jr = (row0 + rb + g < d) ? row0 + rb + g : d - 1;
#pragma unroll
            for (int u = 0; u < CPL; ++u)
                if (on[u]) {
                    w[g][u] = ld_stream(pool + woff[u] + size_t(jr) * nch);
                    sb[g][u] = slots[soff[u] + size_t(jr) * nsb];
                }
        }
        if (rb == 0) {   // h after the first rows' loads are in flight
#pragma unroll
            for (int u = 0; u < CPL; ++u)
                if (on[u])
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        hx[u][q] = reinterpret_cast<const float4 *>(h + hoff[u])[q];
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int u = 0; u < CPL; ++u)
                if (on[u])
                    acc[rb + g] = dot16_mxfp4(w[g][u], mx_scale(sb[g][u]), hx[u], acc[rb + g]);
    }
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        const float sr = wave_sum(acc[r]);
        if (lane == 0) part[wave][r] = sr;
    }
    __syncthreads();
    if (threadIdx.x < RW && row0 + int(threadIdx.x) < d) {
        float sr = 0.f;
#pragma unroll
        for (int q = 0; q < WAVES; ++q) sr += part[q][threadIdx.x];
        const int row = row0 + threadIdx.x;
        y[row] = (accumulate ? y[row] : 0.f) + sr;
    }
}

}  // namespace

namespace apex {

apex_status ffn_b1_mxfp4(const float *x, int d, int I, int E, int k, const int32_t *exec_idx,
                         const float *exec_gate, const int32_t *slot_of_expert,
                         const uint8_t *slots, int n_slots, float *h, float *y, int accumulate,
                         hipStream_t stream) {
    const size_t slot_bytes = apex_expert_bytes_mxfp4(d, I);
    // tile shapes measured on MI355X (timing probe, the calls of one workload cycling over
    // a 1.5 GB pool)
    using UpKernel = decltype(&up_b1_mxfp4<1, 1, 4>);
    UpKernel up;
    dim3 gu, bu;
    if (d > 1024 && d <= 4096) {
        // a workgroup of 2 or 4 wavefronts per two (more than 16384 row pairs: four) row
        // pairs, one 16-code unit of the row per lane.  Up projection against one row pair
        // per wavefront (up_b1_mxfp4), us: Granite-3B 5.90 -> 5.10, OLMoE 9.49 -> 7.16,
        // Phi-7B 6.14 -> 5.04, Mixtral 44.1 -> 28.9; whole 32-code blocks per lane were
        // slower (Mixtral 29.5-59.1); at d = 1024 the two are level (4.33, 4.28)
        const bool four = size_t(I) * k > 16384;
        if (d <= 2048) up = four ? up_sk_mxfp4<4, 2> : up_sk_mxfp4<2, 2>;
        else up = four ? up_sk_mxfp4<4, 4> : up_sk_mxfp4<2, 4>;
        gu = four ? dim3(I / 4 + (I % 4 != 0), k) : dim3(I / 2 + (I % 2 != 0), k);
        bu = dim3((d <= 2048 ? 2 : 4) * kWave);
    } else {
        // one row pair per wavefront; the whole row in one pass up to 1024 values, 4096
        // values per pass beyond (2 rows per wavefront took 178 VGPRs, 2 wavefronts per
        // SIMD, and left the conversions and the loads little to overlap with)
        const bool shortrow = d <= 1024;
        up = shortrow ? up_b1_mxfp4<1, 1, 4> : up_b1_mxfp4<4, 1, 4>;
        gu = dim3(I / 4 + (I % 4 != 0), k);
        bu = dim3(256);
    }
    hipLaunchKernelGGL(up, gu, bu, 0, stream, x, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                       slots, n_slots, slot_bytes, h);
    APEX_HIP(hipGetLastError());
    if (d <= 2048) {
        // two output rows per wavefront (against one: OLMoE 7.60 -> 6.34 us, Granite-3B
        // 4.84 -> 4.36, Granite-1B 4.38 -> 4.09)
        hipLaunchKernelGGL((down_b1_mxfp4<2, 1, 8>), dim3(d / 2 + (d % 2 != 0)), dim3(64), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_bytes, h, y, accumulate);
    } else if (size_t(k) * (I / 16) > 1024 && size_t(k) * (I / 16) <= 2048) {
        // long flattened rows: h held in registers, 16 output rows streamed per workgroup
        // of 16 wavefronts, four at a time (Mixtral call 50.7 -> 47.3 us against four rows
        // per wavefront; at Phi-7B, 104 units, it lost: 5.5 against 4.5 us for the down
        // projection).  Four rows per step against two, Mixtral, down alone 18.5 -> 17.8
        // us, the call 45.6-47.9 -> 44.6 us; eight 18.4-18.5 us; eight rows per workgroup
        // 24.5-25.4 us; eight wavefronts of four units per lane 18.7-20.2 us
        hipLaunchKernelGGL((down_rows_mxfp4<16, 4, 16, 2>), dim3(d / 16 + (d % 16 != 0)),
                           dim3(1024), 0, stream, d, I, E, k, exec_idx, slot_of_expert, slots,
                           n_slots, slot_bytes, h, y, accumulate);
    } else {
        hipLaunchKernelGGL((down_b1_mxfp4<4, 4, 4>), dim3(d / 16 + (d % 16 != 0)), dim3(256), 0,
                           stream, d, I, E, k, exec_idx, slot_of_expert, slots, n_slots,
                           slot_bytes, h, y, accumulate);
    }
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex
