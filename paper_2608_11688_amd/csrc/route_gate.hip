// Prefetch router (apex_prefetch_route) and original-router top-k (apex_gate_topk).
//
// One workgroup of 16 wavefronts per token.  Every wavefront streams whole rows of the
// bf16 router matrix with 16-byte loads (up to 4 experts at a time, sharing each read of
// the hidden state, all loads of a row issued together up to d = 2048) and reduces its
// dot products with cross-lane shuffles.  Softmax,
// ranking and the selection rules then run in wavefront 0 with one lane per expert
// (E <= 64), exchanging values through registers (readlane, shuffles, ballots).
// Optionally each token's workgroup then writes `seq` into done[token], after its
// outputs and a system-scope fence, so that a host polling pinned memory learns that the
// outputs are there before the kernel's completion signal reaches it.
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.h"
#include "route_internal.h"

namespace {

constexpr int kWave = 64;
constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxD = 65536;

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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// z[e] = W[e, :] . h (+ bias[e]) for all experts, into LDS.  All threads call it.
// Wavefront w takes experts w, w + 16, ... (EPP of them).  A pass covers NC 16-byte
// chunks per lane (64 * NC * 8 elements of d), and every load of a pass, weights and
// hidden state, is issued before the first multiply, so d <= 512 * NC costs one memory
// round trip.  The hidden state is read straight from global memory (every wavefront
// reads the same chunks, so after the first they hit the vector cache).
template <int NC, int EPP>
__device__ void token_logits(const float *__restrict__ h, const uint16_t *__restrict__ W,
                             const float *__restrict__ bias, int d, int E, float *z_lds) {
    const float4 *h4 = reinterpret_cast<const float4 *>(h);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int nch = d / 8;
    for (int e0 = wave; e0 < E; e0 += kWaves * EPP) {
        float acc[EPP];
        const uint4 *rows[EPP];
#pragma unroll
        for (int u = 0; u < EPP; ++u) {
            acc[u] = 0.f;
            const int e = e0 + u * kWaves;
            rows[u] = reinterpret_cast<const uint4 *>(W + size_t(e < E ? e : 0) * d);
        }
        for (int c0 = 0; c0 < nch; c0 += kWave * NC) {
            uint4 w[EPP][NC];
            float4 a[NC], b[NC];
#pragma unroll
            for (int n = 0; n < NC; ++n) {
                const int c = min(c0 + lane + n * kWave, nch - 1);
                a[n] = h4[2 * c];
                b[n] = h4[2 * c + 1];
#pragma unroll
                for (int u = 0; u < EPP; ++u) w[u][n] = rows[u][c];   // rows past E repeat row 0
            }
#pragma unroll
            for (int n = 0; n < NC; ++n)
                if (c0 + lane + n * kWave < nch)
#pragma unroll
                    for (int u = 0; u < EPP; ++u)
                        if (e0 + u * kWaves < E) acc[u] = dot8(w[u][n], a[n], b[n], acc[u]);
        }
#pragma unroll
        for (int u = 0; u < EPP; ++u) {
            const int e = e0 + u * kWaves;
            const float s = wave_sum(acc[u]);
            if (lane == 0 && e < E) z_lds[e] = s + (bias ? bias[e] : 0.f);
        }
    }
    __syncthreads();
}

// Position of expert `lane` when experts are ordered by descending logit, lower id
// first on equal logits, counting only experts whose bit is set in `mask` (no bit at or
// beyond E).  The logits are read from LDS four at a time, every lane at the same address
// (a broadcast): against other lanes' logits read with readlane (register to scalar, one
// at a time) the router took 6.20 -> 5.51 us at the Granite-1B shape and 11.34 -> 10.63
// at OLMoE's, with the same ranks.  z_lds is 16-byte aligned and holds 64 entries.
__device__ __forceinline__ int masked_rank(const float *z_lds, float z, int E, int lane,
                                           unsigned long long mask) {
    int r = 0;
    const float4 *z4 = reinterpret_cast<const float4 *>(z_lds);
    for (int j4 = 0; j4 < (E + 3) / 4; ++j4) {
        const float4 q = z4[j4];
        const int j = 4 * j4;
        const unsigned long long mb = mask >> j;
        r += ((mb & 1ull) && (q.x > z || (q.x == z && j < lane))) ? 1 : 0;
        r += ((mb & 2ull) && (q.y > z || (q.y == z && j + 1 < lane))) ? 1 : 0;
        r += ((mb & 4ull) && (q.z > z || (q.z == z && j + 2 < lane))) ? 1 : 0;
        r += ((mb & 8ull) && (q.w > z || (q.w == z && j + 3 < lane))) ? 1 : 0;
    }
    return r;
}

// Marks token b's outputs as written: every store of this wavefront first reaches the
// system (host memory included), then done[b] = seq, written by lane 0 (a vector store).
__device__ __forceinline__ void signal_done(int32_t *done, int32_t seq, int b, int lane) {
    if (!done) return;
    __threadfence_system();
    if (lane == 0) __hip_atomic_store(done + b, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ float logit_of(float tau) {
    if (tau <= 0.f) return -INFINITY;
    if (tau >= 1.f) return INFINITY;
    return logf(tau / (1.f - tau));
}

template <int NC, int EPP>
__global__ __launch_bounds__(kThreads) void prefetch_route_kernel(
    const float *__restrict__ h_pre, const uint16_t *__restrict__ w_pf,
    const float *__restrict__ b_pf, int d, int E, int k, int k_max, int policy, float tau,
    int static_delta, const float *__restrict__ cdf_w, const float *__restrict__ cdf_theta,
    int32_t *__restrict__ pf_idx, int32_t *__restrict__ pf_count, float *__restrict__ pf_prob,
    int32_t *__restrict__ done, int32_t seq) {
    __shared__ __align__(16) float z_lds[APEX_MAX_EXPERTS];
    __shared__ float sorted_q[APEX_MAX_EXPERTS];
    __shared__ int sorted_id[APEX_MAX_EXPERTS];

    const int b = blockIdx.x;
    token_logits<NC, EPP>(h_pre + size_t(b) * d, w_pf, b_pf, d, E, z_lds);

    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (wave != 0) return;   // selection is one wavefront's work; no barriers follow

    const bool live = lane < E;
    const float z = live ? z_lds[lane] : -INFINITY;
    const float mx = wave_max(z);
    const float p = live ? expf(z - mx) : 0.f;
    const float q = p / wave_sum(p);
    const unsigned long long all = (E == 64) ? ~0ull : ((1ull << E) - 1ull);
    const int r = masked_rank(z_lds, z, E, lane, all);
    if (live) {
        sorted_q[r] = q;
        sorted_id[r] = lane;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    const float qs = live ? sorted_q[lane] : 0.f;

    int m;
    if (policy == APEX_SEL_CUMPROB) {
        float S = qs;   // inclusive prefix sum in ranked order
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const float t = __shfl_up(S, o, kWave);
            if (lane >= o) S += t;
        }
        const unsigned long long hit = __ballot(live && S >= tau);
        const int m_star = hit ? __ffsll(static_cast<long long>(hit)) : E;
        m = min(max(m_star, k), k_max);
    } else if (policy == APEX_SEL_ORDINAL_CDF) {
        const float s = wave_sum(live ? cdf_w[lane] * qs : 0.f);
        const float thr = logit_of(tau);
        const bool ok = (lane <= E - k) && (cdf_theta[lane <= E - k ? lane : 0] - s >= thr);
        const unsigned long long hit = __ballot(ok);
        const int delta_hat = hit ? __ffsll(static_cast<long long>(hit)) - 1 : E - k;
        m = min(k + delta_hat, k_max);
    } else if (policy == APEX_SEL_STATIC) {
        m = min(k + static_delta, k_max);
    } else {
        m = 0;   // APEX_SEL_NONE
    }
    if (lane < k_max) pf_idx[size_t(b) * k_max + lane] = lane < m ? sorted_id[lane] : -1;
    if (lane == 0) pf_count[b] = m;
    if (pf_prob && live) pf_prob[size_t(b) * E + lane] = q;
    signal_done(done, seq, b, lane);
}

template <int NC, int EPP>
__global__ __launch_bounds__(kThreads) void gate_topk_kernel(
    const float *__restrict__ h_post, const uint16_t *__restrict__ w_g,
    const float *__restrict__ b_g, int d, int E, int k, int mode,
    const uint8_t *__restrict__ avail, int avail_stride, int32_t *__restrict__ route_idx,
    float *__restrict__ route_gate, int32_t *__restrict__ exec_idx,
    float *__restrict__ exec_gate, float *__restrict__ gate_prob, int32_t *__restrict__ done,
    int32_t seq) {
    __shared__ __align__(16) float z_lds[APEX_MAX_EXPERTS];

    const int b = blockIdx.x;
    token_logits<NC, EPP>(h_post + size_t(b) * d, w_g, b_g, d, E, z_lds);

    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (wave != 0) return;

    const bool live = lane < E;
    const float z = live ? z_lds[lane] : -INFINITY;
    const float mx = wave_max(z);
    const float p = live ? expf(z - mx) : 0.f;
    const float psum = wave_sum(p);
    const unsigned long long all = (E == 64) ? ~0ull : ((1ull << E) - 1ull);

    const int r = masked_rank(z_lds, z, E, lane, all);
    const bool sel_r = live && r < k;
    const float rsum = wave_sum(sel_r ? p : 0.f);
    const size_t row = size_t(b) * k;
    if (sel_r) {
        route_idx[row + r] = lane;
        route_gate[row + r] = p / rsum;
    }
    if (mode == APEX_MODE_EXACT) {
        if (sel_r) {
            exec_idx[row + r] = lane;
            exec_gate[row + r] = p / rsum;
        }
    } else {
        const bool a = live && avail[size_t(b) * avail_stride + lane] != 0;
        const unsigned long long amask = __ballot(a);
        const int ra = masked_rank(z_lds, z, E, lane, amask);
        const bool sel = a && ra < k;
        const int n_sel = __popcll(__ballot(sel));
        const float xsum = wave_sum(sel ? p : 0.f);
        if (sel) {
            exec_idx[row + ra] = lane;
            exec_gate[row + ra] = p / xsum;
        }
        if (lane >= n_sel && lane < k) {
            exec_idx[row + lane] = -1;
            exec_gate[row + lane] = 0.f;
        }
    }
    if (gate_prob && live) gate_prob[size_t(b) * E + lane] = p / psum;
    signal_done(done, seq, b, lane);
}

// Shape of token_logits: experts per wavefront (1, 2 or 4 for E <= 16, 32, 64) and
// 16-byte chunks per lane per pass (1, 2 or 4; one pass up to d = 2048), with the
// staged loads of a pass, (EPP + 2) * NC * 4 registers, kept within the 128 registers a
// lane has in a 1024-thread workgroup.
struct LogitShape {
    int nc, epp;
};
LogitShape logit_shape(int d, int E) {
    const int nch = d / 8;
    const int epp = E <= kWaves ? 1 : (E <= 2 * kWaves ? 2 : 4);
    int nc = nch <= kWave ? 1 : (nch <= 2 * kWave ? 2 : 4);
    if (epp == 4 && nc == 4) nc = 2;
    return {nc, epp};
}

apex_status check_router_args(const char *fn, const float *h, const uint16_t *w, int B, int d,
                              int E, int k) {
    APEX_REQUIRE(B >= 0, "%s: B=%d must be >= 0", fn, B);
    APEX_REQUIRE(E >= 1, "%s: E=%d must be >= 1", fn, E);
    if (E > APEX_MAX_EXPERTS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: E=%d exceeds %d", fn, E, APEX_MAX_EXPERTS);
    APEX_REQUIRE(k >= 1 && k <= E, "%s: k=%d out of [1, E=%d]", fn, k, E);
    APEX_REQUIRE(d >= 8 && d % 8 == 0, "%s: d=%d must be a positive multiple of 8", fn, d);
    if (d > kMaxD) return apex::fail(APEX_E_UNSUPPORTED, "%s: d=%d exceeds %d", fn, d, kMaxD);
    if (B == 0) return APEX_OK;
    APEX_REQUIRE(h && w, "%s: NULL input pointer", fn);
    APEX_REQUIRE(apex::aligned16(h) && apex::aligned16(w), "%s: inputs must be 16-byte aligned",
                 fn);
    return APEX_OK;
}

}  // namespace

namespace apex {

apex_status prefetch_route(const float *h_pre, const uint16_t *w_pf, const float *b_pf, int B,
                           int d, int E, int k, int k_max, int policy, float tau,
                           int static_delta, const float *cdf_w, const float *cdf_theta,
                           int32_t *pf_idx, int32_t *pf_count, float *pf_prob, int32_t *done,
                           int32_t seq, hipStream_t stream) {
    const char *fn = "apex_prefetch_route";
    apex_status st = check_router_args(fn, h_pre, w_pf, B, d, E, k);
    if (st != APEX_OK) return st;
    APEX_REQUIRE(k_max >= k && k_max <= E, "%s: k_max=%d out of [k=%d, E=%d]", fn, k_max, k, E);
    APEX_REQUIRE(policy == APEX_SEL_CUMPROB || policy == APEX_SEL_ORDINAL_CDF ||
                     policy == APEX_SEL_STATIC || policy == APEX_SEL_NONE,
                 "%s: unknown policy %d", fn, policy);
    APEX_REQUIRE(policy == APEX_SEL_STATIC || policy == APEX_SEL_NONE ||
                     (tau >= 0.f && tau <= 1.f),
                 "%s: tau=%g out of [0, 1]", fn, double(tau));
    APEX_REQUIRE(policy != APEX_SEL_STATIC || static_delta >= 0, "%s: static_delta=%d < 0", fn,
                 static_delta);
    APEX_REQUIRE(policy != APEX_SEL_ORDINAL_CDF || (cdf_w && cdf_theta),
                 "%s: ORDINAL_CDF needs cdf_w and cdf_theta", fn);
    if (B == 0) return APEX_OK;
    APEX_REQUIRE(pf_idx && pf_count, "%s: NULL output pointer", fn);
#define APEX_ROUTE(NC_, EPP_)                                                              \
    hipLaunchKernelGGL((prefetch_route_kernel<NC_, EPP_>), dim3(B), dim3(kThreads), 0, stream,  \
                       h_pre, w_pf, b_pf, d, E, k, k_max, policy, tau, static_delta, cdf_w,    \
                       cdf_theta, pf_idx, pf_count, pf_prob, done, seq)
    const LogitShape sh = logit_shape(d, E);
    if (sh.epp == 1) {
        if (sh.nc == 1) APEX_ROUTE(1, 1);
        else if (sh.nc == 2) APEX_ROUTE(2, 1);
        else APEX_ROUTE(4, 1);
    } else if (sh.epp == 2) {
        if (sh.nc == 1) APEX_ROUTE(1, 2);
        else if (sh.nc == 2) APEX_ROUTE(2, 2);
        else APEX_ROUTE(4, 2);
    } else {
        if (sh.nc == 1) APEX_ROUTE(1, 4);
        else APEX_ROUTE(2, 4);
    }
#undef APEX_ROUTE
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

apex_status gate_topk(const float *h_post, const uint16_t *w_g, const float *b_g, int B, int d,
                      int E, int k, int mode, const uint8_t *avail, int avail_stride,
                      int32_t *route_idx, float *route_gate, int32_t *exec_idx, float *exec_gate,
                      float *gate_prob, int32_t *done, int32_t seq, hipStream_t stream) {
    const char *fn = "apex_gate_topk";
    apex_status st = check_router_args(fn, h_post, w_g, B, d, E, k);
    if (st != APEX_OK) return st;
    APEX_REQUIRE(mode == APEX_MODE_EXACT || mode == APEX_MODE_STALL_FREE, "%s: unknown mode %d",
                 fn, mode);
    if (mode == APEX_MODE_STALL_FREE) {
        APEX_REQUIRE(avail_stride == 0 || avail_stride >= E,
                     "%s: avail_stride=%d must be 0 or >= E", fn, avail_stride);
        APEX_REQUIRE(B == 0 || avail, "%s: STALL_FREE needs avail", fn);
    }
    if (B == 0) return APEX_OK;
    APEX_REQUIRE(route_idx && route_gate && exec_idx && exec_gate, "%s: NULL output pointer", fn);
#define APEX_GATE(NC_, EPP_)                                                               \
    hipLaunchKernelGGL((gate_topk_kernel<NC_, EPP_>), dim3(B), dim3(kThreads), 0, stream,       \
                       h_post, w_g, b_g, d, E, k, mode, avail, avail_stride, route_idx,        \
                       route_gate, exec_idx, exec_gate, gate_prob, done, seq)
    const LogitShape sh = logit_shape(d, E);
    if (sh.epp == 1) {
        if (sh.nc == 1) APEX_GATE(1, 1);
        else if (sh.nc == 2) APEX_GATE(2, 1);
        else APEX_GATE(4, 1);
    } else if (sh.epp == 2) {
        if (sh.nc == 1) APEX_GATE(1, 2);
        else if (sh.nc == 2) APEX_GATE(2, 2);
        else APEX_GATE(4, 2);
    } else {
        if (sh.nc == 1) APEX_GATE(1, 4);
        else APEX_GATE(2, 4);
    }
#undef APEX_GATE
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace apex

extern "C" apex_status apex_prefetch_route(const float *h_pre, const uint16_t *w_pf,
                                           const float *b_pf, int B, int d, int E, int k,
                                           int k_max, int policy, float tau, int static_delta,
                                           const float *cdf_w, const float *cdf_theta,
                                           int32_t *pf_idx, int32_t *pf_count, float *pf_prob,
                                           hipStream_t stream) {
    return apex::prefetch_route(h_pre, w_pf, b_pf, B, d, E, k, k_max, policy, tau, static_delta,
                                cdf_w, cdf_theta, pf_idx, pf_count, pf_prob, nullptr, 0, stream);
}

extern "C" apex_status apex_gate_topk(const float *h_post, const uint16_t *w_g, const float *b_g,
                                      int B, int d, int E, int k, int mode,
                                      const uint8_t *avail, int avail_stride, int32_t *route_idx,
                                      float *route_gate, int32_t *exec_idx, float *exec_gate,
                                      float *gate_prob, hipStream_t stream) {
    return apex::gate_topk(h_post, w_g, b_g, B, d, E, k, mode, avail, avail_stride, route_idx,
                           route_gate, exec_idx, exec_gate, gate_prob, nullptr, 0, stream);
}
