// Decode driver: every layer of one decode step in native code (see apex.h).
//
// The host only has to see the prefetched set (to plan and issue the copies) and, in
// the correctness-preserving mode, the routed set (to fetch misses).  Both are written
// by the kernels straight into pinned host memory, each followed by a completion flag
// the host spins on, so the hand-off costs microseconds.  Overlap statistics are folded
// in lazily, once a layer's gate is known to have finished.
//
// A layer whose every expert is resident (C = E, no slot empty) can neither copy nor
// miss, so the host needs neither set in time: its router, window, gate and FFN go to
// the compute stream back to back with no wait, and the prefetched sets, the statistics
// and the host's cache plan (which then only renews last uses) are taken when the
// layer-step is folded, before the layer's next router writes its staging again.
// Recorded steps take the general route.
//
// Two streams.  The compute stream carries the chain that bounds a layer whenever the
// copies cannot be hidden: router, expert copies, expert FFN, next layer's router.
// Kernels back to back on one queue start without a gap, while an event recorded
// between them costs the queue several microseconds and a wait on another queue's event
// about ten, so that chain holds no events.  The side stream carries the work that only
// has to finish before the FFN: the slot-table publish, the attention window and the
// gate (and the shared experts).  The host orders the two through the flags: it enqueues
// the side stream's work once it has seen the router's flags (the router follows the
// previous layer's FFN, so that FFN is done too), and the FFN once it has seen the
// gate's, where the FFN queues behind the copies still in flight.  Slot reuse needs no
// event: a layer's copies follow, on the compute stream, every earlier kernel that read
// those slots.  Only the shared experts, which publish no flag, and the miss
// copy of the correctness-preserving mode are waited for with an event: the missing
// experts travel on the side stream while the first FFN pass runs, and the second pass
// waits for them.  A layer-step that copies nothing else keeps its other work on the
// compute stream: with no copy to hide behind, the hand-offs between streams would only
// add their latency.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
#include <cstring>
#include <vector>

#include "common.h"
#include "prefetch_internal.h"
#include "route_internal.h"

struct apex_decode {
    apex_decode_config cfg;
    std::vector<apex_decode_layer> layers;
    std::vector<const uint4 *> host_view;   // device view of each layer's pinned experts
    uint16_t *scratch = nullptr;
    int32_t *miss_table = nullptr;
    int32_t *exec_idx = nullptr;
    float *exec_gate = nullptr;
    void *ws = nullptr;
    size_t ws_bytes = 0;
    hipStream_t compute = nullptr, side = nullptr;
    size_t expert_bytes = 0;
    // attention window (attn_heads > 0)
    void *attn_ws = nullptr;
    size_t attn_ws_bytes = 0;
    // shared experts (n_shared > 0): every token runs shared expert s at position s with
    // gate 1 over a pool whose slot s is expert s
    int32_t *shared_idx = nullptr;     // device [B][n_shared]
    float *shared_gate = nullptr;      // device [B][n_shared]
    int32_t *shared_table = nullptr;   // device [n_shared]
    // pinned staging
    int32_t *pf_idx_h = nullptr;      // [L][B][k_max], one slice per layer
    int32_t *pf_count_h = nullptr;    // [L][B]
    int32_t *route_idx_h = nullptr;   // [L][B][k]
    float *route_gate_h = nullptr;    // [L][B][k]
    // completion flags the router and gate kernels write into pinned memory after their
    // outputs: route_done[b], gate_done_h[l][b] = the layer-step's sequence number
    int32_t *route_done = nullptr;    // [B]
    int32_t *gate_done_h = nullptr;   // [L][B]
    int32_t seq = 0;
    // event after the shared experts (side stream)
    hipEvent_t shared_done = nullptr;
    // event after a layer-step's miss copy (side stream), waited for by the second pass
    hipEvent_t miss_ready = nullptr;
    // statistics of layers whose gate may still be running
    struct Pending {
        int layer;
        int32_t seq;                   // the layer-step's sequence number
        hipStream_t gate_stream;       // the stream the layer-step's gate ran on
        std::vector<int32_t> pf;       // [B][k_max]
        std::vector<int32_t> cnt;      // [B]
        std::vector<char> resident;    // [E]
        int copies, misses;
        // a layer-step whose every expert was resident, enqueued without waiting for the
        // router: its prefetched sets are read (and the host's cache plan, which then
        // only renews last uses, is run) when it is folded
        bool deferred = false;
        int64_t step = 0;
    };
    std::vector<Pending> pending;
};

namespace {

// Waits until a kernel enqueued on `stream` has published its outputs: every done[b]
// equals seq (the kernel writes them after its outputs, behind a system-scope fence), or
// the stream has drained, whichever the host sees first.  Busy-polls (lower wake-up
// latency than a blocking wait); the stream query, every 256 polls, reports a device
// error, and after 30 s the call gives up, so that a device that stopped making progress
// surfaces as an error.
apex_status poll_done(const int32_t *done, int n, int32_t seq, hipStream_t stream) {
    const auto t0 = std::chrono::steady_clock::now();
    for (unsigned it = 0;; ++it) {
        bool all = true;
        for (int b = 0; b < n && all; ++b)
            all = __atomic_load_n(done + b, __ATOMIC_ACQUIRE) == seq;
        if (all) return APEX_OK;
        if ((it & 255u) == 255u) {
            const hipError_t e = hipStreamQuery(stream);
            if (e == hipSuccess) return APEX_OK;
            if (e != hipErrorNotReady)
                return apex::fail(APEX_E_HIP, "hipStreamQuery failed: %s", hipGetErrorString(e));
            if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(30))
                return apex::fail(APEX_E_HIP, "apex_decode_step: kernel not done after 30 s");
        }
    }
}

void fold(apex_decode *dec, const apex_decode::Pending &p, apex_decode_stats *st) {
    if (!st) return;
    const apex_decode_config &c = dec->cfg;
    const int32_t *route = dec->route_idx_h + size_t(p.layer) * c.B * c.k;
    for (int b = 0; b < c.B; ++b) {
        char in_p[APEX_MAX_EXPERTS] = {0};
        for (int j = 0; j < p.cnt[b]; ++j) in_p[p.pf[size_t(b) * c.k_max + j]] = 1;
        int both = 0, hit = 0;
        for (int j = 0; j < c.k; ++j) {
            const int e = route[size_t(b) * c.k + j];
            if (e < 0 || e >= c.E) continue;
            both += in_p[e];
            hit += p.resident[e];
        }
        st->overlap_sum += double(both) / c.k;
        st->hit_sum += double(hit) / c.k;
        st->coverage_count += both == c.k ? 1 : 0;
        // delta_hat in [0, E - k] (Eq. 9); the no-prefetch baseline fetches no extra
        // experts, so its empty prefetched set counts 0
        st->delta_hat_sum += std::max(p.cnt[b] - c.k, 0);
    }
    st->tokens += c.B;
    st->layer_steps += 1;
    st->copies += p.copies;
    st->misses += p.misses;
}

// One expert-FFN pass in the layer's weight format.
apex_status run_ffn(apex_decode *dec, const float *x, int I, int E, int k, const int32_t *idx,
                    const float *gate, const int32_t *slot_of_expert, const void *slots,
                    int n_slots, float *y, int accumulate, hipStream_t stream) {
    const apex_decode_config &c = dec->cfg;
    if (c.weights == APEX_WEIGHTS_FP8_E4M3)
        return apex_moe_ffn_fp8(x, c.B, c.d, I, E, k, idx, gate, slot_of_expert, slots, n_slots,
                                y, accumulate, dec->ws, dec->ws_bytes, stream);
    if (c.weights == APEX_WEIGHTS_MXFP4)
        return apex_moe_ffn_mxfp4(x, c.B, c.d, I, E, k, idx, gate, slot_of_expert, slots,
                                  n_slots, y, accumulate, dec->ws, dec->ws_bytes, stream);
    if (c.weights == APEX_WEIGHTS_FP32)
        return apex_moe_ffn_fp32(x, c.B, c.d, I, E, k, idx, gate, slot_of_expert, slots,
                                 n_slots, y, accumulate, dec->ws, dec->ws_bytes, stream);
    return apex_moe_ffn(x, c.B, c.d, I, E, k, idx, gate, slot_of_expert,
                        static_cast<const uint16_t *>(slots), n_slots, y, accumulate, dec->ws,
                        dec->ws_bytes, stream);
}

// The routed experts' executed sets over the given slot pool.
apex_status ffn(apex_decode *dec, const float *x, const int32_t *slot_of_expert,
                const uint16_t *slots, int n_slots, float *y, int accumulate) {
    const apex_decode_config &c = dec->cfg;
    return run_ffn(dec, x, c.I, c.E, c.k, dec->exec_idx, dec->exec_gate, slot_of_expert, slots,
                   n_slots, y, accumulate, dec->compute);
}

// Folds one pending layer-step once its gate has published the routed sets (normally
// long done: it precedes that layer's FFN).  A deferred layer-step first takes its
// prefetched sets from the layer's staging slice (the router ran before the gate on the
// same stream) and runs the host's cache plan on them, which with every expert resident
// copies nothing and only renews last uses.
apex_status fold_one(apex_decode *dec, apex_decode::Pending &p, apex_decode_stats *st) {
    const apex_decode_config &c = dec->cfg;
    const int B = c.B;
    apex_status s = poll_done(dec->gate_done_h + size_t(p.layer) * B, B, p.seq, p.gate_stream);
    if (s != APEX_OK) return s;
    if (p.deferred) {
        const int32_t *pf = dec->pf_idx_h + size_t(p.layer) * B * c.k_max;
        const int32_t *cnt = dec->pf_count_h + size_t(p.layer) * B;
        p.pf.assign(pf, pf + size_t(B) * c.k_max);
        p.cnt.assign(cnt, cnt + B);
        const apex_decode_layer &Ly = dec->layers[p.layer];
        int32_t ce[APEX_MAX_EXPERTS], cs[APEX_MAX_EXPERTS];
        int n = 0;
        s = apex_plan_residency(c.E, c.C, pf, cnt, B, c.k_max, p.step, Ly.expert_of_slot,
                                Ly.last_used, ce, cs, &n);
        if (s != APEX_OK) return s;
        APEX_REQUIRE(n == 0, "apex_decode_step: layer %d planned %d copies with every expert "
                     "resident", p.layer, n);
    }
    fold(dec, p, st);
    return APEX_OK;
}

// Folds every pending layer-step (layer < 0), or those of one layer.
apex_status fold_pending(apex_decode *dec, apex_decode_stats *st, int layer = -1) {
    auto &v = dec->pending;
    size_t keep = 0;
    for (size_t i = 0; i < v.size(); ++i) {
        if (layer >= 0 && v[i].layer != layer) {
            if (keep != i) v[keep] = std::move(v[i]);
            ++keep;
            continue;
        }
        const apex_status s = fold_one(dec, v[i], st);
        if (s != APEX_OK) return s;
    }
    v.resize(keep);
    return APEX_OK;
}

// Every expert of the layer is resident (C = E, no slot empty): no copy and no miss can
// happen, so nothing of the layer-step waits for the host.
bool all_resident(const apex_decode_config &c, const apex_decode_layer &Ly) {
    if (c.C < c.E) return false;
    for (int s = 0; s < c.C; ++s)
        if (Ly.expert_of_slot[s] < 0) return false;
    return true;
}

// The attention window of layer l on `stream`: the layer's decode attention, or the
// spin of t_attn_us.
apex_status window(apex_decode *dec, int l, const float *h_pre, hipStream_t stream) {
    const apex_decode_config &c = dec->cfg;
    const apex_decode_layer &Ly = dec->layers[l];
    if (c.attn_heads > 0)
        return apex_attention_decode(h_pre, Ly.w_qkv, Ly.w_o, c.B, c.d, c.attn_heads,
                                     c.attn_kv_heads, c.d / c.attn_heads, Ly.k_cache,
                                     Ly.v_cache, c.attn_ctx + 1, c.attn_ctx, Ly.attn_out,
                                     dec->attn_ws, dec->attn_ws_bytes, stream);
    if (c.t_attn_us > 0) return apex_spin_us(c.t_attn_us, stream);
    return APEX_OK;
}

// A layer-step with every expert resident: router, window, gate (with the shared
// experts) and FFN queued back to back on the compute stream, no host wait.  Nothing is
// copied or missed; the statistics and the host's cache plan wait for the fold.
apex_status enqueue_resident(apex_decode *dec, int l, int64_t step, int32_t seq,
                             const float *h_pre, const float *h_post, float *y) {
    const apex_decode_config &c = dec->cfg;
    const apex_decode_layer &Ly = dec->layers[l];
    const hipStream_t cs = dec->compute;
    int32_t *pf_h = dec->pf_idx_h + size_t(l) * c.B * c.k_max;
    int32_t *pfc_h = dec->pf_count_h + size_t(l) * c.B;
    apex_status st;
    if (c.policy != APEX_SEL_NONE) {
        // the flag is not waited for, but its system-scope fence orders the sets in host
        // memory before the gate's flag, which the fold waits for
        st = apex::prefetch_route(h_pre, Ly.w_pf, Ly.b_pf, c.B, c.d, c.E, c.k, c.k_max,
                                  c.policy, c.tau, c.static_delta, Ly.cdf_w, Ly.cdf_theta, pf_h,
                                  pfc_h, nullptr, dec->route_done, seq, cs);
        if (st != APEX_OK) return st;
    } else {
        std::fill(pf_h, pf_h + size_t(c.B) * c.k_max, -1);
        std::fill(pfc_h, pfc_h + c.B, 0);
    }
    st = window(dec, l, h_pre, cs);
    if (st != APEX_OK) return st;
    st = apex::gate_topk(h_post, Ly.w_g, Ly.b_g, c.B, c.d, c.E, c.k, c.mode, Ly.avail_dev, 0,
                         dec->route_idx_h + size_t(l) * c.B * c.k,
                         dec->route_gate_h + size_t(l) * c.B * c.k, dec->exec_idx,
                         dec->exec_gate, nullptr, dec->gate_done_h + size_t(l) * c.B, seq, cs);
    if (st != APEX_OK) return st;
    const bool shared = c.n_shared > 0;
    if (shared) {
        st = run_ffn(dec, h_post, c.I_shared, c.n_shared, c.n_shared, dec->shared_idx,
                     dec->shared_gate, dec->shared_table, Ly.shared_slots, c.n_shared, y, 0,
                     cs);
        if (st != APEX_OK) return st;
    }
    st = ffn(dec, h_post, Ly.slot_of_expert_dev, Ly.slots, c.C, y, shared ? 1 : 0);
    if (st != APEX_OK) return st;
    apex_decode::Pending p;
    p.layer = l;
    p.seq = seq;
    p.gate_stream = cs;
    p.resident.assign(c.E, 1);
    p.copies = 0;
    p.misses = 0;
    p.deferred = true;
    p.step = step;
    dec->pending.push_back(std::move(p));
    return APEX_OK;
}

}  // namespace

extern "C" apex_status apex_decode_create(apex_decode **out, const apex_decode_config *cfg,
                                          const apex_decode_layer *layers, uint16_t *scratch,
                                          int32_t *miss_table_dev, int32_t *exec_idx_dev,
                                          float *exec_gate_dev, void *workspace,
                                          size_t workspace_bytes, hipStream_t compute,
                                          hipStream_t side) {
    const char *fn = "apex_decode_create";
    APEX_REQUIRE(out && cfg && layers, "%s: NULL argument", fn);
    const apex_decode_config &c = *cfg;
    APEX_REQUIRE(c.L >= 1 && c.B >= 1, "%s: L=%d B=%d", fn, c.L, c.B);
    APEX_REQUIRE(c.E >= 1 && c.E <= APEX_MAX_EXPERTS, "%s: E=%d", fn, c.E);
    APEX_REQUIRE(c.k >= 1 && c.k <= c.k_max && c.k_max <= c.C && c.C <= c.E,
                 "%s: need 1 <= k <= k_max <= C <= E (k=%d k_max=%d C=%d E=%d)", fn, c.k,
                 c.k_max, c.C, c.E);
    APEX_REQUIRE(c.t_attn_us >= 0.0 && c.t_attn_us <= 1e6, "%s: t_attn_us=%g", fn, c.t_attn_us);
    APEX_REQUIRE(c.weights >= APEX_WEIGHTS_BF16 && c.weights <= APEX_WEIGHTS_FP32,
                 "%s: unknown weight format %d", fn, c.weights);
    if (c.weights == APEX_WEIGHTS_FP32 && c.B != 1)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: 32-bit experts run at batch 1 only (B=%d)",
                          fn, c.B);
    // one 16-byte load holds 4 fp32, 8 bf16 or 16 E4M3 weights; MXFP4 rows are whole
    // 32-value blocks
    const int mult = c.weights == APEX_WEIGHTS_FP32          ? 4
                     : c.weights == APEX_WEIGHTS_BF16        ? 8
                     : c.weights == APEX_WEIGHTS_FP8_E4M3    ? 16
                                                             : 32;
    APEX_REQUIRE(c.d % mult == 0 && c.I % mult == 0,
                 "%s: weight format %d needs d and I multiples of %d (d=%d I=%d)", fn, c.weights,
                 mult, c.d, c.I);
    APEX_REQUIRE(c.mode == APEX_MODE_EXACT || c.mode == APEX_MODE_STALL_FREE, "%s: mode %d", fn,
                 c.mode);
    APEX_REQUIRE(c.mode != APEX_MODE_EXACT || (scratch && miss_table_dev && c.n_scratch >= 1),
                 "%s: EXACT mode needs a miss scratch pool", fn);
    APEX_REQUIRE(exec_idx_dev && exec_gate_dev && workspace, "%s: NULL buffer", fn);
    APEX_REQUIRE(c.n_shared >= 0 && c.n_shared <= APEX_MAX_EXPERTS,
                 "%s: n_shared=%d out of [0, %d]", fn, c.n_shared, APEX_MAX_EXPERTS);
    APEX_REQUIRE(c.n_shared == 0 || (c.I_shared >= mult && c.I_shared % mult == 0),
                 "%s: I_shared=%d must be a positive multiple of %d", fn, c.I_shared, mult);
    if (size_t(c.B) * c.n_shared > APEX_MAX_PAIRS)
        return apex::fail(APEX_E_UNSUPPORTED, "%s: B*n_shared=%d exceeds %d", fn,
                          c.B * c.n_shared, APEX_MAX_PAIRS);
    size_t ws_need = apex_moe_ffn_workspace_bytes(c.B, c.d, c.I, c.k);
    if (c.n_shared > 0)
        ws_need = std::max(ws_need, apex_moe_ffn_workspace_bytes(c.B, c.d, c.I_shared,
                                                                 c.n_shared));
    if (workspace_bytes < ws_need)
        return apex::fail(APEX_E_CAPACITY, "%s: workspace %zu < %zu bytes", fn, workspace_bytes,
                          ws_need);
    const bool attn = c.attn_heads > 0;
    if (attn) {
        APEX_REQUIRE(c.attn_kv_heads >= 1 && c.attn_ctx >= 0 && c.d % c.attn_heads == 0,
                     "%s: attention window: heads=%d kv_heads=%d ctx=%d d=%d", fn, c.attn_heads,
                     c.attn_kv_heads, c.attn_ctx, c.d);
        const int hd = c.d / c.attn_heads;
        APEX_REQUIRE((hd == 64 || hd == 128) && c.attn_heads % c.attn_kv_heads == 0,
                     "%s: attention window: head size %d, heads %d, kv heads %d", fn, hd,
                     c.attn_heads, c.attn_kv_heads);
    }
    for (int l = 0; l < c.L; ++l) {
        const apex_decode_layer &y = layers[l];
        APEX_REQUIRE(y.w_pf && y.w_g && y.host_experts && y.slots && y.slot_of_expert_dev &&
                         y.expert_of_slot && y.last_used,
                     "%s: layer %d has a NULL buffer", fn, l);
        APEX_REQUIRE(c.n_shared == 0 || y.shared_slots,
                     "%s: layer %d has no shared-expert pool", fn, l);
        APEX_REQUIRE(!attn || (y.w_qkv && y.w_o && y.k_cache && y.v_cache && y.attn_out),
                     "%s: layer %d has no attention buffers", fn, l);
    }
    auto *dec = new apex_decode();
    dec->cfg = c;
    dec->layers.assign(layers, layers + c.L);
    dec->host_view.assign(c.L, nullptr);
    dec->scratch = scratch;
    dec->miss_table = miss_table_dev;
    dec->exec_idx = exec_idx_dev;
    dec->exec_gate = exec_gate_dev;
    dec->ws = workspace;
    dec->ws_bytes = workspace_bytes;
    dec->compute = compute;
    dec->side = side;
    dec->expert_bytes = c.weights == APEX_WEIGHTS_FP8_E4M3 ? apex_expert_bytes_fp8(c.d, c.I)
                        : c.weights == APEX_WEIGHTS_MXFP4  ? apex_expert_bytes_mxfp4(c.d, c.I)
                        : c.weights == APEX_WEIGHTS_FP32   ? apex_expert_bytes_fp32(c.d, c.I)
                                                           : apex_expert_bytes(c.d, c.I);
    auto cleanup = [&](apex_status st) {
        apex_decode_destroy(dec);
        return st;
    };
    for (int l = 0; l < c.L; ++l) {
        const apex_status st = apex::pinned_device_view(fn, layers[l].host_experts,
                                                        size_t(c.E) * dec->expert_bytes,
                                                        &dec->host_view[l]);
        if (st != APEX_OK) return cleanup(st);
    }
    hipError_t e = hipSuccess;
    e = hipHostMalloc(reinterpret_cast<void **>(&dec->pf_idx_h),
                      sizeof(int32_t) * c.L * c.B * c.k_max);
    if (e == hipSuccess)
        e = hipHostMalloc(reinterpret_cast<void **>(&dec->pf_count_h),
                          sizeof(int32_t) * c.L * c.B);
    if (e == hipSuccess)
        e = hipHostMalloc(reinterpret_cast<void **>(&dec->route_idx_h),
                          sizeof(int32_t) * c.L * c.B * c.k);
    if (e == hipSuccess)
        e = hipHostMalloc(reinterpret_cast<void **>(&dec->route_gate_h),
                          sizeof(float) * c.L * c.B * c.k);
    if (e == hipSuccess)
        e = hipHostMalloc(reinterpret_cast<void **>(&dec->route_done), sizeof(int32_t) * c.B);
    if (e == hipSuccess)
        e = hipHostMalloc(reinterpret_cast<void **>(&dec->gate_done_h),
                          sizeof(int32_t) * c.L * c.B);
    if (e == hipSuccess) {
        std::fill(dec->route_done, dec->route_done + c.B, 0);
        std::fill(dec->gate_done_h, dec->gate_done_h + size_t(c.L) * c.B, 0);
    }
    if (e != hipSuccess)
        return cleanup(apex::fail(APEX_E_HIP, "%s: hipHostMalloc failed: %s", fn,
                                  hipGetErrorString(e)));
    auto mk = [&](hipEvent_t *ev) {
        return hipEventCreateWithFlags(ev, hipEventDisableTiming);
    };
    if (mk(&dec->shared_done) != hipSuccess || mk(&dec->miss_ready) != hipSuccess)
        return cleanup(apex::fail(APEX_E_HIP, "%s: event creation failed", fn));
    if (c.n_shared > 0) {
        const size_t pairs = size_t(c.B) * c.n_shared;
        std::vector<int32_t> idx(pairs), table(c.n_shared);
        std::vector<float> gate(pairs, 1.f);
        for (size_t i = 0; i < pairs; ++i) idx[i] = int32_t(i % c.n_shared);
        for (int s2 = 0; s2 < c.n_shared; ++s2) table[s2] = s2;
        e = hipMalloc(reinterpret_cast<void **>(&dec->shared_idx), 4 * pairs);
        if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&dec->shared_gate), 4 * pairs);
        if (e == hipSuccess)
            e = hipMalloc(reinterpret_cast<void **>(&dec->shared_table), 4 * size_t(c.n_shared));
        if (e == hipSuccess)
            e = hipMemcpy(dec->shared_idx, idx.data(), 4 * pairs, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = hipMemcpy(dec->shared_gate, gate.data(), 4 * pairs, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = hipMemcpy(dec->shared_table, table.data(), 4 * size_t(c.n_shared),
                          hipMemcpyHostToDevice);
        if (e != hipSuccess)
            return cleanup(apex::fail(APEX_E_HIP, "%s: shared-expert lists: %s", fn,
                                      hipGetErrorString(e)));
    }
    if (attn) {
        dec->attn_ws_bytes = apex_attention_workspace_bytes(c.B, c.attn_heads, c.attn_kv_heads,
                                                            c.d / c.attn_heads, c.attn_ctx + 1);
        e = hipMalloc(&dec->attn_ws, dec->attn_ws_bytes);
        if (e != hipSuccess)
            return cleanup(apex::fail(APEX_E_HIP, "%s: hipMalloc failed: %s", fn,
                                      hipGetErrorString(e)));
    }
    *out = dec;
    return APEX_OK;
}

extern "C" apex_status apex_decode_step(apex_decode *dec, int64_t step,
                                        const float *const *h_pre, const float *const *h_post,
                                        float *const *y, apex_decode_stats *stats,
                                        apex_decode_record *rec) {
    const char *fn = "apex_decode_step";
    APEX_REQUIRE(dec && h_pre && h_post && y, "%s: NULL argument", fn);
    const apex_decode_config &c = dec->cfg;
    const hipStream_t cs = dec->compute, ss = dec->side;
    std::vector<int32_t> copied(c.C), missing(c.E);
    apex_status st;
    for (int l = 0; l < c.L; ++l) {
        const apex_decode_layer &Ly = dec->layers[l];
        // prefetch stage: router on the pre-attention state, then the attention window
        // (the no-prefetch baseline has no router: its prefetched sets are empty)
        const bool route = c.policy != APEX_SEL_NONE;
        // sequence number of this layer-step (never 0, the flags' initial value)
        dec->seq = dec->seq == INT32_MAX ? 1 : dec->seq + 1;
        const int32_t seq = dec->seq;
        // this layer's previous layer-step is folded before its staging is written again
        st = fold_pending(dec, stats, l);
        if (st != APEX_OK) return st;
        if (!rec && all_resident(c, Ly)) {
            st = enqueue_resident(dec, l, step, seq, h_pre[l], h_post[l], y[l]);
            if (st != APEX_OK) return st;
            continue;
        }
        int32_t *pf_h = dec->pf_idx_h + size_t(l) * c.B * c.k_max;
        int32_t *pfc_h = dec->pf_count_h + size_t(l) * c.B;
        if (route) {
            st = apex::prefetch_route(h_pre[l], Ly.w_pf, Ly.b_pf, c.B, c.d, c.E, c.k, c.k_max,
                                      c.policy, c.tau, c.static_delta, Ly.cdf_w, Ly.cdf_theta,
                                      pf_h, pfc_h, nullptr, dec->route_done, seq, cs);
            if (st != APEX_OK) return st;
        } else {
            std::fill(pf_h, pf_h + size_t(c.B) * c.k_max, -1);
            std::fill(pfc_h, pfc_h + c.B, 0);
        }
        if (route) {
            st = poll_done(dec->route_done, c.B, seq, cs);
            if (st != APEX_OK) return st;
        }
        // copies on the compute stream (after every earlier reader of the slots), the new
        // slot table on the stream of the gate, which masks with it: the side stream if
        // anything is copied (the no-prefetch baseline never copies)
        int n_copy = 0;
        st = apex::expert_prefetch(dec->host_view[l], Ly.slots, c.E, c.C, dec->expert_bytes,
                                   pf_h, pfc_h, c.B, c.k_max, step,
                                   Ly.expert_of_slot, Ly.last_used, Ly.slot_of_expert_dev,
                                   Ly.avail_dev, cs, ss, cs, nullptr, nullptr, copied.data(),
                                   &n_copy, false);
        if (st != APEX_OK) return st;
        const bool split = n_copy > 0;
        const hipStream_t ws = split ? ss : cs;
        // the attention window
        st = window(dec, l, h_pre[l], ws);
        if (st != APEX_OK) return st;
        // earlier layer-steps' statistics, now that this layer's copies are on their way
        st = fold_pending(dec, stats);
        if (st != APEX_OK) return st;
        apex_decode::Pending p;
        p.layer = l;
        p.seq = seq;
        p.gate_stream = ws;
        p.pf.assign(pf_h, pf_h + size_t(c.B) * c.k_max);
        p.cnt.assign(pfc_h, pfc_h + c.B);
        p.resident.assign(c.E, 0);
        for (int s = 0; s < c.C; ++s)
            if (Ly.expert_of_slot[s] >= 0) p.resident[Ly.expert_of_slot[s]] = 1;
        p.copies = n_copy;
        p.misses = 0;
        if (rec) {
            if (rec->pf_idx)
                std::memcpy(rec->pf_idx + size_t(l) * c.B * c.k_max, pf_h,
                            sizeof(int32_t) * c.B * c.k_max);
            if (rec->pf_count)
                std::memcpy(rec->pf_count + size_t(l) * c.B, pfc_h,
                            sizeof(int32_t) * c.B);
            if (rec->resident)
                std::memcpy(rec->resident + size_t(l) * c.C, Ly.expert_of_slot,
                            sizeof(int32_t) * c.C);
            if (rec->n_copies) rec->n_copies[l] = n_copy;
        }
        // execution stage: original router
        int32_t *route_h = dec->route_idx_h + size_t(l) * c.B * c.k;
        float *route_g = dec->route_gate_h + size_t(l) * c.B * c.k;
        int32_t *gate_flags = dec->gate_done_h + size_t(l) * c.B;
        st = apex::gate_topk(h_post[l], Ly.w_g, Ly.b_g, c.B, c.d, c.E, c.k, c.mode,
                             Ly.avail_dev, 0, route_h, route_g, dec->exec_idx, dec->exec_gate,
                             nullptr, gate_flags, seq, ws);
        if (st != APEX_OK) return st;
        // shared experts: they need no copy, so they run beside the copies
        const bool shared = c.n_shared > 0;
        if (shared) {
            st = run_ffn(dec, h_post[l], c.I_shared, c.n_shared, c.n_shared, dec->shared_idx,
                         dec->shared_gate, dec->shared_table, Ly.shared_slots, c.n_shared, y[l],
                         0, ws);
            if (st != APEX_OK) return st;
            if (split) APEX_HIP(hipEventRecord(dec->shared_done, ss));
        }
        // on one stream the first FFN pass follows the gate in stream order; across
        // streams it is enqueued once the gate has published the executed sets, behind the
        // copies still in flight
        const int acc = shared ? 1 : 0;
        if (!split) {
            st = ffn(dec, h_post[l], Ly.slot_of_expert_dev, Ly.slots, c.C, y[l], acc);
            if (st != APEX_OK) return st;
        }
        // the correctness-preserving mode needs the routed sets in any case
        if (split || c.mode == APEX_MODE_EXACT) {
            st = poll_done(gate_flags, c.B, seq, ws);
            if (st != APEX_OK) return st;
        }
        if (split) {
            // the routed experts once the copies landed (stream order)
            if (shared) APEX_HIP(hipStreamWaitEvent(cs, dec->shared_done, 0));
            st = ffn(dec, h_post[l], Ly.slot_of_expert_dev, Ly.slots, c.C, y[l], acc);
            if (st != APEX_OK) return st;
        }
        int n_miss = 0;
        if (c.mode == APEX_MODE_EXACT) {
            // asynchronous miss correction (Sec. IV-E): the missing experts are copied on
            // the side stream while the first pass runs on the compute stream; the second
            // pass waits for the copy's event.  The scratch pool is free: the host got here
            // after seeing the flags of this layer-step's router or gate, kernels that
            // follow the previous second pass on the compute stream.
            st = apex::fetch_misses(Ly.host_experts, dec->host_view[l], dec->scratch,
                                    c.n_scratch, c.E, c.C, dec->expert_bytes, route_h, c.B, c.k,
                                    Ly.expert_of_slot, dec->miss_table, ss, cs, nullptr,
                                    dec->miss_ready, missing.data(), &n_miss);
            if (st != APEX_OK) return st;
        }
        if (n_miss > 0) {
            APEX_HIP(hipStreamWaitEvent(cs, dec->miss_ready, 0));
            st = ffn(dec, h_post[l], dec->miss_table, dec->scratch, c.n_scratch, y[l], 1);
            if (st != APEX_OK) return st;
        }
        p.misses = n_miss;
        dec->pending.push_back(std::move(p));
        if (rec) {
            APEX_HIP(hipStreamSynchronize(cs));
            const size_t bk = size_t(c.B) * c.k;
            if (rec->route_idx) std::memcpy(rec->route_idx + l * bk, route_h, 4 * bk);
            if (rec->route_gate) std::memcpy(rec->route_gate + l * bk, route_g, 4 * bk);
            if (rec->exec_idx)
                APEX_HIP(hipMemcpy(rec->exec_idx + l * bk, dec->exec_idx, 4 * bk,
                                   hipMemcpyDeviceToHost));
            if (rec->exec_gate)
                APEX_HIP(hipMemcpy(rec->exec_gate + l * bk, dec->exec_gate, 4 * bk,
                                   hipMemcpyDeviceToHost));
            if (rec->missing)
                for (int i = 0; i < n_miss; ++i) rec->missing[size_t(l) * c.E + i] = missing[i];
            if (rec->n_missing) rec->n_missing[l] = n_miss;
        }
    }
    if (rec) return fold_pending(dec, stats);
    return APEX_OK;
}

extern "C" apex_status apex_decode_finish(apex_decode *dec, apex_decode_stats *stats) {
    APEX_REQUIRE(dec, "apex_decode_finish: NULL driver");
    APEX_HIP(hipStreamSynchronize(dec->compute));
    APEX_HIP(hipStreamSynchronize(dec->side));
    return fold_pending(dec, stats);
}

extern "C" apex_status apex_decode_destroy(apex_decode *dec) {
    if (!dec) return APEX_OK;
    if (dec->compute) (void)hipStreamSynchronize(dec->compute);
    if (dec->side) (void)hipStreamSynchronize(dec->side);
    if (dec->shared_done) (void)hipEventDestroy(dec->shared_done);
    if (dec->miss_ready) (void)hipEventDestroy(dec->miss_ready);
    for (void *p : {static_cast<void *>(dec->pf_idx_h), static_cast<void *>(dec->pf_count_h),
                    static_cast<void *>(dec->route_idx_h), static_cast<void *>(dec->route_gate_h),
                    static_cast<void *>(dec->route_done), static_cast<void *>(dec->gate_done_h)})
        if (p) (void)hipHostFree(p);
    if (dec->attn_ws) (void)hipFree(dec->attn_ws);
    for (void *p : {static_cast<void *>(dec->shared_idx), static_cast<void *>(dec->shared_gate),
                    static_cast<void *>(dec->shared_table)})
        if (p) (void)hipFree(p);
    delete dec;
    return APEX_OK;
}
