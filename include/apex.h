/*
 * apex.h - C ABI of the MI355X (gfx950) hot path of adaptive expert prefetching for
 * Mixture-of-Experts decode (APEX: Adaptive Expert Prefetching for Memory-Efficient
 * Edge MoE Inference).
 *
 * One MoE layer, one decode step, runs as:
 *   apex_prefetch_route   prefetch router on the pre-attention state, ranked list,
 *                         adaptive prefetch set K_p                  (Sec. IV-A..IV-C)
 *   apex_expert_prefetch  cache plan + host-to-HBM copies of non-resident experts of
 *                         K_p on a side stream while attention runs  (Sec. IV-A, IV-D)
 *   apex_gate_topk        original router top-k K_r; executed set in correctness-
 *                         preserving or stall-free mode              (Sec. IV-E, Alg. 1)
 *   apex_moe_ffn          gated SwiGLU experts read from HBM slots   (Sec. III-A, IV-E)
 *   apex_expert_fetch_misses + a second apex_moe_ffn pass (accumulate = 1): the
 *                         asynchronous miss correction of the correctness-preserving
 *                         mode                                       (Sec. IV-E)
 *
 * Conventions, for every entry point:
 *  - Buffers are owned by the caller.  No entry point allocates or frees memory, except
 *    apex_decode_create and apex_decode_destroy, which set up and release the decode
 *    driver's own staging and tables (setup time, not the hot path).
 *  - "device" pointers are HBM addresses (hipMalloc or equivalent); "host" pointers
 *    are ordinary host memory; "pinned" pointers are page-locked host memory
 *    (hipHostMalloc or equivalent).  Device pointers must be 16-byte aligned.
 *  - Matrices are row-major.  bf16 values are passed as uint16_t bit patterns.
 *  - Work is enqueued on the given stream and runs asynchronously to the host unless
 *    the entry point says otherwise.  A NULL stream is the default stream.
 *  - Arguments are validated before anything is enqueued; on an invalid argument the
 *    call returns an error, enqueues nothing and leaves every output untouched.  The
 *    message of the last failing call on the calling thread is apex_last_error().
 *  - Supported sizes: 1 <= E <= 64 experts, 1 <= k <= k_max <= E, d and I multiples
 *    of 8 (16-byte rows of bf16), B >= 0 tokens (B = 0 enqueues nothing).
 *  - apex_prefetch_route, apex_gate_topk and the apex_moe_ffn entry points only launch
 *    kernels on the given stream (no allocation, memory set, copy or synchronisation),
 *    so a caller may capture them in a HIP graph; apex_moe_ffn_noalloc's first call on
 *    a device looks up that device's scratch array and must come before the capture.
 */
#ifndef APEX_H
#define APEX_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define APEX_ABI_VERSION 4
#define APEX_MAX_EXPERTS 64
#define APEX_MAX_PAIRS 1024     /* B * k limit of apex_moe_ffn */

typedef enum {
    APEX_OK = 0,
    APEX_E_INVAL = -1,        /* invalid argument (NULL, size, alignment, range)     */
    APEX_E_UNSUPPORTED = -2,  /* valid but outside the supported sizes above        */
    APEX_E_HIP = -3,          /* a HIP runtime call failed; message names it        */
    APEX_E_CAPACITY = -4      /* workspace or cache capacity too small              */
} apex_status;

/* Prefetch-set selection rule of apex_prefetch_route. */
typedef enum {
    APEX_SEL_CUMPROB = 0,     /* smallest ranked prefix whose prefetch probabilities
                                 sum to >= tau, clamped to [k, k_max]               */
    APEX_SEL_ORDINAL_CDF = 1, /* Eq. 8-9: delta_hat = min{delta : sigmoid(theta_delta
                                 - w.x) >= tau}, m = min(k + delta_hat, k_max)      */
    APEX_SEL_STATIC = 2,      /* m = min(k + static_delta, k_max) (static over-fetch) */
    APEX_SEL_NONE = 3         /* no prefetch, the No-Prefetch baseline of Sec. V-A: m = 0
                                 and pf_idx is all -1.  apex_decode_step does not run
                                 the prefetch router at all under this policy.       */
} apex_policy;

/* Expert weight format: apex_pack_expert (bf16), apex_pack_expert_fp8 (E4M3),
 * apex_pack_expert_mxfp4 (MXFP4) or apex_pack_expert_fp32 (fp32). */
typedef enum {
    APEX_WEIGHTS_BF16 = 0,
    APEX_WEIGHTS_FP8_E4M3 = 1,
    APEX_WEIGHTS_MXFP4 = 2,
    APEX_WEIGHTS_FP32 = 3
} apex_weights;

/* Execution mode of apex_gate_topk (Sec. IV-E). */
typedef enum {
    APEX_MODE_EXACT = 0,      /* correctness-preserving: executed set = K_r          */
    APEX_MODE_STALL_FREE = 1  /* stall-free: top-k of the available experts (Alg. 1) */
} apex_mode;

int apex_abi_version(void);
const char *apex_last_error(void);

/*
 * Prefetch stage (Sec. IV-A step 1; Sec. IV-B Eq. 1; Sec. IV-C Eq. 8-9; Sec. IV-D).
 * For each token b: z = W_pf h_pre[b] (+ b_pf), q_p = softmax(z), the ranked list E
 * (descending z, lower expert id first on equal logits) and the prefetch set
 * K_p = first m entries of E, m chosen by `policy`:
 *   CUMPROB     first m with q_p(e_1) + ... + q_p(e_m) >= tau (m = E if none), then
 *               clamped to [k, k_max];
 *   ORDINAL_CDF x = q_p in ranked (descending) order, s = cdf_w . x; delta_hat = the
 *               first delta in 0..E-k with cdf_theta[delta] - s >= ln(tau/(1-tau))
 *               (E-k if none); m = min(k + delta_hat, k_max);
 *   STATIC      m = min(k + static_delta, k_max).
 * Arithmetic in fp32 (bf16 weights widened exactly).
 *   h_pre      device fp32 [B, d]
 *   w_pf       device bf16 [E, d]
 *   b_pf       device fp32 [E] or NULL (no bias)
 *   tau        coverage target in [0, 1] (CUMPROB, ORDINAL_CDF)
 *   static_delta >= 0 (STATIC)
 *   cdf_w      device fp32 [E], cdf_theta device fp32 [E-k+1] (ORDINAL_CDF only; may
 *              be NULL otherwise)
 *   pf_idx     device int32 [B, k_max] out: K_p in ranked order, -1 after position m
 *   pf_count   device int32 [B] out: m
 *   pf_prob    device fp32 [B, E] out, or NULL: q_p
 */
apex_status apex_prefetch_route(const float *h_pre, const uint16_t *w_pf, const float *b_pf,
                                int B, int d, int E, int k, int k_max,
                                int policy, float tau, int static_delta,
                                const float *cdf_w, const float *cdf_theta,
                                int32_t *pf_idx, int32_t *pf_count, float *pf_prob,
                                hipStream_t stream);

/*
 * Execution stage router (Sec. III-A; Sec. IV-E and Algorithm 1).
 * For each token b: z = W_g h_post[b] (+ b_g), alpha = softmax(z),
 * K_r = the k experts of largest z (lower id first on equal logits), and the executed
 * set K~: K_r in EXACT mode; in STALL_FREE mode the k available experts of largest z,
 * which is the set Algorithm 1 builds (routed experts that are available, topped up
 * with the highest-weight available substitutes).  Gates are alpha renormalised over
 * the set they belong to, so each row sums to 1.  If fewer than k experts are
 * available, all of them are executed and the remaining positions hold -1 / 0.
 * Arithmetic in fp32.
 *   h_post        device fp32 [B, d]
 *   w_g           device bf16 [E, d];  b_g device fp32 [E] or NULL
 *   mode          apex_mode
 *   avail         device uint8 (STALL_FREE only; may be NULL in EXACT mode): expert e
 *                 is available to token b iff avail[b * avail_stride + e] != 0
 *   avail_stride  0 (one mask shared by the batch) or >= E (one mask per token)
 *   route_idx     device int32 [B, k] out: K_r in descending-logit order
 *   route_gate    device fp32 [B, k] out: alpha renormalised over K_r
 *   exec_idx      device int32 [B, k] out: K~ in descending-logit order (-1 padded)
 *   exec_gate     device fp32 [B, k] out: alpha renormalised over K~ (0 padded)
 *   gate_prob     device fp32 [B, E] out, or NULL: alpha
 */
apex_status apex_gate_topk(const float *h_post, const uint16_t *w_g, const float *b_g,
                           int B, int d, int E, int k, int mode,
                           const uint8_t *avail, int avail_stride,
                           int32_t *route_idx, float *route_gate,
                           int32_t *exec_idx, float *exec_gate,
                           float *gate_prob, hipStream_t stream);

/*
 * Expert slot layout.  One expert occupies apex_expert_bytes(d, I) = 6 d I bytes:
 * rows i = 0..I-1 of [W1[i, 0:d] | W3[i, 0:d]] (2 d bf16 each), then W2 [d, I]
 * row-major.  apex_pack_expert writes that layout (host memory to host memory), so
 * one expert moves between host and HBM as one contiguous copy.
 */
size_t apex_expert_bytes(int d, int I);
apex_status apex_pack_expert(const uint16_t *w1, const uint16_t *w3, const uint16_t *w2,
                             int d, int I, uint16_t *out);

/*
 * Experts with 8-bit weights (the precision study of Sec. V-G: smaller experts move
 * fewer bytes over the host link and out of HBM).  Weights are OCP E4M3 codes (1 sign,
 * 4 exponent bits with bias 7, 3 mantissa bits; no infinities; largest value 448) with
 * one fp32 scale per output row: row r of W1, W3 or W2 is s_r * q, where
 * s_r = fp32(max |W[r, :]| / 448) and q rounds W[r, :] / s_r to the nearest code (ties
 * to the even code, sign bit for negative values); an all-zero row has s_r = 0.
 * apex_expert_bytes_fp8(d, I) = 3 d I + 4 (2 I + d) bytes:
 *   rows i = 0..I-1 of [W1[i, 0:d] codes | W3[i, 0:d] codes], then W2 codes [d, I]
 *   row-major, then the fp32 scales of W1's I rows, W3's I rows and W2's d rows.
 * apex_pack_expert_fp8 quantises bf16 experts (w1, w3 [I, d], w2 [d, I]) into that
 * layout (host memory to host memory); d and I must be multiples of 8.
 */
size_t apex_expert_bytes_fp8(int d, int I);
apex_status apex_pack_expert_fp8(const uint16_t *w1, const uint16_t *w3, const uint16_t *w2,
                                 int d, int I, void *out);

/*
 * Experts with 4-bit weights (the precision study of Sec. V-G), in the OCP MXFP4 form:
 * FP4 E2M1 codes (1 sign, 2 exponent bits with bias 1, 1 mantissa bit: magnitudes 0,
 * 0.5, 1, 1.5, 2, 3, 4, 6), two per byte with element 2j in the low nibble of byte j,
 * and one power-of-two scale 2^X per block of 32 consecutive values of a row (along the
 * reduction dimension: d for W1 and W3, I for W2), stored as the byte X + 127.  For each
 * block X = floor(log2 of its largest magnitude) - 2 and the codes round v / 2^X to the
 * nearest E2M1 value (ties to the even code, magnitudes above 6 clamped to 6, sign bit
 * for negative values); a block of zeros has X = -127 and codes 0.  The weights are
 * 2^X * q exactly.
 * apex_expert_bytes_mxfp4(d, I) = 3 d I / 2 + 3 d I / 32 bytes:
 *   rows i = 0..I-1 of [W1[i, 0:d] codes | W3[i, 0:d] codes] (d/2 bytes each), then W2
 *   codes [d, I/2 bytes] row-major, then the scale bytes of W1 [I, d/32], W3 [I, d/32]
 *   and W2 [d, I/32].
 * apex_pack_expert_mxfp4 quantises bf16 experts (w1, w3 [I, d], w2 [d, I]) into that
 * layout (host memory to host memory); d and I must be multiples of 32.
 */
size_t apex_expert_bytes_mxfp4(int d, int I);
apex_status apex_pack_expert_mxfp4(const uint16_t *w1, const uint16_t *w3, const uint16_t *w2,
                                   int d, int I, void *out);

/*
 * Experts with 32-bit weights (the widest point of the precision study of Sec. V-G):
 * fp32 copies of the bf16 experts, twice their bytes over the host link and out of HBM.
 * apex_expert_bytes_fp32(d, I) = 12 d I bytes:
 *   rows i = 0..I-1 of [W1[i, 0:d] | W3[i, 0:d]] (fp32), then W2 [d, I] fp32 row-major.
 * apex_pack_expert_fp32 widens bf16 experts (w1, w3 [I, d], w2 [d, I]) into that layout
 * exactly (host memory to host memory); d and I must be multiples of 4.
 */
size_t apex_expert_bytes_fp32(int d, int I);
apex_status apex_pack_expert_fp32(const uint16_t *w1, const uint16_t *w3, const uint16_t *w2,
                                  int d, int I, void *out);

/*
 * Gated SwiGLU experts (Sec. III-A weighted sum; Sec. IV-E aggregation with the
 * original router weights).  For every token b and position j with e = exec_idx[b, j]
 * in [0, E) and s = slot_of_expert[e] in [0, n_slots):
 *   y[b] (+)= exec_gate[b, j] * W2_e (silu(W1_e x[b]) * (W3_e x[b])),
 * silu(u) = u / (1 + exp(-u)), with W1_e, W3_e, W2_e read from slot s of `slots`.
 * Pairs whose expert has no slot are left out of this pass, which is how the miss
 * correction runs the missing experts in a second pass with accumulate = 1.
 * Each expert's weights are read from HBM once per call whatever the number of
 * tokens routed to it.  Arithmetic: fp32 accumulation; at B = 1 the activations stay
 * fp32, at B >= 2 the matrix cores take x and the intermediate h rounded to bf16.
 * No atomics: the result is deterministic for given inputs.
 *   x               device fp32 [B, d]
 *   exec_idx        device int32 [B, k];  exec_gate device fp32 [B, k]
 *   slot_of_expert  device int32 [E]: slot index or -1
 *   slots           device bf16 slot pool, slot s at byte offset s * apex_expert_bytes
 *   y               device fp32 [B, d] out: overwritten (accumulate = 0) or added to
 *                   (accumulate = 1); rows of tokens with no executed expert in this
 *                   pass become 0 (accumulate = 0) or stay unchanged
 *   workspace       device, >= apex_moe_ffn_workspace_bytes(B, d, I, k) bytes; contents
 *                   on entry are ignored; must not be shared by calls that may overlap
 * Requires B * k <= APEX_MAX_PAIRS.
 */
size_t apex_moe_ffn_workspace_bytes(int B, int d, int I, int k);
apex_status apex_moe_ffn(const float *x, int B, int d, int I, int E, int k,
                         const int32_t *exec_idx, const float *exec_gate,
                         const int32_t *slot_of_expert, const uint16_t *slots, int n_slots,
                         float *y, int accumulate, void *workspace, size_t workspace_bytes,
                         hipStream_t stream);

/*
 * apex_moe_ffn over experts packed by apex_pack_expert_fp8: slot s starts at byte
 * s * apex_expert_bytes_fp8(d, I) of `slots` (16-byte aligned).  The same sum, with
 * every weight taken as s_r * q exactly; the row scales multiply the fp32 dot products.
 * Same arguments, workspace size (apex_moe_ffn_workspace_bytes) and error behaviour.
 */
apex_status apex_moe_ffn_fp8(const float *x, int B, int d, int I, int E, int k,
                             const int32_t *exec_idx, const float *exec_gate,
                             const int32_t *slot_of_expert, const void *slots, int n_slots,
                             float *y, int accumulate, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

/*
 * apex_moe_ffn over experts packed by apex_pack_expert_mxfp4: slot s starts at byte
 * s * apex_expert_bytes_mxfp4(d, I) of `slots` (16-byte aligned); d and I multiples of
 * 32.  The same sum with every weight taken as 2^X * q exactly (the block scales are
 * applied as the codes are converted).  Same arguments, workspace size
 * (apex_moe_ffn_workspace_bytes) and error behaviour.
 */
apex_status apex_moe_ffn_mxfp4(const float *x, int B, int d, int I, int E, int k,
                               const int32_t *exec_idx, const float *exec_gate,
                               const int32_t *slot_of_expert, const void *slots, int n_slots,
                               float *y, int accumulate, void *workspace,
                               size_t workspace_bytes, hipStream_t stream);

/*
 * apex_moe_ffn over experts packed by apex_pack_expert_fp32: slot s starts at byte
 * s * apex_expert_bytes_fp32(d, I) of `slots` (16-byte aligned); d and I multiples of 4.
 * The same sum over fp32 weights.  Batch 1 only: B >= 2 returns APEX_E_UNSUPPORTED
 * before anything is enqueued (the matrix-core path multiplies bf16 operands, which
 * would drop the format's width).  Same arguments, workspace size
 * (apex_moe_ffn_workspace_bytes) and other errors as apex_moe_ffn.
 */
apex_status apex_moe_ffn_fp32(const float *x, int B, int d, int I, int E, int k,
                              const int32_t *exec_idx, const float *exec_gate,
                              const int32_t *slot_of_expert, const void *slots, int n_slots,
                              float *y, int accumulate, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/*
 * apex_moe_ffn without a workspace argument, for callers that cannot allocate device
 * memory: code being captured into a graph, tight serving loops, harnesses that forbid
 * allocation.  Same computation, arguments and error behaviour as apex_moe_ffn,
 * apex_moe_ffn_fp8, apex_moe_ffn_mxfp4 or apex_moe_ffn_fp32, chosen by `weights`
 * (apex_weights), with the
 * workspace taken from a fixed device array of APEX_NOALLOC_WORKSPACE_BYTES bytes that
 * the library holds on each GPU it runs on, from the first call on that GPU until the
 * process ends.  The call allocates and frees nothing.
 *   weights  APEX_WEIGHTS_BF16, APEX_WEIGHTS_FP8_E4M3, APEX_WEIGHTS_MXFP4 or
 *            APEX_WEIGHTS_FP32: the layout of `slots` (apex_pack_expert, _fp8, _mxfp4
 *            or _fp32)
 * Errors, before anything is enqueued: APEX_E_CAPACITY when
 * apex_moe_ffn_workspace_bytes(B, d, I, k) exceeds APEX_NOALLOC_WORKSPACE_BYTES (every
 * workload shape here needs at most 34 MiB); the errors of apex_moe_ffn otherwise.
 * Every call on one GPU uses that GPU's one array: calls that may overlap on one GPU
 * (on different streams, or from different host threads) race, and the caller must
 * order them.  The array's contents between calls are not meaningful; nothing in it
 * has to start at zero.
 */
#define APEX_NOALLOC_WORKSPACE_BYTES (64u << 20)
apex_status apex_moe_ffn_noalloc(const float *x, int B, int d, int I, int E, int k,
                                 const int32_t *exec_idx, const float *exec_gate,
                                 const int32_t *slot_of_expert, const void *slots, int n_slots,
                                 int weights, float *y, int accumulate, hipStream_t stream);

/*
 * The launch plan apex_moe_ffn (weights = APEX_WEIGHTS_BF16), apex_moe_ffn_fp8 and
 * apex_moe_ffn_mxfp4 take for B >= 2 tokens with E experts of which n_slots have a slot
 * (host only; no GPU work): plan[0] = 16-token tiles per pass (1, 2 or 4), plan[1] = K
 * splits of the gate/up projection, plan[2] = K splits of the down projection (1 to 4
 * each; splits of one projection are added in a fixed order, so the result depends on
 * the plan but not on timing).  B < 2 (the batch-1 kernels) gives {0, 0, 0}.
 *   plan   host int32 [3] out
 * Errors: APEX_E_INVAL for a NULL plan, an unknown weights value or sizes out of range;
 * APEX_E_UNSUPPORTED for APEX_WEIGHTS_FP32 with B >= 2 (batch 1 only).
 */
apex_status apex_moe_ffn_plan(int B, int d, int I, int E, int k, int n_slots, int weights,
                              int32_t *plan);

/*
 * Decode attention of one layer: the block that runs between the prefetch router and
 * the gate, and whose duration the expert copies overlap (Sec. IV-A; Eq. 12).  The
 * paper does not specify the block; this is grouped-query attention with H query
 * heads, G key/value heads and head size hd (64 or 128; H a multiple of G with
 * H / G in {1, 2, 3, 4, 8}).  For every token b:
 *   [q; k; v] = W_qkv h[b]            (rows: H query heads, G key heads, G value heads,
 *                                      hd rows each; W_qkv bf16 [(H + 2G) hd, d])
 *   k and v are rounded to bf16 and written to position pos of the caches;
 *   a_i = sum_{j <= pos} softmax_j(q_i . K_g[j] / sqrt(hd)) V_g[j],  g = i / (H / G);
 *   o[b] = W_o [a_0; ...; a_{H-1}]    (W_o bf16 [d, H hd]).
 * fp32 arithmetic, deterministic.
 *   h          device fp32 [B, d]
 *   k_cache, v_cache  device bf16 [B, G, ctx_max, hd]: positions 0..pos-1 are read,
 *              position pos is written (0 <= pos < ctx_max)
 *   o          device fp32 [B, d] out (overwritten)
 *   workspace  device, >= apex_attention_workspace_bytes(B, H, G, hd, ctx_max) bytes
 */
size_t apex_attention_workspace_bytes(int B, int H, int G, int hd, int ctx_max);
apex_status apex_attention_decode(const float *h, const uint16_t *w_qkv, const uint16_t *w_o,
                                  int B, int d, int H, int G, int hd, uint16_t *k_cache,
                                  uint16_t *v_cache, int ctx_max, int pos, float *o,
                                  void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Cache plan of one layer for one decode step (pure host function, no HIP calls).
 * The paper keeps a per-layer buffer that receives the prefetched set (Sec. V-C);
 * here each layer owns C persistent HBM slots.  Rule:
 *   P = union of the tokens' prefetched sets; an expert's count is the number of
 *   tokens whose set holds it, its best rank the smallest position it takes in them;
 *   target T = P if |P| <= C, else the first C of P by (count desc, best rank asc,
 *   id asc).  Experts of T already resident stay; each other expert of T, in that
 *   order, goes to the next free slot: empty slots (ascending) first, then slots of
 *   residents outside T by (last_used asc, id asc).  last_used[e] = step for e in T.
 *   pf_idx, pf_count   host [B, k_max], [B] (as written by apex_prefetch_route)
 *   expert_of_slot     host int32 [C] in/out (-1 = empty slot)
 *   last_used          host int64 [E] in/out (-1 = never)
 *   copy_expert, copy_slot  host int32 [C] out: the copies in issue order
 *   n_copies           host out
 */
apex_status apex_plan_residency(int E, int C, const int32_t *pf_idx, const int32_t *pf_count,
                                int B, int k_max, int64_t step,
                                int32_t *expert_of_slot, int64_t *last_used,
                                int32_t *copy_expert, int32_t *copy_slot, int *n_copies);

/*
 * Prefetch of one layer (Sec. IV-A: asynchronous transfers for K_p issued while
 * attention runs; Sec. V-B prefetch-overlap bound, Eq. 12).
 * Runs apex_plan_residency on the host copy of the route output, then:
 *   side:    wait readers_done (if not NULL and not yet complete); one copy-kernel
 *            launch that moves every planned expert, host_experts[e] -> slots[s]
 *            (32 workgroups per expert, reading the pinned copies over PCIe);
 *            record `ready` (if not NULL);
 *   compute: write the new table to slot_of_expert_dev[E] and, if not NULL, the
 *            resident mask to avail_dev[E] (1 = resident).
 * The caller must make the expert FFN wait for `ready` (apex_stream_wait_event)
 * before it reads the slots (when n_copied is 0 the slots are unchanged and that wait
 * may be left out), and record readers_done on the compute stream after the
 * last kernel that reads this layer's slots.  Both events may be NULL when `side` is
 * the stream that runs the readers: stream order then keeps copies and readers apart.  The host call returns once everything
 * is enqueued.
 *   expert_bytes      a positive multiple of 16, below 64 GiB
 *   host_experts      pinned [E][expert_bytes] bytes (apex_pack_expert layout),
 *                     16-byte aligned; memory the device cannot read (pageable, or a
 *                     range whose last byte is not in pinned memory) is refused with
 *                     APEX_E_INVAL before anything changes
 *   slots             device [C][expert_bytes/2]
 *   pf_idx, pf_count  host (pinned or pageable) copies of apex_prefetch_route's output;
 *                     they must be complete when the call is made
 *   expert_of_slot, last_used  host tables as in apex_plan_residency (in/out)
 *   copied_experts    host int32 [C] out or NULL; n_copied host out or NULL
 */
apex_status apex_expert_prefetch(const uint16_t *host_experts, uint16_t *slots,
                                 int E, int C, size_t expert_bytes,
                                 const int32_t *pf_idx, const int32_t *pf_count,
                                 int B, int k_max, int64_t step,
                                 int32_t *expert_of_slot, int64_t *last_used,
                                 int32_t *slot_of_expert_dev, uint8_t *avail_dev,
                                 hipStream_t side, hipStream_t compute,
                                 hipEvent_t readers_done, hipEvent_t ready,
                                 int32_t *copied_experts, int *n_copied);

/*
 * Miss correction of the correctness-preserving mode (Sec. IV-E, asynchronous miss
 * correction): the routed experts of the batch that are not resident,
 *   M = union_b K_r[b] minus {expert_of_slot[s]},
 * in ascending id order, are copied host -> scratch slot i (i = 0..|M|-1) on `side`
 * after waiting for scratch_free (if not NULL), by one launch of the prefetch's copy
 * kernel, then `ready` (if not NULL) is recorded on side.  host_experts follows the
 * prefetch's rules.
 * On `compute`, miss_table_dev[E] is written with miss_table[e] = i for the i-th
 * missing expert and -1 otherwise, so a second apex_moe_ffn pass over the scratch
 * pool with accumulate = 1 adds exactly the missing experts.  If M is empty nothing is
 * enqueued (no second pass is needed; the table and `ready` are left as they were).
 * Returns APEX_E_CAPACITY (enqueueing nothing) if |M| > n_scratch.  A wait on an event
 * that has already completed is skipped (it would be a no-op).
 *   route_idx        host int32 [B, k] (apex_gate_topk route output, complete)
 *   expert_of_slot   host int32 [C] (resident set after this step's prefetch)
 *   missing          host int32 [min(B*k, E)] out or NULL;  n_missing host out
 */
apex_status apex_expert_fetch_misses(const uint16_t *host_experts, uint16_t *scratch,
                                     int n_scratch, int E, int C, size_t expert_bytes,
                                     const int32_t *route_idx, int B, int k,
                                     const int32_t *expert_of_slot,
                                     int32_t *miss_table_dev,
                                     hipStream_t side, hipStream_t compute,
                                     hipEvent_t scratch_free, hipEvent_t ready,
                                     int32_t *missing, int *n_missing);

/*
 * Decode driver: one decode step through every MoE layer, in native code, composed of
 * the entry points above in the order of the paper's two-stage runtime (Sec. IV-A;
 * Sec. IV-D "Runtime Operation"; Sec. IV-E).  Per layer:
 *   compute: apex_prefetch_route (K_p written to pinned host memory);
 *   side:    after the router: attention-window stand-in (apex_spin_us, t_attn_us);
 *   host:    poll until the route is done; apex_expert_prefetch (the copies on compute,
 *            the slot table on side);
 *   side:    apex_gate_topk; the shared experts, if any (apex_moe_ffn over the layer's
 *            shared pool, every token, weight 1);
 *   compute: after the gate (and the shared experts): apex_moe_ffn pass 1 (added to the
 *            shared experts' output);
 *   EXACT:   host waits for the gate; apex_expert_fetch_misses copies the missing
 *            experts on side while pass 1 runs, and, if any expert was missing, pass 2
 *            (accumulate) runs on compute after an event recorded behind that copy.
 * The copies, the FFN and the next layer's router follow each other on the compute
 * stream with no event between them, so a layer's router starts after the previous
 * layer's FFN, as in a model where each layer feeds the next, and the copies of a layer
 * start after every earlier read of its slots.  A layer-step that copies nothing runs
 * the window, the gate and the shared experts on the compute stream instead.  Work still
 * running on the side stream when the step returns is waited for by the compute stream,
 * so synchronizing the compute stream covers the step.
 *
 * Shared experts (n_shared > 0; DeepSeek-style, Sec. V-A) run for every token with
 * weight 1 and stay out of the adaptive decision: they live in a resident pool per layer
 * (shared_slots) and never enter the cache, the prefetch or the miss path.  They run
 * on the side stream while the routed experts' copies are still in flight.
 *
 * With attn_heads > 0 the attention window is the layer's real decode attention
 * (apex_attention_decode on h_pre, writing position attn_ctx of its caches) instead of
 * the spin; its output goes to attn_out and does not feed the MoE input (layers draw
 * their own hidden states).
 *
 * apex_decode_create copies the configuration and the per-layer descriptors (the
 * buffers themselves stay caller-owned and must outlive the driver; every layer's
 * host_experts must be pinned, as for apex_expert_prefetch) and allocates the
 * driver's own events, pinned staging, attention workspace and shared-expert lists
 * (setup time, not the hot path).  `workspace` must hold
 * apex_moe_ffn_workspace_bytes for both the routed (I, k) and the shared (I_shared,
 * n_shared) calls.
 */
typedef struct {
    int L, B, d, E, k, I, C, k_max;
    int policy;            /* apex_policy */
    float tau;
    int static_delta;
    int mode;              /* apex_mode */
    double t_attn_us;      /* attention-window stand-in per layer, >= 0 */
    int n_scratch;         /* miss-scratch slots (EXACT), >= min(E, B*k) recommended */
    int weights;           /* apex_weights: layout of host_experts, slots and scratch */
                           /*   (APEX_WEIGHTS_FP32 needs B = 1)                        */
    int attn_heads;        /* > 0: the attention window is apex_attention_decode with this */
    int attn_kv_heads;     /*   many query / key-value heads over attn_ctx cached positions */
    int attn_ctx;          /*   (caches hold attn_ctx + 1 positions); 0: spin t_attn_us  */
    int n_shared;          /* shared experts per layer, 0..APEX_MAX_EXPERTS (0: none)     */
    int I_shared;          /*   their intermediate size (same rules as I)                 */
} apex_decode_config;

typedef struct {
    const uint16_t *w_pf, *w_g;            /* device bf16 [E, d] */
    const float *b_pf, *b_g;               /* device fp32 [E] or NULL */
    const float *cdf_w, *cdf_theta;        /* device (ORDINAL_CDF only) or NULL */
    const uint16_t *host_experts;          /* pinned, [E] experts in the layout of cfg.weights */
    uint16_t *slots;                       /* device, [C] experts */
    int32_t *slot_of_expert_dev;           /* device int32 [E]: equal to the host tables at
                                              creation; the driver rewrites it (and
                                              avail_dev) whenever a layer-step copies */
    uint8_t *avail_dev;                    /* device uint8 [E] resident mask */
    int32_t *expert_of_slot;               /* host int32 [C] in/out */
    int64_t *last_used;                    /* host int64 [E] in/out */
    const uint16_t *w_qkv, *w_o;           /* attention window only: device bf16 weights, */
    uint16_t *k_cache, *v_cache;           /*   caches [B, G, attn_ctx + 1, hd] and the    */
    float *attn_out;                       /*   block's output [B, d]; NULL otherwise      */
    const void *shared_slots;              /* n_shared > 0: device, [n_shared] experts of  */
                                           /*   intermediate I_shared, cfg.weights layout  */
} apex_decode_layer;

typedef struct {   /* counters the driver adds to at every layer-step */
    double overlap_sum;        /* sum over tokens of |K_r & K_p| / k (Sec. V-C overlap) */
    double hit_sum;            /* sum over tokens of |K_r & resident| / k */
    int64_t coverage_count;    /* tokens with K_r subset of K_p (Eq. 2) */
    int64_t delta_hat_sum;     /* sum of max(m - k, 0): delta_hat of Eq. 9 (0 when nothing
                                  is prefetched, APEX_SEL_NONE) */
    int64_t tokens, layer_steps, copies, misses;
} apex_decode_stats;

typedef struct {   /* optional per-step record, host arrays (caller-owned), any may be NULL */
    int32_t *pf_idx;       /* [L][B][k_max] */
    int32_t *pf_count;     /* [L][B] */
    int32_t *route_idx;    /* [L][B][k] */
    float *route_gate;     /* [L][B][k] */
    int32_t *exec_idx;     /* [L][B][k] */
    float *exec_gate;      /* [L][B][k] */
    int32_t *resident;     /* [L][C] expert_of_slot after the step's prefetch */
    int32_t *n_copies;     /* [L] */
    int32_t *missing;      /* [L][E] missing routed experts (EXACT) */
    int32_t *n_missing;    /* [L] */
} apex_decode_record;

typedef struct apex_decode apex_decode;

apex_status apex_decode_create(apex_decode **out, const apex_decode_config *cfg,
                               const apex_decode_layer *layers, uint16_t *scratch,
                               int32_t *miss_table_dev, int32_t *exec_idx_dev,
                               float *exec_gate_dev, void *workspace, size_t workspace_bytes,
                               hipStream_t compute, hipStream_t side);
/* One decode step.  h_pre, h_post, y: host arrays of L device pointers to [B, d] fp32.
 * Returns when everything is enqueued (with `record`, after the step has completed and
 * the record is filled).  stats (may be NULL) is added to; a layer-step's counters are
 * added once its gate has finished, by this call, a later one or apex_decode_finish.
 * A layer whose every expert is resident (C = E, no slot empty) is enqueued without
 * waiting for its router: its cache plan, which then only renews last_used, runs when
 * the layer-step is counted, so last_used is current after apex_decode_finish, or
 * after a step with `record` (which always waits). */
apex_status apex_decode_step(apex_decode *dec, int64_t step, const float *const *h_pre,
                             const float *const *h_post, float *const *y,
                             apex_decode_stats *stats, apex_decode_record *record);
/* Waits for all enqueued work and folds the statistics of the last layers into stats. */
apex_status apex_decode_finish(apex_decode *dec, apex_decode_stats *stats);
apex_status apex_decode_destroy(apex_decode *dec);

/*
 * Attention-window stand-in: one wavefront that spins for `us` microseconds of the
 * device's constant-rate clock on `stream` (0 <= us <= 1e6), then exits.
 */
apex_status apex_spin_us(double us, hipStream_t stream);

/* Thin event and stream helpers for callers without their own HIP bindings. */
apex_status apex_event_create(hipEvent_t *event, int timing);
apex_status apex_event_destroy(hipEvent_t event);
apex_status apex_event_record(hipEvent_t event, hipStream_t stream);
apex_status apex_event_synchronize(hipEvent_t event);
apex_status apex_event_elapsed_ms(hipEvent_t start, hipEvent_t stop, float *ms);
apex_status apex_stream_wait_event(hipStream_t stream, hipEvent_t event);
apex_status apex_stream_synchronize(hipStream_t stream);

/* Copy `bytes` (multiple of 16) from device src to device dst with a streaming
 * vector-load/store kernel; used to calibrate memory counters and bandwidth. */
apex_status apex_copy_kernel(void *dst, const void *src, size_t bytes, hipStream_t stream);

/* Read `bytes` (multiple of 16) of device memory with a streaming vector-load kernel
 * (four 16-byte loads in flight per thread, 256 threads per workgroup, up to 1024
 * workgroups) that writes only one word per workgroup to `sink`: the read-only rate any
 * kernel can reach at that size, the floor against which the expert FFN is measured.
 * Its loads are non-temporal, as the expert FFN's weight loads are.
 * sink: device uint32 [apex_read_kernel_sink_words(bytes)]. */
size_t apex_read_kernel_sink_words(size_t bytes);
apex_status apex_read_kernel(const void *src, size_t bytes, uint32_t *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* APEX_H */
