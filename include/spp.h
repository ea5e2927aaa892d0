/*
 * spp.h -- C ABI of the MI355X (gfx950) SpecPrefetch offloaded-MoE decode hot path.
 *
 * One decode step of an offloaded MoE layer, as the paper's problem statement
 * and method sections describe it:
 *   native router (softmax, top-K) -> layer-specific low-rank adapter scoring
 *   the next layer's expert priorities -> window-aware prefetch budget ->
 *   routed-expert SwiGLU FFN over an HBM expert-slot cache, while budgeted
 *   host-to-device copies of the next layer's experts overlap with it.
 *
 * Conventions for every call:
 *  - Plain pointers only.  "dev" pointers are device (HBM) addresses on the
 *    device that was current at spp_create; "host" pointers are ordinary host
 *    memory unless stated.  The caller owns every pointer it passes and keeps
 *    it valid for as long as the context may use it (weights and host stores:
 *    until spp_destroy).  The library owns its slot pools, events, copy streams
 *    and scratch.
 *  - Every call returns an spp_status and never throws.  On SPP_EINVAL no
 *    state has changed.  HIP runtime failures return SPP_EHIP.  The message of
 *    the last non-OK status of the calling thread is spp_last_error().
 *  - Device work is enqueued on the compute stream given to spp_create; the
 *    library's two copy streams run host-to-device expert copies beside it
 *    (loads in two halves, one per stream, so that one stream's per-copy
 *    start-up overlaps the other's transfer; prefetches of the default copy
 *    engine whole, in issue order, on the first stream).  Calls
 *    with host outputs return once those outputs are valid.
 *  - Layouts are row-major.  dtype SPP_DTYPE_F32 stores weights and hidden
 *    states as fp32, SPP_DTYPE_BF16 as bf16 (bit patterns, 2 bytes); router
 *    logits, gates, priorities and the router input are always fp32.
 *
 * Expert blob ("blob": one routed or shared expert, W_gate and W_up [I][D],
 * W_down [D][I], 3*I*D elements) in one of two layouts, fixed by the model
 * shape (spp_blob_layout); spp_pack_expert writes either on the host.
 *  SPP_LAYOUT_UNITS (batch-1 contexts): I units of 3*D elements, unit i =
 *    [gate row i, up row i, down column i]:
 *      blob[(3i+0)D + d] = W_gate[i][d],  blob[(3i+1)D + d] = W_up[i][d],
 *      blob[(3i+2)D + d] = W_down[d][i].
 *  SPP_LAYOUT_TILED (bf16 contexts with max_batch > 1, D % 256 == 0 and
 *    I % 16 == 0): with nb = D/256, first the gate/up part in pieces of 8
 *    elements, piece (((t*nb + b)*2 + w)*8 + j)*64 + l (w = 0 gate, 1 up;
 *    t < I/16, b < nb, j < 8, l < 64) holding
 *      W_w[16t + l%16][256b + 32j + 8(l/16) + e], e = 0..7,
 *    then, from element 2*I*D, the down part in runs of 256 elements, run
 *    (s*I + i) (s < nb, i < I) holding W_down[256s + c][i], c = 0..255.
 *  SPP_LAYOUT_Q4_UNITS (expert_codec SPP_CODEC_Q4: dtype bf16, max_batch 1,
 *    D % 256 == 0): 4-bit codes q (0..15) in blocks of 32 elements along D,
 *    one fp16 scale per block, value scale * (q - 8).  I units of
 *    3*D/2 + 3*(D/32)*2 bytes, unit i =
 *      [gate codes | up codes | down codes | gate scales | up scales | down scales],
 *    each code run D/2 bytes (byte j: element 2j in the low nibble, 2j+1 in
 *    the high nibble; the down run holds column i of W_down, element d =
 *    W_down[d][i]), each scale run D/32 fp16 values (scale b covers elements
 *    32b..32b+31 of the run).  The device FFN forms the gate/up products of
 *    these experts exactly in integers, with x of each 32-element block in
 *    fixed point against the block's largest |x| (19 significant bits: an
 *    error of at most 2^-18 of that element), and the down products in fp32.
 * Blobs are placed at a stride of spp_blob_stride(desc) bytes (the blob size
 * rounded up to 4096); the padding is zero.
 */
#ifndef SPP_H
#define SPP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct spp_ctx spp_ctx;
typedef struct spp_slot_policy spp_slot_policy;

typedef enum {
  SPP_OK = 0,
  SPP_EINVAL = -1,  /* bad argument; nothing changed */
  SPP_ENOMEM = -2,  /* device or pinned allocation failed */
  SPP_EHIP = -3,    /* a HIP runtime call failed; see spp_last_error() */
  SPP_ESTATE = -4   /* call not valid in the current state (e.g. layer not bound) */
} spp_status;

enum { SPP_DTYPE_F32 = 0, SPP_DTYPE_BF16 = 1 };
enum { SPP_LAYOUT_UNITS = 0, SPP_LAYOUT_TILED = 1, SPP_LAYOUT_Q4_UNITS = 2 };
enum { SPP_CODEC_PLAIN = 0, SPP_CODEC_Q4 = 1 };
enum { SPP_PREFETCH_ADAPTER = 0, SPP_PREFETCH_PREV_TOKEN = 1 };
enum { SPP_COPY_KERNEL = 0, SPP_COPY_SDMA = 1, SPP_COPY_SPLIT = 2 };

/* Model shape.  Notation of the paper's problem formulation: L MoE layers,
 * n routed experts per layer, top-K routing, router input size D, adapter
 * rank r.  I: SwiGLU intermediate size of an expert; n_shared: always-resident
 * shared experts per layer (weight 1); S: HBM expert slots per layer;
 * max_batch: largest batch B passed to any call (above 1, D must be a
 * multiple of 16); has_proj: 1 if each layer starts with the dense D x D
 * stand-in projection u = h + P rms(h). */
typedef struct {
  int32_t L, D, n, K, I, r, n_shared, S, max_batch, dtype, has_proj;
  float rms_eps;
  int32_t expert_codec;  /* SPP_CODEC_PLAIN: experts in dtype; SPP_CODEC_Q4: 4-bit (see the blob layouts) */
} spp_model_desc;

/* Counters of one moe_layer_forward call. */
typedef struct {
  int32_t hits;           /* routed experts of the batch demand already available (resident or in flight) */
  int32_t misses;         /* on-demand loads issued for this layer */
  int32_t prefetched;     /* prefetch copies issued for layer l+1 */
  int32_t prefetch_used;  /* experts prefetched for this layer that its native router selected */
  int32_t ready_on_time;  /* needed experts whose copy had completed when the FFN was enqueued */
  int32_t token_hits;     /* sum over tokens b of |T_b cap available| before the on-demand loads */
  int32_t waited;         /* needed experts the FFN waited for (loaded by this call, or a copy still in
                           * flight); ready_on_time + waited = the distinct routed experts of the batch */
  /* With spp_set_timing(ctx, 2) only (the call then returns after the layer
   * finished on the device; -1 otherwise): exposed_us = compute-stream time
   * spent on expert copies before and between the FFN rounds (on-demand copy
   * kernels and waits for copies), layer_us = the layer call's span on the
   * compute stream, from its first enqueued operation to its last. */
  float exposed_us;
  float layer_us;
} spp_layer_stats;

/* Accumulated since the last spp_reset_run_stats.  Times come from HIP events
 * on the compute stream (only when timing is enabled). */
typedef struct {
  int64_t layer_calls, hits, misses, prefetched, prefetch_used, ready_on_time, copies;
  int64_t copy_bytes, ffn_launches, window_samples;
  double router_us;   /* router+adapter kernel and result read-back */
  double exposed_us;  /* compute stream waiting on expert copies before the FFN */
  double ffn_us;      /* routed-expert FFN main kernel (kernel begin/end stamps) */
  double tail_us;     /* FFN combine/residual kernel */
  double span_us;     /* first layer start to last layer end */
  double window_us;   /* sum over layer pairs of W_l = t_exec(l+1) - t_pred(l) */
  double compute_window_us;  /* the same minus the copy stalls of both layers inside it */
  /* exposed_us split in three: on-demand copy kernels on the compute stream
   * (with the later rounds of a multi-round step) that had the host link to
   * themselves; the same for layer calls whose on-demand copies were
   * enqueued while a prefetch copy was still in flight on the link (the two
   * share it, so the load takes longer); and waits for copies on the copy
   * streams (prefetches in flight; every load when loads go by DMA).
   * exposed_us = exposed_load_us + exposed_shared_us + exposed_wait_us. */
  double exposed_load_us;
  double exposed_wait_us;
  /* ExpertRecall@M (section "Evaluation Metrics"), counted while timing is on:
   * over the tokens of every layer that a prediction targeted, the sum of
   * |T_b cap Top_M(s)| for M = K/2, K, K+2 (Top_M by s descending, lower
   * index first; M at most n); ExpertRecall@M = recall_hits[j] / (K * recall_tokens) */
  int64_t recall_tokens;
  int64_t recall_hits[3];
  /* Demand against the window (section "Introduction"), counted while timing
   * is on: adapter predictions made, and of those the ones where more than
   * M_max of Top_M(s), M = K/2, K, K+2 (at most n), were not available in
   * layer l+1 when the prediction was made */
  int64_t pred_events;
  int64_t demand_exceeds[3];
  /* the same predictions by how many of Top_M(s) were not available:
   * demand_hist[j][c] counts c missing experts (c = 16 counts 16 or more) */
  int64_t demand_hist[3][17];
  /* batch-1 layer calls whose FFN ran split (spp_set_ffn_overlap) */
  int64_t ffn_split_launches;
  /* see exposed_load_us; shared_calls counts the layer calls it covers */
  double exposed_shared_us;
  int64_t shared_calls;
  /* needed experts the FFN waited for (the layer calls' `waited`) */
  int64_t waited;
  /* prefetch copies issued per prediction (m_l, section "Window-Aware
   * Prefetch Budgeting"): prefetch_hist[m] counts the predictions (layer
   * calls that predict layer l+1, M_max >= 0, and expert_cache_issue_prefetch
   * calls) that issued m copies (m = 16 counts 16 or more) */
  int64_t prefetch_hist[17];
  /* host time of every layer call (timing on or off): from the router
   * launch's return to the routing records being seen (host_route_us: the
   * host waits for the device to reach and finish the router), and from
   * there to the FFN launch's return (host_decide_us: the statistics, slot
   * decisions, on-demand copies and FFN enqueue on the critical path) */
  double host_route_us;
  double host_decide_us;
} spp_run_stats;

/* ---------------------------------------------------------------- lifecycle */

/* Bytes between consecutive expert blobs in a host store or slot pool. */
size_t spp_blob_stride(const spp_model_desc* desc);

/* Blob layout of contexts with this shape: SPP_LAYOUT_UNITS or
 * SPP_LAYOUT_TILED (see the top of this header); -1 if desc is NULL. */
int32_t spp_blob_layout(const spp_model_desc* desc);

/* Pack one expert into its blob on the host, in the layout of
 * spp_blob_layout(desc).  gate, up: host [I][D]; down: host [D][I]; all in
 * the storage dtype; blob: host, spp_blob_stride(desc) bytes (the padding is
 * zeroed).  Host stores and shared-expert blobs must hold blobs in this
 * layout.  Errors: EINVAL for a bad desc (or one with the 4-bit codec: use
 * spp_pack_expert_q4) or a NULL pointer. */
spp_status spp_pack_expert(const spp_model_desc* desc, const void* gate, const void* up, const void* down,
                           void* blob);

/* Pack one 4-bit expert (expert_codec SPP_CODEC_Q4) into its blob on the host.
 * gate_q, up_q: host uint8 [I][D] codes 0..15; down_q: host uint8 [D][I];
 * gate_s, up_s, down_s: host fp16 bit patterns [I][D/32] (down_s[i][b] scales
 * elements 32b..32b+31 of column i).  blob: spp_blob_stride(desc) bytes.
 * Errors: EINVAL for a desc without the 4-bit codec, a code above 15 or a NULL
 * pointer (nothing written). */
spp_status spp_pack_expert_q4(const spp_model_desc* desc, const uint8_t* gate_q, const uint16_t* gate_s,
                              const uint8_t* up_q, const uint16_t* up_s, const uint8_t* down_q,
                              const uint16_t* down_s, void* blob);

/* Create a context on the current device.  hip_stream: the compute stream
 * (hipStream_t, may be NULL for the null stream).  Allocates S slots per layer
 * plus scratch; every slot starts EMPTY.  Errors: EINVAL for inconsistent
 * shapes, among them S < min(n, K*max_batch) for a context whose expert
 * layout is not SPP_LAYOUT_TILED (only the tiled batched path runs a step in
 * on-demand rounds, so elsewhere every distinct routed expert of a call must
 * fit in the slots at once), ENOMEM, EHIP. */
spp_status spp_create(const spp_model_desc* desc, void* hip_stream, spp_ctx** out);
spp_status spp_destroy(spp_ctx* ctx);

/* Bind layer l's weights.  router_w: dev [n,D]; adapter_a: dev [r,D] and
 * adapter_b: dev [n,r] (both NULL for the last layer, which has no adapter);
 * proj_w: dev [D,D] or NULL (required iff has_proj); shared_blobs: dev
 * n_shared blobs at blob stride (NULL iff n_shared == 0); host_store: the
 * offload tier, n*stride bytes of pinned host memory (hipHostMalloc or a
 * pinned torch tensor), 16-byte aligned, expert e at host_store + e*stride.  EINVAL if host_store is not pinned (it has no device-visible
 * address) or not aligned. */
spp_status spp_bind_layer(spp_ctx* ctx, int32_t l, const void* router_w, const void* adapter_a,
                          const void* adapter_b, const void* proj_w, const void* shared_blobs,
                          const void* host_store);

/* Fill slots 0..count-1 of layer l with the listed experts (synchronous
 * copies), stamp 0; the other slots become EMPTY.  count <= S, no duplicates. */
spp_status spp_set_resident(spp_ctx* ctx, int32_t l, const int32_t* experts, int32_t count);

/* ------------------------------------------------------- the four calls */

/* Section "Expert Prediction Adapter": s^{l+1}_e = sum over the B tokens of
 * softmax(B^l A^l x_b)_e.  x_dev: dev fp32 [B,D], the router inputs of layer
 * l; s_out: host fp32 [n].  Synchronous.  ESTATE if layer l has no adapter. */
spp_status adapter_predict(spp_ctx* ctx, int32_t l, const float* x_dev, int32_t B, float* s_out);

/* Section "Window-Aware Prefetch Budgeting": the maximum prefetch budget is the
 * number of whole expert transfers that fit in the profiled overlap window W,
 * M_max = clamp(floor(window_us / per_expert_cost_us), 0, n_experts).
 * window_us <= 0 gives 0.  EINVAL for a non-finite input, a cost <= 0 or
 * n_experts < 0.  Pure host arithmetic; needs no device. */
spp_status select_prefetch_budget(double window_us, double per_expert_cost_us, int32_t n_experts,
                                  int32_t* M_max_out);

/* Same section: P^{l+1} = Top_{M_max}{ s_e : e neither available nor in
 * flight in target_layer }, lowest expert index first on equal priority
 * (an expert with priority -inf is never a candidate),
 * issued as asynchronous host-to-device copies in descending priority, each
 * into a replacement slot (lowest EMPTY slot, else the least recently stamped
 * slot not filled in this step; stops early when none is left).  s_host: host
 * fp32 [n].  issued_out: host int32 [M_max] receives P in issue order; m_out:
 * |P| <= M_max.  Advances the step clock by one.  Returns without waiting for
 * the copies. */
spp_status expert_cache_issue_prefetch(spp_ctx* ctx, int32_t target_layer, const float* s_host,
                                       int32_t M_max, int32_t* issued_out, int32_t* m_out);

/* One MoE layer of one decode step (sections "Problem Formulation" through
 * "Window-Aware Prefetch Budgeting"):
 *   u = h (+ P rms(h) if has_proj); x = rms(u) (fp32, no learned scale);
 *   z = W_r x (fp32); T_b = Top_K(z_b), lowest index first on ties;
 *   g_b = softmax(z_b) renormalised over T_b;
 *   if l < L-1 and M_max >= 0: s = sum_b softmax(B A x_b);
 *   on-demand copies of every expert of the batch demand not available
 *   (replacement: lowest EMPTY slot, else the least recently stamped slot
 *   whose expert the batch does not need); every slot holding a needed
 *   expert takes the step stamp.  When the batch needs more distinct experts
 *   than S (tiled-layout contexts only), the step runs in rounds: load while a victim
 *   exists (third victim class: the lowest-index slot whose expert already
 *   ran this step), run every resident needed expert not yet run, repeat;
 *   if M_max > 0: the expert_cache_issue_prefetch selection for layer l+1
 *   with this s, in the same step (with SPP_PREFETCH_PREV_TOKEN, see
 *   spp_set_prefetch_source, s comes from the preceding step instead and no
 *   adapter runs);
 *   FFN: h_out_b = round(u_b + sum_k g_bk W_down(silu(W_gate x_b) * (W_up x_b))
 *   [+ shared experts, weight 1]), reading each expert from its HBM slot
 *   after its copy completed.
 * h_in_dev / h_out_dev: dev [B,D] in dtype (may not alias).  M_max: -1 = no
 * prediction (OFF), 0 = prediction without transfers, > 0 = budget.
 * topk_out: host int32 [B,K] or NULL; gate_out: host fp32 [B,K] or NULL;
 * stats: host or NULL.  Outputs never depend on M_max, S or the adapter.
 * Advances the step clock by one.  Returns once topk/gates are on the host;
 * h_out is complete when the compute stream reaches that point.  Errors:
 * EINVAL (bad argument) and ESTATE (layer l, or layer l+1 for a budget, not
 * bound) before any device work; a refusal after the routing (a batch demand
 * the slots cannot hold, which spp_create's slot check rules out) restores
 * the step clock and leaves slot tables, prefetch records and statistics as
 * they were. */
spp_status moe_layer_forward(spp_ctx* ctx, int32_t l, const void* h_in_dev, void* h_out_dev, int32_t B,
                             int32_t M_max, int32_t* topk_out, float* gate_out, spp_layer_stats* stats);

/* One whole decode step: moe_layer_forward for layers 0..L-1 in order, each
 * layer reading the previous one's output.  The last layer writes h_out_dev;
 * earlier layers alternate between h_out_dev and h_scratch_dev (layer l
 * writes h_out_dev when L-1-l is even).  h_in_dev, h_out_dev, h_scratch_dev:
 * dev [B,D] in dtype, pairwise distinct.  topk_out / gate_out: host [L,B,K]
 * or NULL; stats: host [L] or NULL.  Saves one host round trip per layer
 * against L separate calls.  Errors: those of moe_layer_forward; on an error
 * in layer l, layers before l have run. */
spp_status spp_decode_step(spp_ctx* ctx, const void* h_in_dev, void* h_out_dev, void* h_scratch_dev, int32_t B,
                           int32_t M_max, int32_t* topk_out, float* gate_out, spp_layer_stats* stats);

/* Message of the calling thread's last non-OK status ("" if none). */
const char* spp_last_error(void);

/* Capacity of adapter_predict_static's scratch, in floats: B * (n + r) at most. */
#define SPP_STATIC_SCRATCH_FLOATS 81920

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * adapter_predict computation, s = sum over the B tokens of
 * softmax(B^l A^l x_b), on explicit device weights and without a context.
 * Its scratch (two completion counters and B * (n + r) floats of adapter
 * hidden units and per-token distributions) is one fixed device array inside
 * the library, 256 + 4 * SPP_STATIC_SCRATCH_FLOATS bytes (328 KiB), which
 * each device the library runs on holds until the process ends; B * (n + r)
 * may not exceed SPP_STATIC_SCRATCH_FLOATS (e.g. 64 tokens with n 1024 and
 * r 256).  Allocates nothing: no hipMalloc or hipFree, no host waits.
 * adapter_a: dev [r, D], adapter_b: dev [n, r], in dtype (SPP_DTYPE_F32 or
 * SPP_DTYPE_BF16); x_dev: dev fp32 [B, D], the router inputs; s_out_dev: dev
 * fp32 [n] receives s.  adapter_a, adapter_b and x_dev 16-byte aligned.
 * Shape limits as spp_create's (D at most 4096 bf16 / 2048 fp32, D a
 * multiple of 16 when B > 1, n <= 1024, 1 <= r <= 256).  The work is
 * enqueued on hip_stream (NULL: the null stream) and the call returns
 * without waiting; s_out_dev is complete when the stream reaches that point.
 * Every call on a device shares that device's scratch, which keeps the last
 * call's contents (the counters are cleared at the start of each call):
 * calls that overlap on one device race, so a caller keeps them on one
 * stream.  Errors: EINVAL (NULL or misaligned pointer, bad shape, B * (n + r)
 * above the limit; nothing enqueued), EHIP. */
spp_status adapter_predict_static(const void* adapter_a, const void* adapter_b, int32_t dtype, int32_t D,
                                  int32_t n, int32_t r, const float* x_dev, int32_t B, float* s_out_dev,
                                  void* hip_stream);

/* ------------------------------------------------------ inspection / runs */

/* Slot table of layer l: experts_out host int32 [S] (-1 = EMPTY), stamps_out
 * host int64 [S] (either may be NULL). */
spp_status spp_get_slot_table(spp_ctx* ctx, int32_t l, int32_t* experts_out, int64_t* stamps_out);

/* Replace layer l's slot table (copies the listed experts in, synchronously).
 * Used to re-synchronise with a reference state. */
spp_status spp_set_slot_table(spp_ctx* ctx, int32_t l, const int32_t* experts, const int64_t* stamps);

/* The step clock: the stamp of the last step taken (0 after spp_create). */
spp_status spp_get_clock(spp_ctx* ctx, int64_t* tau_out);
spp_status spp_set_clock(spp_ctx* ctx, int64_t tau);

/* Transfers of the last moe_layer_forward: loads_out / pref_out host int32
 * [3*cap] as (expert, slot, evicted expert or -1) triples in issue order;
 * n_loads / n_pref receive the counts (may exceed cap: then truncated). */
spp_status spp_get_last_transfers(spp_ctx* ctx, int32_t* loads_out, int32_t* n_loads, int32_t* pref_out,
                                   int32_t* n_pref, int32_t cap);

/* Priorities s (host fp32 [n]) and router inputs x (host fp32 [B,D]) of the
 * last moe_layer_forward (s is undefined when no adapter ran). */
spp_status spp_get_last_priorities(spp_ctx* ctx, float* s_out);
spp_status spp_get_last_router_input(spp_ctx* ctx, float* x_out, int32_t B);

/* Native router logits z (host fp32 [B,n]) of the last moe_layer_forward
 * (the distillation targets of section "Training Objective").  ESTATE when
 * that call ran the adapter at B > 1 (its selection kernel reuses the logit
 * buffer) or after adapter_predict; B at most the last call's batch. */
spp_status spp_get_last_logits(spp_ctx* ctx, float* z_out, int32_t B);

/* Event timing of layer calls (adds ~6 event records per call).  enabled:
 * 0 off, 1 on (run and per-layer totals, no host waits), 2 on and every layer
 * call also fills its spp_layer_stats exposed_us / layer_us, for which it
 * waits until the layer finished on the device (this serialises host and
 * device: use 1 for throughput runs).  EINVAL outside 0..2. */
spp_status spp_set_timing(spp_ctx* ctx, int32_t enabled);
/* Per-layer totals of the timed layer calls since spp_reset_run_stats, for
 * layers 0..L-1 (host arrays of L entries, any may be NULL; L must equal the
 * context's layer count): calls_out = timed calls of layer l; exposed_us_out
 * = their exposed time (as spp_run_stats.exposed_us); latency_us_out = the
 * time from each call's start on the compute stream to the start of the next
 * timed layer call (the per-layer latency of the exposed-transfer share; a
 * run's last call has no successor and contributes only to calls_out and
 * exposed_us_out, and latency_calls_out counts the calls that did
 * contribute).  Waits for all enqueued work first. */
spp_status spp_get_layer_times(spp_ctx* ctx, int32_t L, int64_t* calls_out, double* exposed_us_out,
                               double* latency_us_out, int64_t* latency_calls_out);
/* Waits for all enqueued work, folds finished event timings into the totals. */
spp_status spp_get_run_stats(spp_ctx* ctx, spp_run_stats* out);
spp_status spp_reset_run_stats(spp_ctx* ctx);

/* Measured host-to-device cost of one expert blob on a copy stream with the
 * prefetch engine (average over reps copies from layer l's host store into
 * scratch), in us: the per-expert cost c of the prefetch budget. */
spp_status spp_profile_expert_copy(spp_ctx* ctx, int32_t l, int32_t reps, double* per_expert_us);

/* HBM read ceiling of the batch-1 FFN's access pattern (measurement, not part
 * of the hot path): the loads of one FFN launch over K expert slots -- the
 * same grid, unit order and loads as this context's sweep-order FFN kernel
 * (bf16 experts: 16-byte non-temporal row loads; 4-bit experts: the code and
 * scale loads of each block) -- without its arithmetic, timed by the
 * kernel's own begin/end stamps and averaged over `reps` launches (after two
 * untimed ones), each launch on other slots of the context's pools.  us_out:
 * average time per launch; gbs_out: K expert blobs per launch / that time.
 * Waits for all enqueued work first.  ESTATE unless the experts are bf16 or
 * 4-bit (bf16 storage) in the batch-1 unit layout; EINVAL for reps outside
 * 1..10000. */
spp_status spp_probe_read_ceiling(spp_ctx* ctx, int32_t reps, double* us_out, double* gbs_out);

/* Plain streaming read of the same byte count (measurement, not part of the
 * hot path): K expert blobs' bytes read as one contiguous range of a layer's
 * slot pool by a grid-stride kernel (2048 workgroups, 16-byte non-temporal
 * loads, eight per lane in flight), the ranges rotating over every layer's
 * pool; timed and averaged as spp_probe_read_ceiling.  us_out: average time
 * per launch; gbs_out: the bytes read / that time.  Waits for all enqueued
 * work first.  ESTATE if a layer has fewer than K slots; EINVAL for reps
 * outside 1..10000. */
spp_status spp_probe_stream_read(spp_ctx* ctx, int32_t reps, double* us_out, double* gbs_out);

/* Where moe_layer_forward takes the priorities for the next layer's prefetch
 * (Table 5).  SPP_PREFETCH_ADAPTER (default): the layer's adapter, as above.
 * SPP_PREFETCH_PREV_TOKEN (Naive Prefetch): the experts layer l+1 activated
 * at its preceding call, each scored by its gate mass summed over that
 * call's tokens (fp64 in token order, then fp32), every other expert -inf;
 * no adapter runs.  spp_set_resident starts a new sequence (no preceding
 * call: nothing is prefetched).  EINVAL for an unknown source. */
spp_status spp_set_prefetch_source(spp_ctx* ctx, int32_t source);

/* Launch shape of this context's batch-1 routed-expert FFN over bf16/fp32
 * experts: about `wgs` workgroups share the (expert, unit) work list of one
 * token (default 512; 1..4096).  The 4-bit and batched FFNs choose their own
 * grids. */
spp_status spp_set_ffn_workgroups(spp_ctx* ctx, int32_t wgs);

/* Batch-1 FFN split (default 0, off).  1: when a layer call has both experts
 * whose data is complete (resident, or a copy that finished) and late ones
 * (loaded by this call's on-demand copies, or a prefetch still in flight),
 * the FFN of the complete ones runs on a second stream of the context beside
 * the on-demand copies, and the late ones after their copies on the compute
 * stream; the combine waits for both.  Outputs are bitwise those of the
 * single launch (each FFN workgroup works on one expert; the split is
 * skipped where the launch shape cannot guarantee that).  Batched contexts
 * ignore it.  Waits for the context's streams.  EINVAL unless 0 or 1. */
spp_status spp_set_ffn_overlap(spp_ctx* ctx, int32_t enabled);

/* Parallel prefetches (default 0).  With SPP_COPY_SPLIT and no storage
 * emulation, each prefetch is one whole copy; by default a call's prefetches
 * go in issue order on the first copy stream, so the highest-priority expert
 * finishes first at the link's full rate.  With 1 they alternate between the
 * two copy streams and share the link, so all of them finish together and
 * no per-copy gap on one stream separates them.  Measured on one MI355X:
 * M_max 4 gains 11-25% on the 4-bit workloads, M_max 2 gains 5-15% on the
 * 4-bit DeepSeek-shaped stack and loses 1-4% on the Qwen-shaped pair.  May
 * change between calls; copies into a slot stay ordered.  Outputs are
 * unchanged.  EINVAL unless 0 or 1. */
spp_status spp_set_prefetch_parallel(spp_ctx* ctx, int32_t enabled);

/* Engine of the expert copies from the offload tier.  A copy kernel reads
 * the pinned host store through its device-visible address (shader loads over
 * the host link); the DMA engines copy with hipMemcpyAsync.
 *   SPP_COPY_SPLIT (default): a layer's on-demand loads are one copy kernel
 *     (64 workgroups, all its blobs) on the compute stream ahead of the FFN
 *     that waits for them anyway; prefetches go to the DMA engines on the two
 *     copy streams, since they overlap compute kernels, which copy waves on
 *     the same compute units would slow down.
 *   SPP_COPY_KERNEL: every copy by a copy kernel (32 workgroups per half blob)
 *     on the copy streams.
 *   SPP_COPY_SDMA: every copy by the DMA engines on the copy streams.
 * On the copy streams each blob goes in two halves, one per stream, except
 * SPP_COPY_SPLIT's prefetches: one whole copy each, in issue order on the
 * first copy stream.  The engine may change between calls; a new copy into a
 * slot is ordered after any earlier copy into it still in flight.
 * spp_profile_expert_copy times the prefetch engine.  EINVAL for an unknown
 * engine. */
spp_status spp_set_copy_engine(spp_ctx* ctx, int32_t engine);

/* Storage-speed emulation ("Storage Sensitivity", Figure 5): every expert
 * copy is preceded, on each copy stream, by a bounded busy kernel of about
 * delay_us (0..100000), so one expert takes delay_us plus its transfer --
 * the offload tier behaves like slower storage behind the same link.  The
 * storage serves one expert at a time: while the delay is set, on-demand
 * loads too go through the copy streams (in issue order with the
 * prefetches) instead of the compute stream.  May change between calls.
 * Outputs are unchanged.  EINVAL outside the range. */
spp_status spp_set_tier_delay(spp_ctx* ctx, int32_t delay_us);

/* Test hooks for the copy/compute fences (for tests, not for production runs).
 * Poison: before every expert copy the target slot is filled with 0xFF bytes
 * (NaN in bf16 and fp32) on the stream that copies, so a kernel that read a
 * slot before its copy completed would produce NaN.  Copy delay: a bounded
 * busy kernel of about delay_us (0..100000) runs on that stream before every
 * copy (the mechanism of spp_set_tier_delay), so copies are still in flight
 * when the FFN is enqueued and the compute stream must wait for them.
 * Outputs are unchanged by both. */
spp_status spp_debug_set_poison(spp_ctx* ctx, int32_t enabled);
spp_status spp_debug_set_copy_delay(spp_ctx* ctx, int32_t delay_us);

/* ------------------------------------- host replacement policy (no device) */

/* The slot-replacement and prefetch-selection policy the context runs for
 * each layer, as a host-only object (no HIP calls), so that it can be driven
 * without a GPU.  Semantics are exactly those of the calls above. */
spp_status spp_policy_create(int32_t S, int32_t n, const int32_t* resident, int32_t count,
                             spp_slot_policy** out);
spp_status spp_policy_destroy(spp_slot_policy* p);
/* needed: the batch demand (any order, duplicates allowed); loads_out host
 * int32 [3*n] receives (expert, slot, evicted) triples in load order.  A
 * demand of more distinct experts than S is served in rounds (see
 * moe_layer_forward).  EINVAL for an out-of-range id. */
spp_status spp_policy_on_demand(spp_slot_policy* p, const int32_t* needed, int32_t count, int64_t tau,
                                int32_t* loads_out, int32_t* n_loads);
/* Prefetch selection + placement with priorities s (host fp32 [n]);
 * placed_out host int32 [3*max(M_max,0)]. */
spp_status spp_policy_prefetch(spp_slot_policy* p, const float* s, int32_t M_max, int64_t tau,
                               int32_t* placed_out, int32_t* n_placed);
spp_status spp_policy_get(spp_slot_policy* p, int32_t* experts_out, int64_t* stamps_out);

#ifdef __cplusplus
}
#endif

#endif /* SPP_H */
