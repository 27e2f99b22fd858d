/*
 * rkv.h - layer-routed KV-cache eviction on AMD Instinct MI355X (gfx950).
 *
 * C ABI of librkv.so.  It executes a static layer-wise eviction plan in the
 * sense of "Exploring a Layer-Wise Design Space for KV Cache Eviction":
 * Section 3.1, Eq. 1 defines the plan as, for every layer and phase
 * (prefill, decode), an operator r and a nominal retained-token capacity b;
 * Section 3.3, Eq. 3 defines how a fixed total capacity is split across
 * layers; Section 3.4 defines the adapter interface (a prompt-compression
 * handler and an incremental-update handler per operator, a plan loaded once).
 *
 * Operators: FULL (no eviction), STREAMING (StreamingLLM: attention sinks plus
 * recent tokens), SNAPKV (observation-window scoring with max-pooling),
 * H2O (accumulated-attention heavy hitters plus recent tokens), TOVA (the
 * current query's attention), H2O_FULL (H2O accumulating over every prompt
 * query).  Section 2.1 names these rule families; their arithmetic is stated at
 * each entry point.
 *
 * Conventions shared by every entry point
 *  - Every function returns an rkv_status; RKV_OK is 0.  On failure a message
 *    is available from rkv_last_error() (thread-local, valid until the next
 *    rkv call on the same thread) and no output buffer has been written.
 *  - Device buffers are owned by the caller (any allocator), as is the stream.
 *    The library allocates no device memory in rkv_prefill_evict or
 *    rkv_decode_step, never frees caller memory and never synchronises the
 *    stream: results are valid once the caller's stream has been synchronised.
 *  - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 *  - bf16 tensors are IEEE bfloat16, row-major, densely packed, with the
 *    shapes stated below.  Positions are token indices within the sequence.
 *  - A plan is immutable after creation; any number of host threads may use it.
 *  - Residency: rkv_prefill_evict's window-scoring kernel is persistent (one
 *    workgroup per compute unit, each waiting, with a bounded wait, for row sums
 *    stored by the others), so it needs every one of its workgroups resident at
 *    once.  Do not run it concurrently with other kernels on the same GPU (other
 *    streams, other processes, a second rkv_prefill_evict): serialize such calls
 *    on one stream.  If co-residency is denied anyway, a wait gives up, status
 *    bit 0 of the workspace is set (rkv_prefill_check) and that call's outputs
 *    are invalid; nothing hangs.
 */
#ifndef RKV_H
#define RKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RKV_VERSION 2

typedef enum {
  RKV_OK = 0,
  RKV_ERR_INVALID_ARG = 1, /* null pointer, negative size, unknown enum value */
  RKV_ERR_SHAPE = 2,       /* inconsistent shape (e.g. Hq not a multiple of Hkv, window > L) */
  RKV_ERR_PLAN = 3,        /* plan violates Eq. 1 constraints (operator not valid in that phase) */
  RKV_ERR_UNSUPPORTED = 4, /* valid request this build does not implement (e.g. head_dim != 128) */
  RKV_ERR_WORKSPACE = 5,   /* workspace missing, too small or misaligned */
  RKV_ERR_HIP = 6,         /* a HIP runtime call failed; rkv_last_error() has hipGetErrorString */
  RKV_ERR_DEVICE = 7       /* a kernel reported an internal failure (see rkv_prefill_check) */
} rkv_status;

/* Bits of the device status word in a prefill workspace (rkv_prefill_check).  Cleared by the
 * first kernel of every rkv_prefill_evict call and only OR-ed into afterwards, so it covers
 * every launch group of the call. */
#define RKV_STATUS_TIMEOUT 1u   /* a bounded wait gave up: this call's outputs are invalid */
#define RKV_STATUS_INVALID 2u   /* a score could not be repaired: this call's outputs are invalid */
#define RKV_STATUS_REPAIRED 4u  /* a row overflowed the fast path's fixed reference and the job was
                                   rescored exactly on the device: outputs valid */

/* Operators (Section 2.1 rule families; Section 3.1 r_{l,phi} values). */
typedef enum { RKV_FULL = 0, RKV_STREAMING = 1, RKV_SNAPKV = 2, RKV_H2O = 3, RKV_TOVA = 4, RKV_H2O_FULL = 5 } rkv_rule;
typedef enum { RKV_PHASE_PREFILL = 0, RKV_PHASE_DECODE = 1 } rkv_phase;
/* Deployment scope delta of a routed operator (Section 3.1): the phases it is active in; the
 * other phase uses FULL.  BOTH is a tied route: one operator in both phases. */
typedef enum { RKV_SCOPE_PREFILL = 0, RKV_SCOPE_DECODE = 1, RKV_SCOPE_BOTH = 2 } rkv_scope;
/* Score transforms T of Section 3.3: identity (attention entropy) or a cap at the
 * across-layer 95th percentile (PPL degradation). */
typedef enum { RKV_T_IDENTITY = 0, RKV_T_PPL_CAP = 1 } rkv_transform;

/* One row of the plan Pi of Eq. 1: operator and nominal capacity per phase.
 * Budgets are ignored for FULL. */
typedef struct {
  int32_t rule_prefill, budget_prefill;
  int32_t rule_decode, budget_decode;
} rkv_layer;

/* Operator parameters shared by all layers of a plan.
 *  window       w: number of observation-window queries (the last w prompt positions).
 *  pool_kernel  odd max-pool width used by SNAPKV (stride 1, clipped to the prefix).
 *  n_sink       StreamingLLM sink count; s0 = min(n_sink, b) first positions are kept.
 *  recent_num/recent_den  H2O keeps r = floor(b * num / den) most recent positions. */
typedef struct {
  int32_t window, pool_kernel, n_sink, recent_num, recent_den;
} rkv_params;

/* Tensor shape of one call: B sequences of seq_len positions, Hq query heads,
 * Hkv KV heads (Hq % Hkv == 0; query head hq reads KV head hq / (Hq/Hkv)), head_dim d. */
typedef struct {
  int32_t batch, seq_len, n_q_heads, n_kv_heads, head_dim;
} rkv_shape;

typedef struct rkv_plan rkv_plan;

/* One layer of a routed plan in the form of Section 3.2's completed routes: an operator, the
 * scope it is deployed in and its nominal capacity. */
typedef struct {
  int32_t rule, scope, budget;
} rkv_route_layer;

/* Per-layer device pointers of one prefill call (host arrays of n_layers pointers).
 *  q_win[l]     bf16 [B, Hq, w, d]   queries of positions L-w..L-1 (post-RoPE); [B, Hq, L, d],
 *               every position, for an H2O_FULL layer; a TOVA layer reads only row w-1 (the
 *               query of position L-1); may be NULL for layers whose prefill operator does not
 *               score (FULL, STREAMING).
 *  k[l], v[l]   bf16 [B, Hkv, L, d]  the prompt's keys and values.
 *  k_out[l], v_out[l]  bf16 [B, Hkv, n_l, d]  compacted cache, n_l = retained count
 *               (rkv_plan_retained_counts); row m holds position idx_out[l][..., m].
 *  idx_out[l]   int32 [B, Hkv, n_l]  retained positions, strictly ascending.
 *  score_out    NULL, or array whose entries are NULL or fp32 [B, Hkv, L]: the score each
 *               candidate position was ranked by (defined on the operator's candidate
 *               range [0, cand_end); other entries unspecified).  Debug/test output.
 *  acc_out      NULL, or array whose entries are NULL or fp32 [B, Hkv, n_l]: for scoring
 *               operators the unpooled group-mean score of each retained position (the
 *               window score for SNAPKV / H2O, the full-span score for H2O_FULL, the last
 *               query's attention for TOVA; it seeds H2O's decode-phase accumulated score);
 *               0 for FULL / STREAMING. */
typedef struct {
  const void* const* q_win;
  const void* const* k;
  const void* const* v;
  void* const* k_out;
  void* const* v_out;
  int32_t* const* idx_out;
  float* const* score_out;
  float* const* acc_out;
} rkv_prefill_io;

/* Decode-phase cache of every layer with a decode operator (entries of FULL layers may be NULL).
 *  k_cache[l], v_cache[l]  bf16 [B, Hkv, C_l, d], C_l = the layer's retained decode count.
 *  pos[l]   int32 [B, Hkv, C_l]  position held by each slot (slot order is arbitrary).
 *  acc[l]   fp32  [B, Hkv, C_l]  H2O accumulated attention of each slot (NULL allowed for
 *           layers whose decode operator is not H2O). */
typedef struct {
  void* const* k_cache;
  void* const* v_cache;
  int32_t* const* pos;
  float* const* acc;
} rkv_decode_state;

/* One decode step's new token per layer:
 *  q[l] bf16 [B, Hq, d]; k[l], v[l] bf16 [B, Hkv, d];
 *  victim_out NULL or entries NULL / int32 [B, Hkv]: slot overwritten by the new token, or -1
 *  when the new token itself was the one evicted. */
typedef struct {
  const void* const* q;
  const void* const* k;
  const void* const* v;
  int32_t* const* victim_out;
} rkv_decode_input;

/* Section 3.3, Eq. 3: split `total` retained positions over n_layers layers.
 * scores[n_layers] (host) -> T(scores) (transform), shift by (-min + 1e-6) if min <= 0,
 * weights w_l = T_l / sum T, provisional b_l = total * w_l; layers below b_min are fixed
 * at b_min and the rest is re-shared by weight until none falls below; then floor and hand
 * the residual units to the largest fractional remainders (equal remainders: lower layer).
 * budgets_out[n_layers] (host).  Host only, no GPU needed.
 * Errors: RKV_ERR_INVALID_ARG for null pointers, n_layers < 1, b_min < 0,
 * total < n_layers * b_min, non-finite scores or an unknown transform. */
int rkv_allocate_budgets(const double* scores, int32_t n_layers, int32_t transform, int64_t total,
                         int32_t b_min, int32_t* budgets_out);

/* Section 3.4: every operator adapter declares the phases it is compatible with; these
 * declarations define R_pre, R_dec and, for tied both-phase routes, their intersection.
 * *phase_mask receives bit 0 (valid in prefill) and bit 1 (valid in decode):
 *   FULL, STREAMING, H2O, TOVA: both phases; SNAPKV, H2O_FULL: prefill only (they rank prompt
 *   positions by prompt queries).  RKV_ERR_INVALID_ARG for an unknown rule or a null pointer. */
int rkv_rule_phases(int32_t rule, int32_t* phase_mask);

/* Section 3.1 (Eq. 1) and 3.4: validate and freeze a plan.  Host only.
 * rule_prefill must lie in R_pre and rule_decode in R_dec (rkv_rule_phases) -> RKV_ERR_PLAN
 * otherwise.  Budgets must be >= 0 (>= 2 for a decode H2O layer, >= 1 for decode STREAMING and
 * TOVA); window >= 1, pool_kernel odd >= 1, n_sink >= 0, 0 <= recent_num <= recent_den,
 * recent_den >= 1.  *out receives a new plan. */
int rkv_plan_create(const rkv_layer* layers, int32_t n_layers, const rkv_params* params, rkv_plan** out);

/* Sections 3.1 and 3.2: a plan from a completed route.  Layer l runs route[l].rule with nominal
 * capacity route[l].budget in the phases of route[l].scope and FULL in the other phase.  A
 * RKV_SCOPE_BOTH layer is a tied both-phase route: the operator must be in R_pre and R_dec (the
 * intersection of the Section 3.4 declarations), else RKV_ERR_PLAN; a PREFILL / DECODE layer's
 * operator must be in that phase's set.  RKV_ERR_INVALID_ARG for an unknown scope or rule; the
 * remaining checks are those of rkv_plan_create.  *out receives a new plan. */
int rkv_plan_from_route(const rkv_route_layer* route, int32_t n_layers, const rkv_params* params, rkv_plan** out);
void rkv_plan_destroy(rkv_plan* plan);
/* Implementation call (plan bookkeeping): the plan's layer count. */
int rkv_plan_num_layers(const rkv_plan* plan, int32_t* n_layers);

/* Sections 3.1 and 3.4: the plan is fixed offline and loaded once per run.  A serialized plan is
 * a little-endian byte record: "RKVP", int32 format version (1), int32 n_layers, the five
 * rkv_params fields, then per layer (rule_prefill, budget_prefill, rule_decode, budget_decode);
 * 32 + 16 * n_layers bytes.  Host only.
 * rkv_plan_serialize: writes the record into buf if cap is large enough and always sets *size
 *   to the record's length (buf may be NULL to query it); RKV_ERR_INVALID_ARG if cap is too small.
 * rkv_plan_deserialize: parses and re-validates as rkv_plan_create does (same errors), plus
 *   RKV_ERR_INVALID_ARG for a wrong magic, version or length.  *out receives a new plan. */
int rkv_plan_serialize(const rkv_plan* plan, void* buf, size_t cap, size_t* size);
int rkv_plan_deserialize(const void* buf, size_t size, rkv_plan** out);

/* Section 3.1: b_{l,phi} is a nominal capacity, so the positions a layer actually retains in
 * `phase` for a prompt of seq_len tokens are FULL -> seq_len, otherwise min(budget, seq_len)
 * (Section 3.1 matches configured capacities, not retained counts).  counts_out[n_layers]
 * (host).  Errors: RKV_ERR_INVALID_ARG for null pointers, an unknown phase or seq_len < 0. */
int rkv_plan_retained_counts(const rkv_plan* plan, int32_t phase, int32_t seq_len, int32_t* counts_out);

/* Implementation call (no paper passage): bytes of device workspace rkv_prefill_evict needs for
 * `shape` (the base must be 256-byte aligned).  The workspace holds the status word, per-slice
 * row sums, scores and the slice-edge sums of the scoring kernels.  Errors: as the shape checks
 * of rkv_prefill_evict. */
int rkv_prefill_workspace_size(const rkv_plan* plan, const rkv_shape* shape, size_t* bytes);

/* Prefill prompt compression of every layer (the prompt-compression handler of Section 3.4),
 * enqueued on `stream`.  Per sequence, layer and KV head h with G = Hq / Hkv:
 *   A[hq, j] = sum_{i<w} softmax_j( Q[hq,i] . K[h,j] / sqrt(d) ), row i at position L-w+i
 *              seeing keys j <= L-w+i (causal inside the window);
 *   SNAPKV:   S[h,j] = mean_g maxpool_j(A[hG+g, .]) over the prefix [0, L-w);
 *             keep top-(b-w) of S plus the window [L-w, L) (b <= w: the last b positions);
 *   H2O:      S[h,j] = mean_g A[hG+g, j]; r = floor(b*num/den);
 *             keep top-(b-r) of S over [0, L-r) plus [L-r, L);
 *   H2O_FULL: H2O whose accumulation spans every prompt query (q_win[l] then holds all L
 *             positions, bf16 [B, Hq, L, d]): S[h,j] = mean_g sum_{t>=j} softmax_j(Q[hG+g,t] .
 *             K[h,.] / sqrt(d)) over keys <= t; the same selection as H2O;
 *   TOVA:     S[h,j] = mean_g softmax_j(Q[hG+g, w-1] . K[h,j] / sqrt(d)) over all L keys (the
 *             attention of the prompt's last query, position L-1); keep the top-b of [0, L);
 *   STREAMING: keep [0, min(n_sink,b)) plus the last b - min(n_sink,b) positions;
 *   FULL, or b >= L: keep everything.
 * Top-k order is (score descending, position ascending) on fp32 scores.  K/V rows are
 * copied bit-exactly into k_out / v_out in ascending position order.
 * Numerics: SNAPKV / H2O / H2O_FULL take their exponentials against a per-row reference, the
 * larger of the row's logits with its own key and with key 0.  A row with a key more than about
 * 88 natural-log units above that reference overflows that path.  A SNAPKV / H2O job where
 * this happens is rescored exactly on the device before selection (RKV_STATUS_REPAIRED; outputs
 * valid); an H2O_FULL layer reports RKV_STATUS_INVALID.  TOVA is exact by construction (per-head
 * running maxima).  The status word (rkv_prefill_check) must be clean of RKV_STATUS_TIMEOUT and
 * RKV_STATUS_INVALID for the outputs to be valid; the call itself cannot report them, since
 * it returns before the kernels run.
 * ws: caller-owned device workspace of at least rkv_prefill_workspace_size bytes, 256-byte
 * aligned; one workspace per call in flight (see Residency above).
 * Errors: RKV_ERR_INVALID_ARG (null io / pointer for a layer that needs it), RKV_ERR_SHAPE,
 * RKV_ERR_UNSUPPORTED (head_dim != 128, G * ceil(w/32) > 8 for window-scored layers,
 * Hq / Hkv not in {1, 2, 4, 8} for TOVA / H2O_FULL layers, seq_len > 2^24),
 * RKV_ERR_WORKSPACE, RKV_ERR_HIP (launch failure).  Validation ends before the first launch: a
 * failed call enqueues nothing. */
int rkv_prefill_evict(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* io,
                      void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): rkv_prefill_evict with the library's own workspace,
 * a static device array of 64 MiB per GPU (held until the process ends; enough for a 32-layer
 * route of one 8192-token sequence).  Arguments, outputs and errors are those of
 * rkv_prefill_evict; a call needing more than 64 MiB (rkv_prefill_workspace_size) fails with
 * RKV_ERR_WORKSPACE before anything is enqueued.  status_out: NULL, or a device uint32 that
 * receives the call's status word (RKV_STATUS_* bits) on `stream` after the pass.  Allocates
 * nothing: no hipMalloc / hipFree, no allocating library routine.  Every call on one GPU shares
 * the array; calls that overlap on one GPU (several streams or threads) race and must be
 * serialised by the caller. */
int rkv_prefill_evict_noalloc(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* io,
                              uint32_t* status_out, void* stream);

/* Implementation call (failure reporting of rkv_prefill_evict): synchronously read the status
 * word a previous rkv_prefill_evict left in `ws` (RKV_STATUS_* bits; 0 = clean).  Outputs are
 * valid unless RKV_STATUS_TIMEOUT or RKV_STATUS_INVALID is set.  Uses a blocking copy (waits
 * for the device), so it belongs after the caller's own synchronisation; for tests, debugging
 * and callers that want to raise on failure.  Errors: RKV_ERR_INVALID_ARG, RKV_ERR_WORKSPACE,
 * RKV_ERR_HIP. */
int rkv_prefill_check(const void* ws, size_t ws_bytes, int32_t* status_out);

/* One decode step (the incremental-update handler of Section 3.4) for every layer, on `stream`.
 * shape->seq_len is ignored; `position` is the new token's position p.
 * H2O: per (sequence, layer, KV head) the new key joins the C cached ones; each of the G query
 *   heads takes softmax(q . k / sqrt(d)) over the C+1 entries; every entry's acc grows by the
 *   group mean (new entry from 0, fp32); among entries with pos <= p - r
 *   (r = floor(C*num/den)) the smallest acc is evicted, ties to the smallest position;
 *   the new token (k, v, pos = p, acc) takes the victim's slot.
 * TOVA (Section 2.1, attention of the current query): the same C+1 entries and softmax; an
 *   entry's score is the group mean of its probabilities at this step (nothing accumulates);
 *   the smallest score among all C+1 entries (the new one included) is evicted, ties to the
 *   smallest position; the new token (k, v, pos = p) takes the victim's slot.  acc is neither
 *   read nor written (state->acc[l] may be NULL for such a layer).
 * STREAMING: the slot with the smallest position >= n_sink is replaced by the new token.
 * FULL: the layer is skipped.
 * Errors: as rkv_prefill_evict; RKV_ERR_SHAPE if position < C.  Every layer is validated
 * before the first launch: a failed call enqueues nothing. */
int rkv_decode_step(const rkv_plan* plan, const rkv_shape* shape, const rkv_decode_state* state,
                    const rkv_decode_input* input, int32_t position, void* stream);

/* Section 3.4: the runtime tracks the prefill-to-decoding transition.  This is that hand-off:
 * for every layer whose decode operator is not FULL, the prompt cache a rkv_prefill_evict call
 * left in `prefill` (same plan and shape, shape->seq_len = the prompt length L) becomes the
 * layer's decode cache:  k_cache[l] <- k_out[l], v_cache[l] <- v_out[l], pos[l] <- idx_out[l]
 * and, for a decode H2O layer, acc[l] <- acc_out[l] (the seed of the accumulated attention:
 * the unpooled score of each retained position; 0 when the prefill operator does not score).
 * The layer's decode capacity must equal its prefill retained count (FULL: L, else
 * min(budget, L)), else RKV_ERR_SHAPE.  A decode H2O layer whose prefill operator scores needs
 * acc_out[l] (else RKV_ERR_INVALID_ARG).  Entries where source and destination are the same
 * buffer are left as they are, so a caller may also decode in the prefill outputs directly.
 * One copy kernel per 32 layers on `stream`; no allocation, no synchronisation.  The prefill
 * call's status word still decides whether its outputs (and so this cache) are valid.
 * Errors: RKV_ERR_INVALID_ARG (null pointers), RKV_ERR_SHAPE, RKV_ERR_HIP.  Validation ends
 * before the first launch. */
int rkv_decode_init_from_prefill(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* prefill,
                                 const rkv_decode_state* state, void* stream);

/* Section 3.3: the attention-entropy layer score H_l, the mean over sequences, query heads and
 * profiled query positions of the Shannon entropy (nats) of each query's causal attention row
 * softmax_j(q_t . k_j / sqrt(d)), j = 0..t (query head hq reads KV head hq / G).  Entropy
 * allocation feeds H_l unchanged (identity transform) into rkv_allocate_budgets with b_min 32.
 * shape: batch B, seq_len L, Hq, Hkv (Hq / Hkv in {1, 2, 4, 8}), head_dim 128.
 * q[l]: bf16 [B, Hq, n_q, d], the queries of the last n_q positions L - n_q .. L - 1 of layer l
 *   (n_q = L profiles every query); k[l]: bf16 [B, Hkv, L, d].  Device pointers, host arrays.
 * rows_out: device fp32 [n_layers, B, Hq, n_q], every profiled row's entropy;
 * h_out: device fp32 [n_layers]; status: device uint32, cleared by the call's first launch and
 *   then OR-ed into: bit 0 (1) when some row is not finite (h_out is then invalid), bit 2 (4)
 *   when a block of rows overflowed the fast path's per-row reference (a logit more than ~88
 *   natural-log units above the larger of the row's logits with its own key and with key 0)
 *   and was recomputed exactly (results valid).
 * ws: caller-owned device workspace of at least rkv_entropy_workspace_size bytes (8-byte
 *   aligned; per-block partial sums).  Enqueued on `stream`; no allocation.
 * Errors: RKV_ERR_INVALID_ARG (null pointers, n_layers < 1, n_q outside [1, L]), RKV_ERR_SHAPE,
 *   RKV_ERR_UNSUPPORTED (head_dim != 128 or Hq / Hkv not in {1, 2, 4, 8}), RKV_ERR_WORKSPACE,
 *   RKV_ERR_HIP. */
int rkv_entropy_workspace_size(const rkv_shape* shape, int32_t n_layers, int32_t n_q, size_t* bytes);
int rkv_entropy_profile(const rkv_shape* shape, int32_t n_layers, int32_t n_q, const void* const* q,
                        const void* const* k, float* rows_out, float* h_out, uint32_t* status, void* ws,
                        size_t ws_bytes, void* stream);

/* Implementation calls (measurement, no paper passage): kernel timing for benchmarks and tests.
 * rkv_profile_enable(stage) makes every following
 * launch of that stage record a pair of HIP events around it on the caller's stream
 * (stage: 0 counter reset, 1 scoring, 2 selection, 3 gather, 4 decode; -1 disables).
 * Up to 4096 launches are kept.  rkv_profile_read synchronises on the recorded events,
 * returns the number of launches and their summed duration in milliseconds, and clears
 * the record.  Host-side state shared by all threads. */
int rkv_profile_enable(int32_t stage);
int rkv_profile_read(int32_t* n_launches, double* total_ms);

/* Implementation calls: the message of the calling thread's last failed call, and the ABI
 * version (RKV_VERSION). */
const char* rkv_last_error(void);
int rkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RKV_H */
