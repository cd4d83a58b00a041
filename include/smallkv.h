/*
 * smallkv.h -- C ABI of the MI355X (gfx950) library for SmallKV's
 * per-decode-step compensated attention (arXiv 2508.02751).
 *
 * One decode step has three stages (Algorithm 1, decode branch):
 *   1. smallkv_small_attn  -- the small model's full decode attention over
 *      its uncompressed cache (the selection of the "Saliency Shift
 *      Compensation" paragraph is made from this full small cache);
 *   2. smallkv_partition   -- per small head, the tokens ordered by the small
 *      model's attention split into critical (TopK), marginal (Top(P-K)) and
 *      evicted sets (Eq. 4 read as "keep the top-scored tokens", Eq. 6);
 *   3. smallkv_hybrid_attn -- each large head i reads the partition of small
 *      head f(i) (Eq. 3): exact softmax attention over its critical keys
 *      (O_c), the small model's probabilities times the large model's V for
 *      the marginal tokens (O_m), evicted tokens contribute nothing, and the
 *      output O_c + O_m as weighted by smallkv_norm_t (Eq. 6; Algorithm 1,
 *      "Attention Output by O_c + O_m").
 * smallkv_step runs all three for every layer of both models.
 *
 * Conventions shared by every entry point
 *   - Pointers named in the structs and arguments are DEVICE pointers unless
 *     stated otherwise; the descriptor structs themselves live in host memory
 *     and are read only during the call.
 *   - Ownership: the caller allocates and owns every buffer, including the
 *     workspace.  The library allocates no device memory, keeps no state
 *     between calls and never synchronises: work is enqueued on `stream`
 *     (a hipStream_t; NULL is the null stream) and the call returns.  The one
 *     exception is smallkv_step_noalloc, which takes no workspace and runs on
 *     a static device array of the library's (one per GPU, see there).
 *   - Errors: a negative status is returned, before anything is enqueued,
 *     for every condition visible on the host (null pointers, sizes, head
 *     dims, dtype, workspace too small, head counts).  A kernel launch
 *     failure returns SMALLKV_EDEVICE.  Values that live in device memory
 *     (seq_len, k_crit, k_marg, head_map, indices) cannot be checked on the
 *     host: the kernels clamp them into range (see smallkv_batch_t) so that no
 *     access leaves its buffer, and results outside the stated
 *     preconditions are unspecified.
 *   - Layout: every tensor is dense row-major in the order its comment gives.
 *   - Numerics: logits are fp32 and bit-reproducible: each is a sequential
 *     fp32 fused multiply-add chain over the head dimension starting from +0,
 *     then one fp32 multiply by `scale`, with -0 returned as +0.  The
 *     partition ranks on these logits (larger first, equal logits by lower
 *     token index), so it is exact and deterministic.  Softmax statistics,
 *     probabilities and outputs are fp32 arithmetic, rounded to the model
 *     dtype (round to nearest even) on output.
 */
#ifndef SMALLKV_H
#define SMALLKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SMALLKV_ABI_VERSION 8

typedef enum { SMALLKV_F32 = 0, SMALLKV_BF16 = 1 } smallkv_dtype_t;

/* Weights of the two parts of the compensated row: O = alpha_C*O_c + alpha_M*O_m,
 * with S'_C, S'_M the small head's probability mass on the critical and
 * marginal sets.  O_c is the large head's softmax over its critical keys
 * (weights summing to 1); O_m = sum over marginal t of p'_t * V_t. */
typedef enum {
  SMALLKV_NORM_REMAINING = 0, /* default: alpha_C = 1 - S'_M, alpha_M = 1.  The
                                 marginal tokens keep the small model's
                                 probabilities; the critical softmax fills the
                                 remaining mass, so the weights sum to 1 */
  SMALLKV_NORM_NONE = 1,      /* alpha_C = 1, alpha_M = 1: the sum O_c + O_m
                                 exactly as the implementation pseudocode adds
                                 them (weights sum to 1 + S'_M) */
  SMALLKV_NORM_SLM_CRIT = 2,  /* alpha_C = S'_C, alpha_M = 1: Eq. 6 with the
                                 large model's full-row denominator estimated
                                 by the small model's */
  SMALLKV_NORM_RETAINED = 3,  /* alpha_C = S'_C/(S'_C+S'_M), alpha_M = 1/(S'_C+S'_M) */
  SMALLKV_NORM_MARG_FILL = 4  /* alpha_C = S'_C, alpha_M = (1-S'_C)/S'_M (0 if S'_M = 0) */
} smallkv_norm_t;

enum {
  SMALLKV_OK = 0,
  SMALLKV_EINVAL = -1,       /* a null pointer, a bad size or an inconsistent shape */
  SMALLKV_EUNSUPPORTED = -2, /* a valid request outside what the kernels implement */
  SMALLKV_EWORKSPACE = -3,   /* ws_bytes below smallkv_workspace_size() */
  SMALLKV_EDEVICE = -4       /* a HIP launch error */
};

/* One model's attention operands for one decode step (all layers). */
typedef struct {
  int32_t n_layers;   /* l (small) or L (large) */
  int32_t n_q_heads;  /* query heads per layer */
  int32_t n_kv_heads; /* kv heads per layer; n_q_heads % n_kv_heads == 0, query
                         head h reads kv head h / (n_q_heads / n_kv_heads) */
  int32_t head_dim;   /* 64 or 128 */
  int32_t dtype;      /* smallkv_dtype_t of q, k, v and out */
  float scale;        /* softmax scale, normally 1/sqrt(head_dim) */
  const void *q;      /* [B][n_layers][n_q_heads][head_dim] */
  const void *k;      /* [B][n_layers][n_kv_heads][n_rows][head_dim] */
  const void *v;      /* same layout as k */
  int64_t n_rows;     /* rows per (sequence, layer, kv head): n_cap for a full
                         cache, or the capacity of a compact store */
  const int32_t *k_slot; /* large model only, optional: [B][n_layers][n_kv_heads][n_cap]
                            token -> row of k (-1: not held); NULL means row = token */
  const int32_t *v_slot; /* same for v */
  void *out;          /* [B][n_layers][n_q_heads][head_dim] attention output */
  /* Small model only, optional, both or neither: the small model's own KV
   * eviction (its cache compressed, "Implementation Optimization" (2)).
   * held[b]: rows of its cache in use, clamped to [1, n_rows] (precondition
   * held[b] <= N_b); row_pos [B][n_layers][n_kv_heads][n_rows]: the token
   * position each row holds, strictly ascending over the first held[b] rows
   * and below N_b.  k and v then hold n_rows <= n_cap rows per kv head.
   * Stages 1-2 run over the held rows: logits rows have stride n_rows and
   * entry r is row r's logit; the partition ranks rows (recent tokens are the
   * last rows) and names tokens by row_pos (clamped to [0, N_b - 1]); a
   * token the small model does not hold is never critical or marginal.
   * NULL: the small cache holds every token (row t = token t). */
  const int32_t *held;
  const int32_t *row_pos;
} smallkv_model_t;

/* The batch of sequences and their budgets. */
typedef struct {
  int32_t batch;          /* B >= 1 */
  int32_t n_cap;          /* max tokens per sequence (cache capacity) >= 1 */
  const int32_t *seq_len; /* [B] current length N_b, the current token included;
                             precondition 1 <= N_b <= n_cap (clamped on device) */
  const int32_t *k_crit;  /* [B] critical budget K_b >= 1 */
  const int32_t *k_marg;  /* [B] marginal budget >= 0 */
  const int32_t *k_recent; /* [B] recent tokens R_b >= 0, or NULL (none).  The
                              experimental setup gives recent tokens a share of
                              the budget (critical : recent : marginal =
                              2 : 1 : 2): the last r_b tokens are critical
                              whatever their score and are not ranked */
  int32_t kc_cap;         /* host: width of the critical index rows, >= 1 */
  int32_t km_cap;         /* host: width of the marginal index rows, >= 0 */
  /* Set sizes, computed on device per sequence:
   *   r     = min(max(R_b, 0), N_b, kc_cap)          (0 when k_recent is NULL)
   *   top   = min(max(K_b, 1), N_b - r, kc_cap - r)  (top-ranked of the older tokens)
   *   |C|   = r + top
   *   |M|   = min(max(k_marg_b, 0), N_b - |C|, km_cap)
   * Within the preconditions (K_b + R_b <= kc_cap, the marginal count <=
   * km_cap) the caps never bind. */
} smallkv_batch_t;

/* Stage 1.  For every sequence b, small layer, small query head h (small head
 * id j = layer * n_q_heads + h) and token t < N_b:
 *   logits[b][j][t] = the fp32 logit described above (entries t >= N_b are
 *                     not written)
 *   row_max[b][j]   = max_t logits,  row_sum[b][j] = sum_t exp(logit - row_max)
 *   small->out      = sum_t (exp(logit - row_max) / row_sum) * V_t
 * logits: [B][n_layers*n_q_heads][n_cap] fp32; row_max, row_sum: [B][n_layers*n_q_heads]
 * fp32.  small->k_slot and v_slot must be NULL; small->n_rows == n_cap, or
 * with small->held the held rows r < held[b] are attended and logits rows
 * have stride n_rows. */
int smallkv_small_attn(const smallkv_batch_t *batch, const smallkv_model_t *small,
                       float *logits, float *row_max, float *row_sum, void *ws,
                       size_t ws_bytes, void *stream);

/* Stage 2.  For every row (b, j), j < n_small_heads: the last r tokens are
 * critical; the older tokens t < N_b - r, ordered by (logit descending, index
 * ascending), give the other |C| - r critical ones, then |M| marginal, the
 * rest evicted (r = 0 without k_recent: every token is ranked).
 * `small` is optional (NULL: the rows are tokens 0..N_b-1); with the small
 * model's own eviction (small->held) the rows are its held rows, ranked the
 * same way and named by small->row_pos, as in smallkv_step; n_small_heads
 * must then be small->n_layers * small->n_q_heads.
 *   crit_idx  [B][n_small_heads][kc_cap] int32, ascending, padded with -1
 *   marg_idx  [B][n_small_heads][km_cap] int32, ascending, padded with -1
 *   marg_prob [B][n_small_heads][km_cap] fp32, p'_t = exp(logit_t - row_max)/row_sum
 *             for marg_idx's token (0 in padding)
 *   mass      [B][n_small_heads][2] fp32, {S'_C, S'_M}: the sum of p' over each set
 * Inputs are stage 1's logits, row_max and row_sum.  Deterministic. */
int smallkv_partition(const smallkv_batch_t *batch, const smallkv_model_t *small,
                      int32_t n_small_heads, const float *logits, const float *row_max,
                      const float *row_sum, int32_t *crit_idx,
                      int32_t *marg_idx, float *marg_prob, float *mass, void *ws,
                      size_t ws_bytes, void *stream);

/* Stage 3.  For every sequence b, large layer and large query head h, with
 * j = head_map[layer * n_q_heads + h] (0 <= j < n_small_heads) and kv head
 * g = h / (n_q_heads / n_kv_heads):
 *   s_t = scale * <q, K_g[row(t)]> for t in crit_idx[b][j]
 *   O_c = sum_C softmax_C(s)_t V_g[row(t)],  O_m = sum_M marg_prob_t V_g[row(t)]
 *   large->out = alpha_C * O_c + alpha_M * O_m   (alphas from `mode` and mass[b][j])
 * head_map: [n_layers * n_q_heads] int32 (device).  Rows come from
 * large->k_slot / v_slot when given.  select = SMALLKV_SELECT_GROUP: the
 * lists are those of the large head's (layer, kv head) and marg_prob / mass
 * its own (the layouts of smallkv_group_select). */
int smallkv_hybrid_attn(const smallkv_batch_t *batch, const smallkv_model_t *large,
                        const int32_t *head_map, int32_t n_small_heads,
                        const int32_t *crit_idx, const int32_t *marg_idx,
                        const float *marg_prob, const float *mass, int32_t mode,
                        int32_t select, void *ws, size_t ws_bytes, void *stream);

/* Stage 3 for the large layers [layer_begin, layer_begin + layer_count)
 * only, as a model that runs its layers one after another calls it (one
 * call per layer, each with that layer's queries in place).  `large`
 * describes the whole stack exactly as for smallkv_hybrid_attn (n_layers =
 * L, the same pointers and layouts); q, k, v, the slot maps and out are
 * touched only in those layers' slices; head_map, the lists and the weights
 * are the step's.  ws_bytes >= smallkv_hybrid_attn_workspace_size for
 * layer_count.  SMALLKV_EINVAL for a range outside [0, L); the other errors
 * as smallkv_hybrid_attn. */
int smallkv_hybrid_attn_layers(const smallkv_batch_t *batch, const smallkv_model_t *large,
                               int32_t layer_begin, int32_t layer_count, const int32_t *head_map,
                               int32_t n_small_heads, const int32_t *crit_idx,
                               const int32_t *marg_idx, const float *marg_prob,
                               const float *mass, int32_t mode, int32_t select, void *ws,
                               size_t ws_bytes, void *stream);

/* Bytes of workspace a stage-3 call over layer_count layers needs
 * (smallkv_hybrid_attn: layer_count = large->n_layers).  Host only. */
int smallkv_hybrid_attn_workspace_size(const smallkv_batch_t *batch,
                                       const smallkv_model_t *large, int32_t layer_count,
                                       int32_t n_small_heads, size_t *bytes);

/* Stage 2 of SMALLKV_SELECT_GROUP (see smallkv_select_t): from stage 1's
 * logits, row_max and row_sum, the lists of every (sequence, large layer, kv
 * head), crit_idx [B][L*Hkv][kc_cap] and marg_idx [B][L*Hkv][km_cap], and the
 * weights of every large query head, marg_prob [B][L*Hq][km_cap] (its own
 * small head's p' on the group's marginal list) and mass [B][L*Hq][2].  Only
 * the shapes of `large` are read.  ws: smallkv_group_select_workspace_size. */
int smallkv_group_select(const smallkv_batch_t *batch, const smallkv_model_t *small,
                         const smallkv_model_t *large, const int32_t *head_map,
                         const float *logits, const float *row_max, const float *row_sum,
                         int32_t *crit_idx, int32_t *marg_idx, float *marg_prob, float *mass,
                         void *ws, size_t ws_bytes, void *stream);
int smallkv_group_select_workspace_size(const smallkv_batch_t *batch,
                                        const smallkv_model_t *small,
                                        const smallkv_model_t *large, size_t *bytes);

/* Stage 2 of SMALLKV_SELECT_ACCUM (see smallkv_select_t): acc_score
 * [B][n_small_heads][n_cap] (the running scores) += this step's
 * probabilities, then the lists and weights in the per-head layout of
 * smallkv_partition.  ws: smallkv_accum_select_workspace_size. */
int smallkv_accum_select(const smallkv_batch_t *batch, const smallkv_model_t *small,
                         const float *logits, const float *row_max, const float *row_sum,
                         float *acc_score, int32_t *crit_idx, int32_t *marg_idx,
                         float *marg_prob, float *mass, void *ws, size_t ws_bytes, void *stream);
int smallkv_accum_select_workspace_size(const smallkv_batch_t *batch,
                                        const smallkv_model_t *small, size_t *bytes);

/* How tokens are selected (smallkv_step_t.select). */
typedef enum {
  SMALLKV_SELECT_HEAD = 0,  /* default: each large head i takes the sets of its
                               small head f(i) (the partition of stage 2) */
  SMALLKV_SELECT_GROUP = 1, /* the query heads of one large kv head share one
                               critical and one marginal set (the cache is
                               stored per kv head), ranked by
                               F(t) = sum over the group's heads h of
                               p_f(h)(t) -- the implementation pseudocode's
                               `.sum.topk` (Appendix D).  F decides integers and
                               is evaluated one way: e = exp32(logit - row_max)
                               (exp32 as for smallkv_match), Zq = the exact
                               integer sum over the row of floor(e * 2^40),
                               Z = fp32(Zq) * 2^-40, F = ((e_0/Z_0 + e_1/Z_1) +
                               ...) in fp32 over the group's heads in ascending
                               order; ranked like the partition (F descending,
                               index ascending; recent tokens first).  Each
                               head keeps its own p' = exp(logit - row_max) /
                               row_sum on the shared marginal set. */
  SMALLKV_SELECT_ACCUM = 2  /* per small head, ranked by an accumulated score
                               (H2O's accumulated attention, the eviction the
                               method builds on): the caller-owned state
                               acc_score [B][n_small_heads][n_cap] (zeroed
                               before the first step) becomes, for t < N_b,
                               acc[t] = acc[t] + e(t)/Z in fp32 (e and Z as
                               for SMALLKV_SELECT_GROUP), and the partition
                               ranks acc (descending, index ascending; recent
                               tokens first); marg_prob and mass are this
                               step's p'.  Layouts as for the default. */
} smallkv_select_t;

/* A whole decode step: stage 1 over every small layer, stage 2 over every
 * small head, stage 3 over every large layer, enqueued back to back on one
 * stream.  The intermediate buffers are the caller's, laid out as above,
 * with n_small_heads = small.n_layers * small.n_q_heads.  With
 * SMALLKV_SELECT_GROUP: crit_idx and marg_idx are [B][L*Hkv][cap] (one row
 * per large layer and kv head), marg_prob [B][L*Hq][km_cap] and mass
 * [B][L*Hq][2] (one row per large query head); the small model's cache must
 * hold every token (small.held NULL) and L's query heads per kv head <= 16.
 * SMALLKV_SELECT_ACCUM also needs small.held NULL. */
typedef struct {
  smallkv_batch_t batch;
  smallkv_model_t small, large;
  const int32_t *head_map; /* [large.n_layers * large.n_q_heads] */
  int32_t mode;            /* smallkv_norm_t */
  float *logits, *row_max, *row_sum;
  int32_t *crit_idx, *marg_idx;
  float *marg_prob, *mass;
  int32_t select;          /* smallkv_select_t */
  float *acc_score;        /* SMALLKV_SELECT_ACCUM only: [B][n_small_heads][n_cap]
                              running scores, read and updated by every step */
} smallkv_step_t;

int smallkv_step(const smallkv_step_t *step, void *ws, size_t ws_bytes, void *stream);

/* smallkv_step that also records the caller's hipEvents on `stream` at the
 * step's stage boundaries, so that the kernels the step runs can be timed
 * by stage: events[0] before stage 1; events[1] after stage 1's per-chunk
 * kernel (per-head selection: stage 1's merge runs in the next kernel,
 * fused with the partition; group and accumulated selection: after stage
 * 1's merge); events[2] after stage 2; events[3] after stage 3.  `events`
 * may be NULL and any entry may be NULL (not recorded).  Same checks,
 * kernels and results as smallkv_step; SMALLKV_EDEVICE if a record fails. */
int smallkv_step_events(const smallkv_step_t *step, void *ws, size_t ws_bytes, void *stream,
                        void *const *events);

/* Bytes of workspace that smallkv_step needs for `step`; the single-stage
 * calls need no more than this for the same shapes.  Host only. */
int smallkv_workspace_size(const smallkv_step_t *step, size_t *bytes);

/* A whole step that allocates nothing and takes no workspace, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same descriptor, kernels,
 * results and errors as smallkv_step; the caller still owns every input,
 * intermediate and output buffer the descriptor names.
 *   - The workspace is a static device array of SMALLKV_NOALLOC_SCRATCH_BYTES
 *     that the library holds on every GPU it runs on, from the first call
 *     there until the process ends.  SMALLKV_EWORKSPACE (nothing enqueued)
 *     when smallkv_workspace_size(step) exceeds it.  The first call on a GPU
 *     (the device `stream` belongs to; the current device for the null
 *     stream) looks the array's address up with that device current;
 *     SMALLKV_EDEVICE if that fails.
 *   - No hipMalloc, hipFree or other allocating call, on any call.
 *   - Every call on one GPU uses that GPU's one array, which keeps the last
 *     call's contents: calls that overlap on one GPU (two streams, two host
 *     threads) race and must be serialised by the caller.  Nothing needs
 *     clearing between calls: a step reads no byte of the array that it has
 *     not written first. */
#define SMALLKV_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int smallkv_step_noalloc(const smallkv_step_t *step, void *stream);

/* ---------------------------------------------------------------------------
 * Retained-store maintenance (Algorithm 1: the critical tokens keep K and V,
 * the marginal tokens V; the paper migrates these rows between host and
 * device memory in parallel with the large model's forward).  After a step's
 * selection, for every (sequence b, large layer, kv head):
 *   U_K = the union of the critical lists of the query heads it serves,
 *   U_V = U_K united with their marginal lists (tokens < N_b);
 *   new_k row r = the K row of U_K's r-th token in ascending order (new_v
 *   likewise over U_V), for r < rows; k_slot[t] = t's row in new_k or -1,
 *   v_slot[t] likewise, for t < N_b (entries t >= N_b are not written).
 * Each row is copied from the old store when its old slot map holds the
 * token (old_k row old_k_slot[t]), else from the full store (row t), so that
 * only tokens new to a set are read from the full store, which may be
 * device memory or pinned host memory (hipHostMalloc; the kernels read it
 * over the host link at the device address the runtime maps it to);
 * pageable host memory gives SMALLKV_EINVAL before anything is enqueued.  The result feeds smallkv_step /
 * smallkv_hybrid_attn as large->k/v (n_rows = rows) with large->k_slot /
 * v_slot.  Deterministic; a union longer than `rows` keeps its first rows
 * and counts reports the full size. */
typedef struct {
  smallkv_batch_t batch;   /* the step's batch: seq_len, n_cap (<= 131072), kc_cap, km_cap */
  int32_t n_layers, n_q_heads, n_kv_heads, head_dim, dtype;  /* the large model */
  const int32_t *head_map; /* the step's head map (per-head lists) */
  int32_t n_small_heads;
  int32_t select;          /* the step's smallkv_select_t: lists per small head,
                              or per (layer, kv head) for SMALLKV_SELECT_GROUP */
  const int32_t *crit_idx, *marg_idx; /* the step's lists */
  const void *full_k, *full_v;        /* [B][L][Hkv][n_cap][head_dim], 16-byte aligned */
  int64_t rows;                       /* rows per kv head of the new and the old store */
  const void *old_k, *old_v;          /* optional previous store [B][L][Hkv][rows][head_dim] */
  const int32_t *old_k_slot, *old_v_slot; /* its slot maps [B][L][Hkv][n_cap] (all four or none) */
  void *new_k, *new_v;                /* out, [B][L][Hkv][rows][head_dim]; not the old store */
  int32_t *k_slot, *v_slot;           /* out, [B][L][Hkv][n_cap] */
  int32_t *counts;                    /* optional out [B][L][Hkv][2]: |U_K|, |U_V| */
} smallkv_store_t;

/* Bytes of device workspace smallkv_store_update needs for `store`:
 * 2 * units * rows * 4 (each union row's source) + 2 * units * 4 (the union
 * sizes, used when counts is null), units = B * n_layers * n_kv_heads.  Host
 * only.  SMALLKV_EINVAL for a null or malformed descriptor (null required
 * pointers, rows < 1, a group size that does not divide, part of an old
 * store only, the old store passed as the new one, unaligned K/V);
 * SMALLKV_EUNSUPPORTED for head_dim other than 64 or 128, n_cap > 131072 or
 * rows >= 2^30. */
int smallkv_store_workspace_size(const smallkv_store_t *store, size_t *bytes);

/* Enqueue the store maintenance on `stream` (a hipStream_t, null = the
 * default stream).  Two launches: the unions, slot maps and row sources,
 * then the row copies.  The caller owns every buffer, including `ws`
 * (ws_bytes >= smallkv_store_workspace_size, else SMALLKV_EWORKSPACE); the
 * library allocates nothing and does not synchronise.  The same errors as
 * smallkv_store_workspace_size, and SMALLKV_EINVAL when full_k / full_v is
 * host memory that is not pinned and mapped for the device, all returned
 * before anything is enqueued; SMALLKV_EDEVICE if a launch fails.  Calls
 * that share a workspace or outputs must not overlap. */
int smallkv_store_update(const smallkv_store_t *store, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Prefill similarity matching (Method section, "Similarity Matching",
 * Eqs. 1-3; Algorithm 1, prefill branch): computes the head map f that the
 * decode step takes as head_map.
 *
 * For each sequence b, over a window of its first w_b prompt tokens, and for
 * every head of both models (large heads i = layer*n_q_heads + h first, then
 * small heads at L*Hq + j):
 *   A      = the causal prefill attention of the window: row u is the softmax
 *            over tokens v <= u of the logits s[u][v]
 *   F_v    = sum over rows u of A[u][v]                               (Eq. 1)
 *   TopK   = the k_b tokens of largest F (equal F: lower token first)
 *   S(i,j) = |TopK_i n TopK'_j| / |TopK_i u TopK'_j|                  (Eq. 2)
 *   head_map[b][i] = argmax over every small head j of S(i, j),
 *                    the lowest j on ties                             (Eq. 3)
 * The TopK sets and the argmax are integer decisions taken on fp32 values,
 * so every value has one defined evaluation and the result is exact and
 * deterministic:
 *   s[u][v] = the fp32 logit of the conventions above (FMA chain, then scale)
 *   m_u     = max over v <= u of s[u][v]
 *   e[u][v] = exp32(s[u][v] - m_u), fp32 subtraction, with exp32(x) for
 *             x <= 0 defined as: k = rne(x * 0x1.715476p+0), r = fma(-k,
 *             0x1.62e4p-1, x), r = fma(-k, 0x1.7f7d1cp-20, r), then Horner's
 *             rule p = fma(p, r, c) from p = 0x1.a01a02p-13 through
 *             c = 0x1.6c16c2p-10, 0x1.111112p-7, 0x1.555556p-5,
 *             0x1.555556p-3, 0.5, 1, 1 (the Taylor coefficients 1/n!), result
 *             p * 2^k; exp32(x) = 0 for x < -80.  Within 1 ulp of exp.
 *   Z_u     = ((e[u][0] + e[u][1]) + ...) + e[u][u]            (fp32 adds)
 *   F_v     = ((p[v][v] + p[v+1][v]) + ...) + p[w-1][v],  p[u][v] = e[u][v] / Z_u
 *             (correctly rounded fp32 division and adds)
 *   S(i,j) compared as exact integer fractions.
 * The paper matches on 100 to 200 prompt tokens, delaying the matching of a
 * shorter prompt and truncating a longer one ("Method Details"); choosing
 * w_b is the caller's (the window is the prompt's first w_b tokens). */

/* One model's operands over the window.  q and k must be 16-byte aligned. */
typedef struct {
  int32_t n_layers, n_q_heads, n_kv_heads; /* as in smallkv_model_t */
  int32_t head_dim;   /* 64 or 128 */
  int32_t dtype;      /* smallkv_dtype_t of q and k */
  float scale;        /* softmax scale, normally 1/sqrt(head_dim) */
  const void *q;      /* [B][n_layers][n_q_heads][w_cap][head_dim] */
  const void *k;      /* [B][n_layers][n_kv_heads][w_cap][head_dim] */
} smallkv_window_t;

typedef struct {
  int32_t batch;            /* B, 1..65535 */
  int32_t w_cap;            /* window capacity, 1..256 (host) */
  const int32_t *win_len;   /* [B] window tokens w_b, clamped to [1, w_cap] on device */
  const int32_t *top_k;     /* [B] K of Eq. 2, clamped to [1, w_b] on device */
  smallkv_window_t large, small;
  int32_t *head_map;        /* out [B][large.n_layers*large.n_q_heads]: small head ids */
  float *scores;            /* optional out (NULL: skipped) [B][H][w_cap] F of Eq. 1,
                               H = L*Hq + l*Hq_s; entries v >= w_b not written */
  uint64_t *top_bits;       /* optional out [B][H][(w_cap+63)/64]: bit v%64 of word v/64
                               set iff token v is in the head's TopK set */
} smallkv_match_t;

/* Bytes of workspace smallkv_match needs: two fp32 [B][H][w_cap][w_cap]
 * logit matrices plus the TopK bitsets.  Host only. */
int smallkv_match_workspace_size(const smallkv_match_t *match, size_t *bytes);

/* Enqueues the matching on `stream` (four kernel launches). */
int smallkv_match(const smallkv_match_t *match, void *ws, size_t ws_bytes, void *stream);

/* A static string for a status code. */
const char *smallkv_status_string(int status);

/* SMALLKV_ABI_VERSION of the loaded library. */
int smallkv_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SMALLKV_H */
