// Host-side launchers of the SmallKV kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "smallkv.h"

namespace smallkv {

// Split-K plan of stage 1: each workgroup covers `chunk` tokens of one
// (sequence, layer, kv head) unit; n_split chunks cover n_cap.
struct SmallPlan {
  int tile;      // tokens staged in LDS per iteration
  int chunk;     // tokens per workgroup (multiple of tile)
  int n_split;   // workgroups per unit
  int gp;        // padded query-group size (4, 8 or 16)
  size_t ws_bytes;
};

SmallPlan plan_small(const smallkv_batch_t &b, const smallkv_model_t &m);

hipError_t launch_small_attn(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                             float *row_max, float *row_sum, float *ws, const SmallPlan &p,
                             hipStream_t st);

// Stage 1 without the merge: per-chunk records only (smallkv_step merges
// them inside the partition kernel).
hipError_t launch_small_split(const smallkv_batch_t &b, const smallkv_model_t &m, float *logits,
                              float *ws, const SmallPlan &p, hipStream_t st);

// List offsets: per partition row and 256-token boundary t < N_b, the
// (critical, marginal) entries with a token below t, [rows][list_blocks].
inline int list_blocks(const smallkv_batch_t &b) { return (b.n_cap + 255) / 256; }
inline size_t list_offsets_bytes(const smallkv_batch_t &b, int n_small_heads) {
  return (size_t)b.batch * n_small_heads * list_blocks(b) * sizeof(int2);
}

// Stage 2 fused with stage 1's merge: writes row_max, row_sum and the small
// model's output, then partitions; also the list offsets when tab is set.
// `b` is the batch as stages 1-2 see it (with the small model's own
// eviction: held rows); with m.row_pos the lists name row_pos[row], clamped
// below tok_len[b] (the sequences' token counts, capacity tok_cap).
hipError_t launch_merge_partition(const smallkv_batch_t &b, const smallkv_model_t &m,
                                  const SmallPlan &p, const float *ws, const float *logits,
                                  float *row_max, float *row_sum, int32_t *crit, int32_t *marg,
                                  float *marg_prob, float *mass, int2 *tab,
                                  const int32_t *tok_len, int tok_cap, hipStream_t st);

// Stage 2 alone; `held` (or null): the small model whose held rows the
// rows are (b is then the batch as stages 1-2 see it), named by its row_pos.
hipError_t launch_partition(const smallkv_batch_t &b, int n_small_heads, const float *logits,
                            const float *row_max, const float *row_sum, int32_t *crit,
                            int32_t *marg, float *marg_prob, float *mass,
                            const smallkv_model_t *held, const int32_t *tok_len, int tok_cap,
                            hipStream_t st);

// Largest kc_cap the per-head hybrid kernel keeps in LDS.
constexpr int kHybridMaxCrit = 12288;

// Plan of the grouped stage-3 kernel (bf16, head_dim 128, group <= 8): each
// (sequence, layer, kv head) is cut into n_split token ranges of `span`
// tokens; with more than one, the workspace holds a record per range and
// query head.
struct GroupPlan {
  bool use;
  int n_split, span;
  size_t ws_bytes;
};

// n_run: the large layers one launch runs (-1: all of m's)
GroupPlan plan_group(const smallkv_batch_t &b, const smallkv_model_t &m, int n_small_heads,
                     int n_run = -1);

// tab: the partition's list offsets, or null; with them the list cursors at
// the start of each token range are read instead of searched.  Layers
// [layer0, layer0 + nl) of m run (m describes the whole stack).  group_sel:
// the lists are per (sequence, layer, kv head) and marg_prob / mass per
// large query head (group selection); otherwise all are per small head f(i).
hipError_t launch_hybrid_group(const smallkv_batch_t &b, const smallkv_model_t &m,
                               const int32_t *head_map, int n_small_heads, const int32_t *crit,
                               const int32_t *marg, const float *marg_prob, const float *mass,
                               int mode, const GroupPlan &p, float *ws, const int2 *tab,
                               bool group_sel, int layer0, int nl, hipStream_t st);

// Group selection (the query heads of a kv head share one selection):
// workspace offsets of its intermediates, placed from `offset` on.
struct GroupLayout {
  size_t zq, keys, key_max, part_mp, part_mass, end;
};
GroupLayout group_layout(const smallkv_batch_t &b, const smallkv_model_t &small,
                         const smallkv_model_t &large, size_t offset, bool accum = false);
// Accumulated-score selection (per small head): acc [B][nsh][n_cap] += this
// step's probabilities, then the partition ranks acc; weights are this
// step's p'.  Lists and weights in the per-head layout.
hipError_t launch_accum_select(const smallkv_batch_t &b, const smallkv_model_t &small,
                               const float *logits, const float *row_max, const float *row_sum,
                               float *acc, int32_t *crit, int32_t *marg, float *marg_prob,
                               float *mass, void *ws, const GroupLayout &lay, hipStream_t st);
// From stage 1's logits and statistics: group lists crit/marg
// [B][L*Hkv][cap] and per-large-head marg_prob/mass [B][L*Hq][...].
hipError_t launch_group_select(const smallkv_batch_t &b, const smallkv_model_t &small,
                               const smallkv_model_t &large, const int32_t *head_map,
                               const float *logits, const float *row_max, const float *row_sum,
                               int32_t *crit, int32_t *marg, float *marg_prob, float *mass,
                               void *ws, const GroupLayout &lay, hipStream_t st);
// The partition over group keys (rows [B][group_rows][n_cap], row maxima).
hipError_t launch_group_partition(const smallkv_batch_t &b, int group_rows, const float *keys,
                                  const float *key_max, int32_t *crit, int32_t *marg,
                                  float *marg_prob, float *mass, int bins_per_binade,
                                  hipStream_t st);

// Retained-store maintenance: workspace bytes (the unions' token lists and
// sizes) and the two launches.
size_t store_workspace(const smallkv_store_t &s);
hipError_t launch_store_update(const smallkv_store_t &s, void *ws, hipStream_t st);

// Workspace of the prefill matching: the logit matrix S of every head
// ([B][H][w_cap][ld] fp32, ld = w_cap rounded up to 4), the row maxima per
// 64-token tile column ([B][H][w_cap][nt] fp32), each row's (max, sum)
// ([B][H][w_cap] float2), then the TopK bitsets ([B][H][nw] words of 64
// tokens).
struct MatchLayout {
  int nw, nt, ld;
  size_t pmax_offset, mz_offset, bits_offset, total;
};
MatchLayout match_layout(const smallkv_match_t &m);
hipError_t launch_match(const smallkv_match_t &m, void *ws, hipStream_t st);

hipError_t launch_hybrid(const smallkv_batch_t &b, const smallkv_model_t &m,
                         const int32_t *head_map, int n_small_heads, const int32_t *crit,
                         const int32_t *marg, const float *marg_prob, const float *mass,
                         int mode, bool group_sel, int layer0, int nl, hipStream_t st);

}  // namespace smallkv
