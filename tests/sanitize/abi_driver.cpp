// Drives the host side of every C-ABI entry point (descriptor checks and
// workspace planning) with descriptors whose pointers are never
// dereferenced, so that an AddressSanitizer / UBSan build of the library's
// host code checks them.  Every call here returns before anything would be
// enqueued.  Exits non-zero on an unexpected status.
#include <stdio.h>
#include <string.h>

#include "smallkv.h"

static int fails = 0;
#define EXPECT(call, want)                                                      \
  do {                                                                          \
    const int rc_ = (call);                                                     \
    if (rc_ != (want)) {                                                        \
      fprintf(stderr, "%s:%d: %s -> %d, want %d\n", __FILE__, __LINE__, #call, rc_, \
              (int)(want));                                                     \
      ++fails;                                                                  \
    }                                                                           \
  } while (0)

static void *P = reinterpret_cast<void *>(0x1000);
static const int32_t *IP = reinterpret_cast<const int32_t *>(0x1000);

struct Shape { int B, n, kc, km, l, hqs, hks, ds, L, hq, hk, d, dtype; };

static smallkv_step_t step_of(const Shape &s, int select) {
  smallkv_step_t st;
  memset(&st, 0, sizeof st);
  st.batch = {s.B, s.n, IP, IP, IP, nullptr, s.kc, s.km};
  st.small = {s.l, s.hqs, s.hks, s.ds, s.dtype, 0.125f, P, P, P, s.n, nullptr, nullptr, P,
              nullptr, nullptr};
  st.large = {s.L, s.hq, s.hk, s.d, s.dtype, 0.088f, P, P, P, s.n, nullptr, nullptr, P,
              nullptr, nullptr};
  st.head_map = IP;
  st.logits = st.row_max = st.row_sum = static_cast<float *>(P);
  st.crit_idx = st.marg_idx = static_cast<int32_t *>(P);
  st.marg_prob = st.mass = static_cast<float *>(P);
  st.select = select;
  st.acc_score = static_cast<float *>(P);
  return st;
}

int main() {
  const Shape shapes[] = {
      {1, 512, 64, 128, 1, 14, 2, 64, 1, 28, 4, 128, SMALLKV_F32},       // tiny fp32
      {1, 8192, 819, 1638, 24, 14, 2, 64, 28, 28, 4, 128, SMALLKV_BF16},  // Qwen2-7B + 0.5B
      {16, 32768, 1638, 4915, 16, 32, 8, 64, 32, 32, 8, 128, SMALLKV_BF16},
      {64, 4352, 870, 1305, 24, 14, 2, 64, 28, 28, 4, 128, SMALLKV_BF16},
      {2, 65536, 1310, 5242, 24, 14, 2, 64, 80, 64, 8, 128, SMALLKV_BF16},
      {3, 1800, 180, 360, 2, 8, 2, 64, 3, 12, 4, 128, SMALLKV_BF16},
  };
  for (const Shape &s : shapes) {
    for (int select = 0; select < 3; ++select) {
      smallkv_step_t st = step_of(s, select);
      size_t ws = 0;
      EXPECT(smallkv_workspace_size(&st, &ws), SMALLKV_OK);
      EXPECT(smallkv_step(&st, nullptr, 0, nullptr), ws ? SMALLKV_EWORKSPACE : SMALLKV_OK);
      if (ws) EXPECT(smallkv_step(&st, P, ws - 1, nullptr), SMALLKV_EWORKSPACE);
      smallkv_step_t bad = st;
      bad.mode = 9;
      EXPECT(smallkv_step_noalloc(&bad, nullptr), SMALLKV_EINVAL);
      bad = st;
      bad.small.head_dim = 96;
      EXPECT(smallkv_workspace_size(&bad, &ws), SMALLKV_EUNSUPPORTED);
      bad = st;
      bad.large.k_slot = IP;  // one slot map without the other
      EXPECT(smallkv_step(&bad, P, 1, nullptr), SMALLKV_EINVAL);
    }
    smallkv_step_t st = step_of(s, 0);
    size_t w1 = 0;
    EXPECT(smallkv_hybrid_attn_workspace_size(&st.batch, &st.large, 1, s.l * s.hqs, &w1),
           SMALLKV_OK);
    EXPECT(smallkv_hybrid_attn_workspace_size(&st.batch, &st.large, s.L + 1, s.l * s.hqs, &w1),
           SMALLKV_EINVAL);
    EXPECT(smallkv_hybrid_attn_layers(&st.batch, &st.large, s.L, 1, IP, s.l * s.hqs, IP, IP,
                                      static_cast<const float *>(P), static_cast<const float *>(P),
                                      0, 0, P, 1u << 30, nullptr),
           SMALLKV_EINVAL);
    size_t wg = 0, wa = 0;
    EXPECT(smallkv_group_select_workspace_size(&st.batch, &st.small, &st.large, &wg), SMALLKV_OK);
    EXPECT(smallkv_accum_select_workspace_size(&st.batch, &st.small, &wa), SMALLKV_OK);
    EXPECT(smallkv_partition(&st.batch, nullptr, 0, st.logits, st.row_max, st.row_sum,
                             st.crit_idx, st.marg_idx, st.marg_prob, st.mass, nullptr, 0, nullptr),
           SMALLKV_EINVAL);
    // the retained store of this step's shapes
    smallkv_store_t so;
    memset(&so, 0, sizeof so);
    so.batch = st.batch;
    so.n_layers = s.L; so.n_q_heads = s.hq; so.n_kv_heads = s.hk; so.head_dim = s.d;
    so.dtype = s.dtype; so.head_map = IP; so.n_small_heads = s.l * s.hqs; so.select = 0;
    so.crit_idx = IP; so.marg_idx = IP; so.full_k = P; so.full_v = P; so.rows = 256;
    so.new_k = reinterpret_cast<void *>(0x2000); so.new_v = reinterpret_cast<void *>(0x3000);
    so.k_slot = reinterpret_cast<int32_t *>(0x4000); so.v_slot = reinterpret_cast<int32_t *>(0x5000);
    size_t wst = 0;
    EXPECT(smallkv_store_workspace_size(&so, &wst), s.n > 131072 ? SMALLKV_EUNSUPPORTED : SMALLKV_OK);
    EXPECT(smallkv_store_update(&so, nullptr, 0, nullptr), SMALLKV_EWORKSPACE);
    so.old_k = P;  // part of an old store only
    EXPECT(smallkv_store_workspace_size(&so, &wst), SMALLKV_EINVAL);
  }
  // prefill matching
  smallkv_match_t m;
  memset(&m, 0, sizeof m);
  m.batch = 2; m.w_cap = 200; m.win_len = IP; m.top_k = IP;
  m.large = {28, 28, 4, 128, SMALLKV_BF16, 0.088f, P, P};
  m.small = {24, 14, 2, 64, SMALLKV_BF16, 0.125f, P, P};
  m.head_map = static_cast<int32_t *>(P);
  size_t wm = 0;
  EXPECT(smallkv_match_workspace_size(&m, &wm), SMALLKV_OK);
  EXPECT(smallkv_match(&m, nullptr, 0, nullptr), SMALLKV_EWORKSPACE);
  m.w_cap = 257;
  EXPECT(smallkv_match_workspace_size(&m, &wm), SMALLKV_EUNSUPPORTED);
  EXPECT(smallkv_abi_version(), SMALLKV_ABI_VERSION);
  for (int c = -5; c <= 1; ++c)
    if (!smallkv_status_string(c)) ++fails;
  if (fails) return 1;
  puts("abi driver ok");
  return 0;
}
