/* Drives every oracle entry point on small random inputs (ragged lengths,
 * recent tokens, the small model's held rows, slot maps, all three
 * selections, a store update from an old store, the prefill matching) so
 * that an AddressSanitizer / UBSan build of the oracle checks its memory
 * accesses and arithmetic.  Exits non-zero on an unexpected status. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "smallkv_oracle.h"

static uint64_t rng = 0x9e3779b97f4a7c15ull;
static float frand(void) {
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (float)((rng >> 11) * (1.0 / 9007199254740992.0)) * 2.0f - 1.0f;
}
static float *fill(size_t n) {
  float *p = malloc(n * sizeof(float));
  for (size_t i = 0; i < n; ++i) p[i] = frand();
  return p;
}
#define CHECK(x)                                                   \
  do {                                                             \
    int rc_ = (x);                                                 \
    if (rc_ != ORC_OK) {                                           \
      fprintf(stderr, "%s:%d: %s -> %d\n", __FILE__, __LINE__, #x, rc_); \
      return 1;                                                    \
    }                                                              \
  } while (0)

static int one_step(int select, int recent, int held, int slots) {
  const int B = 3, n_cap = 97, l = 2, hqs = 4, hks = 2, ds = 64, L = 2, hq = 8, hk = 2, d = 128;
  const int kc_cap = 20, km_cap = 30, nsh = l * hqs;
  int32_t seq[3] = {1, 50, 97}, kc[3] = {1, 6, 9}, km[3] = {0, 10, 21}, kr[3] = {1, 2, 4};
  const int64_t s_rows = held ? 60 : n_cap;
  float *s_q = fill((size_t)B * l * hqs * ds), *s_k = fill((size_t)B * l * hks * s_rows * ds),
        *s_v = fill((size_t)B * l * hks * s_rows * ds);
  float *l_q = fill((size_t)B * L * hq * d), *l_k = fill((size_t)B * L * hk * n_cap * d),
        *l_v = fill((size_t)B * L * hk * n_cap * d);
  int32_t hm[16];
  for (int i = 0; i < L * hq; ++i) hm[i] = (i * 5) % nsh;
  int32_t s_held[3] = {1, 30, 60};
  int32_t *rpos = malloc(sizeof(int32_t) * B * l * hks * s_rows);
  for (int b = 0; b < B; ++b)  /* held rows name positions 0.. (strictly ascending, < seq_len) */
    for (int u = 0; u < l * hks; ++u)
      for (int r = 0; r < s_rows; ++r)
        rpos[((size_t)b * l * hks + u) * s_rows + r] = r < s_held[b] ? r : -1;
  int32_t *ks = NULL, *vs = NULL;
  if (slots) {
    ks = malloc(sizeof(int32_t) * B * L * hk * n_cap);
    vs = malloc(sizeof(int32_t) * B * L * hk * n_cap);
    for (int i = 0; i < B * L * hk * n_cap; ++i) ks[i] = vs[i] = i % n_cap;
  }
  const int lrows = select == ORC_SELECT_GROUP ? L * hk : nsh;
  const int prows = select == ORC_SELECT_GROUP ? L * hq : nsh;
  float *acc = calloc((size_t)B * nsh * n_cap, sizeof(float));
  orc_step_in in;
  memset(&in, 0, sizeof in);
  in.batch = B; in.n_cap = n_cap; in.kc_cap = kc_cap; in.km_cap = km_cap;
  in.seq_len = seq; in.k_crit = kc; in.k_marg = km; in.k_recent = recent ? kr : NULL;
  in.s_layers = l; in.s_q_heads = hqs; in.s_kv_heads = hks; in.s_dim = ds; in.s_scale = 0.125f;
  in.s_q = s_q; in.s_k = s_k; in.s_v = s_v; in.s_rows = s_rows;
  in.s_held = held ? s_held : NULL; in.s_row_pos = held ? rpos : NULL;
  in.l_layers = L; in.l_q_heads = hq; in.l_kv_heads = hk; in.l_dim = d; in.l_scale = 0.0884f;
  in.l_rows = n_cap; in.l_q = l_q; in.l_k = l_k; in.l_v = l_v; in.k_slot = ks; in.v_slot = vs;
  in.head_map = hm; in.mode = 0; in.select = select; in.acc = acc;
  orc_step_out out;
  out.logits = malloc(sizeof(float) * B * nsh * n_cap);
  out.row_max = malloc(sizeof(double) * B * nsh);
  out.row_sum = malloc(sizeof(double) * B * nsh);
  out.small_out = malloc(sizeof(double) * B * nsh * ds);
  out.crit = malloc(sizeof(int32_t) * B * lrows * kc_cap);
  out.marg = malloc(sizeof(int32_t) * B * lrows * km_cap);
  out.marg_prob = malloc(sizeof(double) * B * prows * km_cap);
  out.mass = malloc(sizeof(double) * B * prows * 2);
  out.large_out = malloc(sizeof(double) * B * L * hq * d);
  for (int mode = 0; mode < 5; ++mode) {
    in.mode = mode;
    CHECK(orc_step(&in, &out));
  }
  if (!held) {  /* the store from this step's lists, then again from that store */
    const int64_t rows = 40;
    orc_store_in si;
    memset(&si, 0, sizeof si);
    si.batch = B; si.n_cap = n_cap; si.layers = L; si.q_heads = hq; si.kv_heads = hk; si.dim = d;
    si.select = select == ORC_SELECT_GROUP ? 1 : 0; si.n_small_heads = nsh;
    si.kc_cap = kc_cap; si.km_cap = km_cap; si.rows = rows; si.seq_len = seq; si.head_map = hm;
    si.crit = out.crit; si.marg = out.marg; si.full_k = l_k; si.full_v = l_v;
    const size_t nst = (size_t)B * L * hk * rows * d, nsl = (size_t)B * L * hk * n_cap;
    float *k0 = calloc(nst, 4), *v0 = calloc(nst, 4), *k1 = calloc(nst, 4), *v1 = calloc(nst, 4);
    int32_t *ks0 = malloc(nsl * 4), *vs0 = malloc(nsl * 4), *ks1 = malloc(nsl * 4),
            *vs1 = malloc(nsl * 4), *cnt = malloc(sizeof(int32_t) * B * L * hk * 2);
    for (size_t i = 0; i < nsl; ++i) ks0[i] = vs0[i] = ks1[i] = vs1[i] = -1;
    CHECK(orc_store_update(&si, k0, v0, ks0, vs0, cnt));
    si.old_k = k0; si.old_v = v0; si.old_k_slot = ks0; si.old_v_slot = vs0;
    CHECK(orc_store_update(&si, k1, v1, ks1, vs1, cnt));
    free(k0); free(v0); free(k1); free(v1); free(ks0); free(vs0); free(ks1); free(vs1); free(cnt);
  }
  free(s_q); free(s_k); free(s_v); free(l_q); free(l_k); free(l_v); free(rpos); free(ks); free(vs);
  free(acc); free(out.logits); free(out.row_max); free(out.row_sum); free(out.small_out);
  free(out.crit); free(out.marg); free(out.marg_prob); free(out.mass); free(out.large_out);
  return 0;
}

static int one_match(void) {
  const int B = 2, w_cap = 70, L = 2, hq = 4, hk = 2, d = 128, l = 2, hqs = 4, hks = 2, ds = 64;
  int32_t win[2] = {1, 70}, topk[2] = {1, 7};
  float *lq = fill((size_t)B * L * hq * w_cap * d), *lk = fill((size_t)B * L * hk * w_cap * d);
  float *sq = fill((size_t)B * l * hqs * w_cap * ds), *sk = fill((size_t)B * l * hks * w_cap * ds);
  orc_match_in m;
  m.batch = B; m.w_cap = w_cap; m.win_len = win; m.top_k = topk;
  m.large = (orc_window){L, hq, hk, d, 0.0884f, lq, lk};
  m.small = (orc_window){l, hqs, hks, ds, 0.125f, sq, sk};
  const int H = L * hq + l * hqs;
  int32_t *hm = malloc(sizeof(int32_t) * B * L * hq);
  float *sc = malloc(sizeof(float) * B * H * w_cap);
  uint8_t *top = malloc((size_t)B * H * w_cap);
  CHECK(orc_match(&m, hm, sc, top));
  free(lq); free(lk); free(sq); free(sk); free(hm); free(sc); free(top);
  return 0;
}

int main(void) {
  for (int select = 0; select < 3; ++select)
    for (int recent = 0; recent < 2; ++recent)
      if (one_step(select, recent, 0, select != ORC_SELECT_ACCUM)) return 1;
  if (one_step(ORC_SELECT_HEAD, 1, 1, 0)) return 1;
  if (one_match()) return 1;
  puts("oracle driver ok");
  return 0;
}
