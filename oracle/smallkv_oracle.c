/*
 * smallkv_oracle.c -- plain, slow, single-threaded CPU oracle of SmallKV's
 * per-decode-step compensated attention (arXiv 2508.02751).
 *
 * TEST INFRASTRUCTURE ONLY: called by the test suite, the smoke check and
 * the benchmark's CPU-baseline leg; never by the product path.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fPIC -shared ... -lm.
 * fp contraction is off so that no expression below is silently fused; the
 * only fused multiply-adds are the explicit fmaf calls of orc_logit, which
 * are correctly rounded IEEE-754 operations.
 */
#include "smallkv_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- keys -- */

/* Ranking key: the small model's logit for one token (the decode row of the
 * attention matrix before its softmax, Method section, "Similarity
 * Matching").  The paper does not fix an evaluation order; the order used
 * here is a sequential fp32 FMA chain over the head dimension, then one fp32
 * multiply by the softmax scale 1/sqrt(d_h).  Ranking on the logit is the
 * same as ranking on the exact probability exp(s - m)/Z, since exp is
 * monotone, and avoids ties created by rounding the probability. */
float orc_logit(int d, float scale, const float *q, const float *k) {
  float a = 0.0f;
  for (int c = 0; c < d; ++c) a = fmaf(q[c], k[c], a);
  float s = a * scale;
  if (s == 0.0f) s = 0.0f; /* canonical +0 */
  return s;
}

uint32_t orc_key(float s) {
  uint32_t u;
  if (s == 0.0f) s = 0.0f;
  memcpy(&u, &s, sizeof u);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

/* ------------------------------------------------------------ stage 1 -- */

/* Full decode attention of the small model over its uncompressed cache
 * (Algorithm 1, decode branch: the small model's forward updates A'_j; the
 * selection of the "Saliency Shift Compensation" paragraph uses the full
 * small cache C^s_all). */
int orc_small_head(int n, int d, float scale, const float *q, const float *K,
                   const float *V, float *logits, double *m_out, double *Z_out,
                   double *O) {
  if (n < 1 || d < 1) return ORC_EINVAL;
  double m = -INFINITY;
  for (int t = 0; t < n; ++t) {
    float s = orc_logit(d, scale, q, K + (size_t)t * d);
    if (!isfinite(s)) return ORC_ENONFINITE;
    logits[t] = s;
    if ((double)s > m) m = (double)s;
  }
  double Z = 0.0;
  for (int t = 0; t < n; ++t) Z += exp((double)logits[t] - m);
  for (int c = 0; c < d; ++c) O[c] = 0.0;
  for (int t = 0; t < n; ++t) {
    double p = exp((double)logits[t] - m) / Z;
    const float *v = V + (size_t)t * d;
    for (int c = 0; c < d; ++c) O[c] += p * (double)v[c];
  }
  *m_out = m;
  *Z_out = Z;
  return ORC_OK;
}

/* ------------------------------------------------------------ stage 2 -- */

typedef struct {
  uint32_t key;
  int32_t idx;
} orc_item;

/* Total order: larger key first; equal keys by lower token index first. */
static int orc_rank_cmp(const void *a, const void *b) {
  const orc_item *x = (const orc_item *)a, *y = (const orc_item *)b;
  if (x->key != y->key) return x->key > y->key ? -1 : 1;
  return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);
}

static int orc_int_cmp(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* Eq. 4 read as "keep the top-scored tokens" (the printed argmax would evict
 * the most important one, contradicting Eq. 6 and the pseudocode's topk);
 * Eq. 6: TopK gives the critical set, Top(P-K) the next P-K tokens of the
 * same order (the marginal set), everything else is evicted.
 * Recent tokens (experimental setup: a fixed critical : recent : marginal
 * split of the budget, 2 : 1 : 2): the last r = min(k_recent, n) tokens are
 * kept whatever their score, like critical ones; only the n - r older
 * tokens are ranked for the critical and marginal budgets. */
int orc_partition(int n, int k_crit, int k_marg, int k_recent, const float *logits,
                  double m, double Z, int32_t *crit, int kc_cap, int32_t *marg,
                  double *marg_prob, int km_cap, double *mass, int *n_crit,
                  int *n_marg) {
  if (n < 1 || k_crit < 1 || k_marg < 0 || k_recent < 0) return ORC_EINVAL;
  const int r = k_recent < n ? k_recent : n;
  const int older = n - r;
  const int ntop = k_crit < older ? k_crit : older;
  const int nm = k_marg < older - ntop ? k_marg : older - ntop;
  const int nc = ntop + r;
  if (nc > kc_cap || nm > km_cap) return ORC_EINVAL;

  for (int t = 0; t < n; ++t)
    if (!isfinite(logits[t])) return ORC_ENONFINITE;
  orc_item *items = (orc_item *)malloc((size_t)(older > 0 ? older : 1) * sizeof *items);
  if (!items) return ORC_EINVAL;
  for (int t = 0; t < older; ++t) {
    items[t].key = orc_key(logits[t]);
    items[t].idx = t;
  }
  qsort(items, (size_t)older, sizeof *items, orc_rank_cmp);

  for (int i = 0; i < kc_cap; ++i) crit[i] = -1;
  for (int i = 0; i < km_cap; ++i) {
    marg[i] = -1;
    marg_prob[i] = 0.0;
  }
  for (int i = 0; i < ntop; ++i) crit[i] = items[i].idx;
  for (int i = 0; i < r; ++i) crit[ntop + i] = older + i;
  for (int i = 0; i < nm; ++i) marg[i] = items[ntop + i].idx;
  free(items);
  qsort(crit, (size_t)nc, sizeof *crit, orc_int_cmp);
  qsort(marg, (size_t)nm, sizeof *marg, orc_int_cmp);

  double sc = 0.0, sm = 0.0;
  for (int i = 0; i < nc; ++i) sc += exp((double)logits[crit[i]] - m) / Z;
  for (int i = 0; i < nm; ++i) {
    marg_prob[i] = exp((double)logits[marg[i]] - m) / Z;
    sm += marg_prob[i];
  }
  mass[0] = sc;
  mass[1] = sm;
  *n_crit = nc;
  *n_marg = nm;
  return ORC_OK;
}

/* ------------------------------------------------------------ stage 3 -- */

static void orc_alphas(int mode, double sc, double sm, double *ac, double *am) {
  switch (mode) {
    case ORC_NORM_NONE:
      *ac = 1.0;
      *am = 1.0;
      break;
    case ORC_NORM_SLM_CRIT:
      *ac = sc;
      *am = 1.0;
      break;
    case ORC_NORM_RETAINED:
      *ac = sc / (sc + sm);
      *am = 1.0 / (sc + sm);
      break;
    case ORC_NORM_MARG_FILL:
      *ac = sc;
      *am = sm > 0.0 ? (1.0 - sc) / sm : 0.0;
      break;
    default: /* ORC_NORM_REMAINING */
      *ac = 1.0 - sm;
      *am = 1.0;
      break;
  }
}

/* Eq. 6 for one large head i: exact attention on the critical tokens
 * (Algorithm 1, "Calculate attention output O_c of critical tokens"), the
 * small head f(i)'s probabilities times the large model's V rows for the
 * marginal tokens ("O_m ... using Eq. (6)"), evicted tokens weight 0, and
 * the attention output O_c + O_m with the weights of `mode`. */
int orc_hybrid_head(int d, float scale, const float *q, const float *K,
                    const float *V, const int32_t *k_slot,
                    const int32_t *v_slot, int n_crit, const int32_t *crit,
                    int n_marg, const int32_t *marg, const double *marg_prob,
                    const double *mass, int mode, double *O) {
  if (d < 1 || n_crit < 1 || n_marg < 0) return ORC_EINVAL;
  if (mode < ORC_NORM_REMAINING || mode > ORC_NORM_MARG_FILL) return ORC_EINVAL;

  double *s = (double *)malloc((size_t)n_crit * sizeof *s);
  if (!s) return ORC_EINVAL;
  double mx = -INFINITY;
  for (int i = 0; i < n_crit; ++i) {
    int32_t t = crit[i];
    int32_t r = k_slot ? k_slot[t] : t;
    if (t < 0 || r < 0) {
      free(s);
      return ORC_EINVAL;
    }
    const float *k = K + (size_t)r * d;
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += (double)q[c] * (double)k[c];
    s[i] = (double)scale * acc;
    if (!isfinite(s[i])) {
      free(s);
      return ORC_ENONFINITE;
    }
    if (s[i] > mx) mx = s[i];
  }

  double zc = 0.0;
  for (int i = 0; i < n_crit; ++i) zc += exp(s[i] - mx);

  double *oc = (double *)calloc((size_t)d, sizeof *oc);
  double *om = (double *)calloc((size_t)d, sizeof *om);
  if (!oc || !om) {
    free(s);
    free(oc);
    free(om);
    return ORC_EINVAL;
  }
  int rc = ORC_OK;
  for (int i = 0; i < n_crit && rc == ORC_OK; ++i) {
    int32_t t = crit[i];
    int32_t r = v_slot ? v_slot[t] : t;
    if (r < 0) {
      rc = ORC_EINVAL;
      break;
    }
    double w = exp(s[i] - mx) / zc;
    const float *v = V + (size_t)r * d;
    for (int c = 0; c < d; ++c) oc[c] += w * (double)v[c];
  }
  for (int i = 0; i < n_marg && rc == ORC_OK; ++i) {
    int32_t t = marg[i];
    int32_t r = t < 0 ? -1 : (v_slot ? v_slot[t] : t);
    if (r < 0) {
      rc = ORC_EINVAL;
      break;
    }
    const float *v = V + (size_t)r * d;
    for (int c = 0; c < d; ++c) om[c] += marg_prob[i] * (double)v[c];
  }
  if (rc == ORC_OK) {
    double ac, am;
    orc_alphas(mode, mass[0], mass[1], &ac, &am);
    for (int c = 0; c < d; ++c) O[c] = ac * oc[c] + am * om[c];
  }
  free(s);
  free(oc);
  free(om);
  return rc;
}

/* ---------------------------------------------------------- one step -- */

/* Algorithm 1, decode branch, restricted to attention: the small model's
 * attention over all its layers, the selection for every small head, then
 * every large layer's compensated attention through the head map. */
/* ---------------------------------------------------- group selection -- */

/* The implementation pseudocode selects the large model's cache with the
 * top of the mapped small-model attention summed (`.sum.topk`); the cache is
 * stored per kv head, so the query heads sharing one are summed.  The sum is
 * an fp32 value that decides integers: it is evaluated in one defined way,
 * with orc_exp and a normaliser that is an exact fixed-point sum. */
float orc_zq(int n, const float *logits, float m) {
  uint64_t z = 0;
  for (int t = 0; t < n; ++t) {
    const float e = orc_exp(logits[t] - m);
    z += (uint64_t)ldexp((double)e, 40); /* exact scaling, then truncation */
  }
  return ldexpf((float)z, -40);
}

void orc_group_key(int n, int g, const float *const *logits, const float *m, const float *zq,
                   float *F) {
  for (int t = 0; t < n; ++t) {
    float f = 0.0f;
    for (int h = 0; h < g; ++h) f = f + orc_exp(logits[h][t] - m[h]) / zq[h];
    F[t] = f;
  }
}

/* Group mode of orc_step for sequence b, after stage 1 of every small head:
 * one selection per (large layer, kv head) from orc_group_key, the weights of
 * each large head from its own small head, then stage 3. */
static int group_step(const orc_step_in *in, const orc_step_out *out, int b, int n, int ns,
                      int64_t srows, const double *ms, const double *zs) {
  const int l = in->s_layers, hqs = in->s_q_heads;
  const int L = in->l_layers, hq = in->l_q_heads, hk = in->l_kv_heads, d = in->l_dim;
  const int nsh = l * hqs, gl = hq / hk;
  if (in->s_held) return ORC_EINVAL; /* group keys need every token scored */
  (void)srows;
  float *F = (float *)malloc(sizeof(float) * (size_t)n);
  float *zq = (float *)malloc(sizeof(float) * (size_t)nsh);
  float *mf = (float *)malloc(sizeof(float) * (size_t)gl);
  float *zg = (float *)malloc(sizeof(float) * (size_t)gl);
  const float **rows = (const float **)malloc(sizeof(float *) * (size_t)gl);
  double *scratch = (double *)malloc(sizeof(double) * (size_t)(in->km_cap > 0 ? in->km_cap : 1));
  int rc = (F && zq && mf && zg && rows && scratch) ? ORC_OK : ORC_EINVAL;
  for (int j = 0; j < nsh && rc == ORC_OK; ++j)
    zq[j] = orc_zq(n, out->logits + ((size_t)b * nsh + j) * (size_t)in->n_cap, (float)ms[j]);
  for (int li = 0; li < L && rc == ORC_OK; ++li)
    for (int g = 0; g < hk && rc == ORC_OK; ++g) {
      for (int h = 0; h < gl; ++h) {
        const int j = in->head_map[li * hq + g * gl + h];
        if (j < 0 || j >= nsh) {
          rc = ORC_EINVAL;
          break;
        }
        rows[h] = out->logits + ((size_t)b * nsh + j) * (size_t)in->n_cap;
        mf[h] = (float)ms[j];
        zg[h] = zq[j];
      }
      if (rc) break;
      orc_group_key(n, gl, rows, mf, zg, F);
      const size_t grow = ((size_t)b * L + li) * hk + g;
      int32_t *crit = out->crit + grow * in->kc_cap, *marg = out->marg + grow * in->km_cap;
      double mass_g[2];
      int nc, nm;
      /* the lists only: the p' this computes from F are not used */
      rc = orc_partition(n, in->k_crit[b], in->k_marg[b], in->k_recent ? in->k_recent[b] : 0, F,
                         0.0, 1.0, crit, in->kc_cap, marg, scratch, in->km_cap, mass_g, &nc, &nm);
      if (rc) break;
      for (int h = 0; h < gl && rc == ORC_OK; ++h) {
        const int hh = g * gl + h, j = in->head_map[li * hq + hh];
        const float *lg = out->logits + ((size_t)b * nsh + j) * (size_t)in->n_cap;
        const size_t prow = ((size_t)b * L + li) * hq + hh;
        double *mp = out->marg_prob + prow * in->km_cap, *mass = out->mass + prow * 2;
        mass[0] = mass[1] = 0.0;
        for (int i = 0; i < nc; ++i) mass[0] += exp((double)lg[crit[i]] - ms[j]) / zs[j];
        for (int i = 0; i < in->km_cap; ++i) {
          mp[i] = i < nm ? exp((double)lg[marg[i]] - ms[j]) / zs[j] : 0.0;
          mass[1] += mp[i];
        }
        const size_t unit = ((size_t)b * L + li) * hk + g;
        const size_t kv = unit * (size_t)in->l_rows * d;
        const int32_t *ks = in->k_slot ? in->k_slot + unit * in->n_cap : NULL;
        const int32_t *vs = in->v_slot ? in->v_slot + unit * in->n_cap : NULL;
        rc = orc_hybrid_head(d, in->l_scale, in->l_q + prow * d, in->l_k + kv, in->l_v + kv, ks,
                             vs, nc, crit, nm, marg, mp, mass, in->mode,
                             out->large_out + prow * d);
      }
    }
  (void)ns;
  free(F);
  free(zq);
  free(mf);
  free(zg);
  free(rows);
  free(scratch);
  return rc;
}

int orc_step(const orc_step_in *in, const orc_step_out *out) {
  const int B = in->batch, ncap = in->n_cap;
  const int l = in->s_layers, hqs = in->s_q_heads, hks = in->s_kv_heads,
            ds = in->s_dim;
  const int L = in->l_layers, hq = in->l_q_heads, hk = in->l_kv_heads,
            d = in->l_dim;
  if (B < 1 || ncap < 1 || hks < 1 || hk < 1 || hqs % hks || hq % hk)
    return ORC_EINVAL;
  const int gs = hqs / hks, gl = hq / hk;
  const int nsh = l * hqs; /* small heads per sequence */

  double *ms = (double *)malloc((size_t)nsh * sizeof *ms);
  double *zs = (double *)malloc((size_t)nsh * sizeof *zs);
  int *nc = (int *)malloc((size_t)nsh * sizeof *nc);
  int *nm = (int *)malloc((size_t)nsh * sizeof *nm);
  if (!ms || !zs || !nc || !nm) {
    free(ms);
    free(zs);
    free(nc);
    free(nm);
    return ORC_EINVAL;
  }
  int rc = ORC_OK;
  for (int b = 0; b < B && rc == ORC_OK; ++b) {
    const int n = in->seq_len[b];
    if (n < 1 || n > ncap) {
      rc = ORC_EINVAL;
      break;
    }
    /* The small model's cache: every token (row t = token t), or after its
     * own eviction the held rows r < held[b] of token positions row_pos[r]
     * (the small model's KV compression, "Implementation Optimization" (2)).
     * Stages 1-2 run over the rows; the lists name token positions. */
    const int64_t srows = in->s_held ? in->s_rows : ncap;
    const int ns = in->s_held ? in->s_held[b] : n;
    if (ns < 1 || ns > n || ns > srows) {
      rc = ORC_EINVAL;
      break;
    }
    /* stage 1 and stage 2 for every small head j = layer*Hq_s + head */
    for (int j = 0; j < nsh && rc == ORC_OK; ++j) {
      const int layer = j / hqs, h = j % hqs, g = h / gs;
      const size_t row = (size_t)b * nsh + j;
      const float *q = in->s_q + row * ds;
      const size_t unit = ((size_t)b * l + layer) * hks + g;
      const size_t kv = unit * (size_t)srows * ds;
      rc = orc_small_head(ns, ds, in->s_scale, q, in->s_k + kv, in->s_v + kv,
                          out->logits + row * srows, &ms[j], &zs[j],
                          out->small_out + row * ds);
      if (rc != ORC_OK) break;
      out->row_max[row] = ms[j];
      out->row_sum[row] = zs[j];
      if (in->select == ORC_SELECT_GROUP) continue; /* selected per group below */
      if (in->select == ORC_SELECT_ACCUM) {
        /* H2O-style accumulated attention (the baseline the method builds on):
         * this step's probabilities are added to the head's running score,
         * which then ranks the tokens; the weights stay this step's p'. */
        if (in->s_held || !in->acc) {
          rc = ORC_EINVAL;
          break;
        }
        const float *lg = out->logits + row * srows;
        float *acc = in->acc + row * (size_t)ncap;
        const float zq = orc_zq(ns, lg, (float)ms[j]);
        for (int t = 0; t < ns; ++t) acc[t] = acc[t] + orc_exp(lg[t] - (float)ms[j]) / zq;
        rc = orc_partition(ns, in->k_crit[b], in->k_marg[b], in->k_recent ? in->k_recent[b] : 0,
                           acc, 0.0, 1.0, out->crit + row * in->kc_cap, in->kc_cap,
                           out->marg + row * in->km_cap, out->marg_prob + row * in->km_cap,
                           in->km_cap, out->mass + row * 2, &nc[j], &nm[j]);
        if (rc) break;
        double *mp = out->marg_prob + row * in->km_cap, *mass = out->mass + row * 2;
        const int32_t *crit = out->crit + row * in->kc_cap, *marg = out->marg + row * in->km_cap;
        mass[0] = mass[1] = 0.0;
        for (int i = 0; i < nc[j]; ++i) mass[0] += exp((double)lg[crit[i]] - ms[j]) / zs[j];
        for (int i = 0; i < in->km_cap; ++i) {
          mp[i] = i < nm[j] ? exp((double)lg[marg[i]] - ms[j]) / zs[j] : 0.0;
          mass[1] += mp[i];
        }
        continue;
      }
      rc = orc_partition(ns, in->k_crit[b], in->k_marg[b], in->k_recent ? in->k_recent[b] : 0,
                         out->logits + row * srows, ms[j], zs[j],
                         out->crit + row * in->kc_cap, in->kc_cap,
                         out->marg + row * in->km_cap,
                         out->marg_prob + row * in->km_cap, in->km_cap,
                         out->mass + row * 2, &nc[j], &nm[j]);
      if (rc != ORC_OK || !in->s_held) continue;
      const int32_t *pos = in->s_row_pos + unit * (size_t)srows;
      for (int r = 0; r < ns; ++r)
        if (pos[r] < 0 || pos[r] >= n || (r > 0 && pos[r] <= pos[r - 1])) rc = ORC_EINVAL;
      for (int i = 0; i < nc[j] && rc == ORC_OK; ++i)
        out->crit[row * in->kc_cap + i] = pos[out->crit[row * in->kc_cap + i]];
      for (int i = 0; i < nm[j] && rc == ORC_OK; ++i)
        out->marg[row * in->km_cap + i] = pos[out->marg[row * in->km_cap + i]];
    }
    if (rc == ORC_OK && in->select == ORC_SELECT_GROUP) {
      rc = group_step(in, out, b, n, ns, srows, ms, zs);
      continue;
    }
    /* stage 3 for every large head (layer, h) through j = f(layer, h) */
    for (int li = 0; li < L && rc == ORC_OK; ++li) {
      for (int h = 0; h < hq && rc == ORC_OK; ++h) {
        const int j = in->head_map[li * hq + h];
        if (j < 0 || j >= nsh) {
          rc = ORC_EINVAL;
          break;
        }
        const int g = h / gl;
        const size_t row = (size_t)b * nsh + j;
        const size_t unit = ((size_t)b * L + li) * hk + g;
        const size_t kv = unit * (size_t)in->l_rows * d;
        const int32_t *ks = in->k_slot ? in->k_slot + unit * ncap : NULL;
        const int32_t *vs = in->v_slot ? in->v_slot + unit * ncap : NULL;
        const size_t oi = (((size_t)b * L + li) * hq + h) * d;
        rc = orc_hybrid_head(d, in->l_scale, in->l_q + oi, in->l_k + kv,
                             in->l_v + kv, ks, vs, nc[j],
                             out->crit + row * in->kc_cap, nm[j],
                             out->marg + row * in->km_cap,
                             out->marg_prob + row * in->km_cap,
                             out->mass + row * 2, in->mode,
                             out->large_out + oi);
      }
    }
  }
  free(ms);
  free(zs);
  free(nc);
  free(nm);
  return rc;
}

/* ----------------------------------------------------- store maintenance -- */

/* Builds one kv head's store (see orc_store_update in the header). */
static void store_unit(const orc_store_in *in, size_t unit, int n, const uint8_t *inset,
                       const float *full, const float *old, const int32_t *old_slot,
                       float *dst, int32_t *slot, int32_t *count) {
  const int d = in->dim;
  int r = 0;
  for (int t = 0; t < n; ++t) {
    if (!inset[t]) {
      slot[t] = -1;
      continue;
    }
    if (r < in->rows) {
      const int os = old_slot ? old_slot[unit * in->n_cap + t] : -1;
      const float *src = (os >= 0 && os < in->rows)
                             ? old + (unit * (size_t)in->rows + (size_t)os) * d
                             : full + (unit * (size_t)in->n_cap + (size_t)t) * d;
      memcpy(dst + (unit * (size_t)in->rows + (size_t)r) * d, src, sizeof(float) * (size_t)d);
      slot[t] = r;
    } else {
      slot[t] = -1;
    }
    ++r;
  }
  *count = r;
}

int orc_store_update(const orc_store_in *in, float *new_k, float *new_v, int32_t *k_slot,
                     int32_t *v_slot, int32_t *counts) {
  const int B = in->batch, L = in->layers, hq = in->q_heads, hk = in->kv_heads;
  if (B < 1 || L < 1 || hk < 1 || hq % hk || in->n_cap < 1 || in->rows < 1) return ORC_EINVAL;
  const int g = hq / hk;
  uint8_t *inK = (uint8_t *)malloc((size_t)in->n_cap), *inV = (uint8_t *)malloc((size_t)in->n_cap);
  if (!inK || !inV) {
    free(inK);
    free(inV);
    return ORC_EINVAL;
  }
  int rc = ORC_OK;
  for (int b = 0; b < B && rc == ORC_OK; ++b) {
    const int n = in->seq_len[b];
    if (n < 1 || n > in->n_cap) {
      rc = ORC_EINVAL;
      break;
    }
    for (int li = 0; li < L; ++li)
      for (int kv = 0; kv < hk; ++kv) {
        memset(inK, 0, (size_t)n);
        memset(inV, 0, (size_t)n);
        for (int h = 0; h < g; ++h) {
          /* the lists this query head reads */
          size_t row;
          if (in->select == 1) {
            row = ((size_t)b * L + li) * hk + kv;
          } else {
            const int j = in->head_map[li * hq + kv * g + h];
            row = (size_t)b * in->n_small_heads + j;
          }
          const int32_t *c = in->crit + row * in->kc_cap, *m = in->marg + row * in->km_cap;
          for (int i = 0; i < in->kc_cap; ++i)
            if (c[i] >= 0 && c[i] < n) inK[c[i]] = inV[c[i]] = 1;
          for (int i = 0; i < in->km_cap; ++i)
            if (m[i] >= 0 && m[i] < n) inV[m[i]] = 1;
        }
        const size_t unit = ((size_t)b * L + li) * hk + kv;
        store_unit(in, unit, n, inK, in->full_k, in->old_k, in->old_k_slot, new_k,
                   k_slot + unit * in->n_cap, &counts[2 * unit]);
        store_unit(in, unit, n, inV, in->full_v, in->old_v, in->old_v_slot, new_v,
                   v_slot + unit * in->n_cap, &counts[2 * unit + 1]);
      }
  }
  free(inK);
  free(inV);
  return rc;
}
