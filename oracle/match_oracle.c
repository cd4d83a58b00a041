/*
 * match_oracle.c -- plain, slow, single-threaded CPU oracle of SmallKV's
 * prefill similarity matching (arXiv 2508.02751, Method section,
 * "Similarity Matching", Eqs. 1-3).
 *
 * TEST INFRASTRUCTURE ONLY (see smallkv_oracle.h): called by the test suite,
 * never by the product path; shares nothing with the HIP library.
 *
 * The matching turns fp32 sums into integer decisions (TopK sets, then an
 * argmax over Jaccard ratios).  For those decisions to be reproducible every
 * value that feeds them has one defined evaluation, stated where it is
 * computed: the logit of orc_logit, the exponential of orc_exp, and sums
 * taken one term at a time in ascending index order.  Each fp32 operation
 * is a correctly rounded IEEE-754 one (the file is built without fp
 * contraction or fast-math).
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include "smallkv_oracle.h"

/* ------------------------------------------------------------ exp -- */

/* exp(x) for x <= 0 in fp32, by Cody and Waite's argument reduction and a
 * degree-7 Taylor polynomial:
 *   k = round-to-nearest-even(x * fl(1/ln 2)),
 *   r = (x - k*LN2_HI) - k*LN2_LO         (two fused multiply-adds; LN2_HI
 *                                          has 16 significant bits, so
 *                                          k*LN2_HI is exact for |k| < 2^8),
 *   e^r = 1 + r + r^2/2! + ... + r^7/7!   (Horner's rule, fused multiply-adds,
 *                                          coefficients 1/n! rounded to fp32),
 *   exp(x) = e^r * 2^k                    (exact scaling).
 * Inputs below -80 (and NaN) give 0, which keeps every result a normal
 * number.  On [-80, 0] the result is within 1 ulp of exp(x). */
float orc_exp(float x) {
  if (!(x >= -80.0f)) return 0.0f;
  const float log2e = 0x1.715476p+0f;
  const float ln2_hi = 0x1.62e4p-1f;
  const float ln2_lo = 0x1.7f7d1cp-20f;
  const float k = rintf(x * log2e);
  float r = fmaf(-k, ln2_hi, x);
  r = fmaf(-k, ln2_lo, r);
  float p = 0x1.a01a02p-13f; /* 1/7! */
  p = fmaf(p, r, 0x1.6c16c2p-10f); /* 1/6! */
  p = fmaf(p, r, 0x1.111112p-7f);  /* 1/5! */
  p = fmaf(p, r, 0x1.555556p-5f);  /* 1/4! */
  p = fmaf(p, r, 0x1.555556p-3f);  /* 1/3! */
  p = fmaf(p, r, 0.5f);            /* 1/2! */
  p = fmaf(p, r, 1.0f);
  p = fmaf(p, r, 1.0f);
  return ldexpf(p, (int)k);
}

void orc_exp_n(int n, const float *x, float *y) {
  for (int i = 0; i < n; ++i) y[i] = orc_exp(x[i]);
}

/* ------------------------------------------------------ Eq. 1 scores -- */

/* Accumulative attention score of one head over a w-token prompt window.
 * The attention matrix is the prefill one, A = softmax(Q K^T / sqrt(d_h)),
 * with the causal mask every decoder applies in prefill: row u attends to
 * tokens v <= u.  Eq. 1: F_v = sum over rows u of A[u][v].
 *   s[u][v] = orc_logit(q_u, k_v)                    (v <= u)
 *   m_u     = max over v <= u of s[u][v]
 *   e[u][v] = orc_exp(s[u][v] - m_u)                 (fp32 subtraction)
 *   Z_u     = e[u][0] + e[u][1] + ... + e[u][u]      (fp32, left to right)
 *   F_v     = e[v][v]/Z_v + e[v+1][v]/Z_{v+1} + ... + e[w-1][v]/Z_{w-1}
 *                                                     (fp32 divisions, then
 *                                                      fp32 sums left to right)
 * Q, K: [w][d] fp32; F: [w]. */
int orc_match_scores(int w, int d, float scale, const float *Q, const float *K, float *F) {
  if (w < 1 || d < 1) return ORC_EINVAL;
  float *s = (float *)malloc(sizeof(float) * (size_t)w * (size_t)w);
  float *m = (float *)malloc(sizeof(float) * (size_t)w);
  float *Z = (float *)malloc(sizeof(float) * (size_t)w);
  if (!s || !m || !Z) {
    free(s);
    free(m);
    free(Z);
    return ORC_EINVAL;
  }
  int rc = ORC_OK;
  for (int u = 0; u < w && rc == ORC_OK; ++u)
    for (int v = 0; v <= u; ++v) {
      const float x = orc_logit(d, scale, Q + (size_t)u * d, K + (size_t)v * d);
      if (!isfinite(x)) {
        rc = ORC_ENONFINITE;
        break;
      }
      s[(size_t)u * w + v] = x;
    }
  if (rc == ORC_OK) {
    for (int u = 0; u < w; ++u) {
      float mu = s[(size_t)u * w];
      for (int v = 1; v <= u; ++v)
        if (s[(size_t)u * w + v] > mu) mu = s[(size_t)u * w + v];
      float z = 0.0f;
      for (int v = 0; v <= u; ++v) z = z + orc_exp(s[(size_t)u * w + v] - mu);
      m[u] = mu;
      Z[u] = z;
    }
    for (int v = 0; v < w; ++v) {
      float f = 0.0f;
      for (int u = v; u < w; ++u) f = f + orc_exp(s[(size_t)u * w + v] - m[u]) / Z[u];
      F[v] = f;
    }
  }
  free(s);
  free(m);
  free(Z);
  return rc;
}

/* ------------------------------------------------------- Eq. 2 TopK -- */

typedef struct {
  float f;
  int idx;
} orc_scored;

/* Larger score first; equal scores by lower token index first. */
static int scored_cmp(const void *a, const void *b) {
  const orc_scored *x = (const orc_scored *)a, *y = (const orc_scored *)b;
  if (x->f != y->f) return x->f > y->f ? -1 : 1;
  return (x->idx > y->idx) - (x->idx < y->idx);
}

/* TopK(F): in_top[v] = 1 for the k first tokens of the order above. */
int orc_topk(int w, int k, const float *F, uint8_t *in_top) {
  if (w < 1 || k < 1 || k > w) return ORC_EINVAL;
  orc_scored *it = (orc_scored *)malloc(sizeof(orc_scored) * (size_t)w);
  if (!it) return ORC_EINVAL;
  for (int v = 0; v < w; ++v) {
    it[v].f = F[v];
    it[v].idx = v;
  }
  qsort(it, (size_t)w, sizeof(orc_scored), scored_cmp);
  memset(in_top, 0, (size_t)w);
  for (int r = 0; r < k; ++r) in_top[it[r].idx] = 1;
  free(it);
  return ORC_OK;
}

/* Eq. 2 as a fraction: |A n B| / |A u B| of two token sets over w tokens. */
void orc_jaccard(int w, const uint8_t *a, const uint8_t *b, int *num, int *den) {
  int in = 0, un = 0;
  for (int v = 0; v < w; ++v) {
    in += a[v] && b[v];
    un += a[v] || b[v];
  }
  *num = in;
  *den = un;
}

/* ------------------------------------------------------ Eq. 3 map -- */

static int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

/* One model's window operands, layouts as in the header. */
static int window_scores(const orc_window *m, int b, int w_cap, int w, float *F_out,
                         uint8_t *top, int k, int head0, int n_heads_total, float *scores,
                         uint8_t *top_out) {
  const int g = m->q_heads / m->kv_heads;
  for (int layer = 0; layer < m->layers; ++layer)
    for (int h = 0; h < m->q_heads; ++h) {
      const int j = layer * m->q_heads + h;
      const float *Q =
          m->q + ((((size_t)b * m->layers + layer) * m->q_heads + h) * w_cap) * m->dim;
      const float *K =
          m->k + ((((size_t)b * m->layers + layer) * m->kv_heads + h / g) * w_cap) * m->dim;
      float *F = F_out + (size_t)j * w;
      int rc = orc_match_scores(w, m->dim, m->scale, Q, K, F);
      if (rc) return rc;
      rc = orc_topk(w, k, F, top + (size_t)j * w);
      if (rc) return rc;
      const size_t row = (size_t)b * n_heads_total + head0 + j;
      if (scores) memcpy(scores + row * w_cap, F, sizeof(float) * (size_t)w);
      if (top_out) memcpy(top_out + row * w_cap, top + (size_t)j * w, (size_t)w);
    }
  return ORC_OK;
}

/* f(i) = argmax_j S(A_i, A'_j) over every small head j of every small layer
 * (Eq. 3); a tie goes to the lowest j.  Ratios are compared exactly as
 * fractions of integers. */
int orc_match(const orc_match_in *in, int32_t *head_map, float *scores, uint8_t *top_out) {
  if (!in || in->batch < 1 || in->w_cap < 1 || !in->win_len || !in->top_k) return ORC_EINVAL;
  const orc_window *L = &in->large, *S = &in->small;
  if (L->layers < 1 || L->q_heads < 1 || L->kv_heads < 1 || L->q_heads % L->kv_heads ||
      S->layers < 1 || S->q_heads < 1 || S->kv_heads < 1 || S->q_heads % S->kv_heads)
    return ORC_EINVAL;
  const int nl = L->layers * L->q_heads, ns = S->layers * S->q_heads;
  const int w_cap = in->w_cap;
  float *Fl = (float *)malloc(sizeof(float) * (size_t)nl * w_cap);
  float *Fs = (float *)malloc(sizeof(float) * (size_t)ns * w_cap);
  uint8_t *Tl = (uint8_t *)malloc((size_t)nl * w_cap);
  uint8_t *Ts = (uint8_t *)malloc((size_t)ns * w_cap);
  int rc = (Fl && Fs && Tl && Ts) ? ORC_OK : ORC_EINVAL;
  for (int b = 0; b < in->batch && rc == ORC_OK; ++b) {
    const int w = clampi(in->win_len[b], 1, w_cap);
    const int k = clampi(in->top_k[b], 1, w);
    rc = window_scores(L, b, w_cap, w, Fl, Tl, k, 0, nl + ns, scores, top_out);
    if (rc) break;
    rc = window_scores(S, b, w_cap, w, Fs, Ts, k, nl, nl + ns, scores, top_out);
    if (rc) break;
    for (int i = 0; i < nl; ++i) {
      int best = 0, bn = -1, bd = 1;
      for (int j = 0; j < ns; ++j) {
        int n, d;
        orc_jaccard(w, Tl + (size_t)i * w, Ts + (size_t)j * w, &n, &d);
        if ((long long)n * bd > (long long)bn * d) {
          best = j;
          bn = n;
          bd = d;
        }
      }
      head_map[(size_t)b * nl + i] = best;
    }
  }
  free(Fl);
  free(Fs);
  free(Tl);
  free(Ts);
  return rc;
}
