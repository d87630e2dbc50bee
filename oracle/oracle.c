/*
 * oracle.c -- CPU oracle for PruneKV.  TEST INFRASTRUCTURE ONLY: loaded by the
 * tests, the smoke check and the benchmark's CPU-baseline leg, never by the
 * product path; shares no source with the GPU library.
 *
 * Plain loops, double precision, libm exp.  Each function names the passage of
 * the paper it follows; where the paper is silent the reading used is stated
 * next to the code (all readings are listed in the design notes).
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* bf16 bit pattern -> exact double. */
static double bf(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* fp32 -> bf16, round to nearest, ties to even (finite inputs). */
static uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t lsb = (u >> 16) & 1u;
  return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

/* bf16 bit pattern -> fp32 (exact). */
static float bf32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* ------------------------------------------------------------------------ */
/* Budgets: Eq. (parabolic), its normalisation, RR = p*q*(h/L)*m, Alg. 1.    */
/* ------------------------------------------------------------------------ */

typedef struct {
  double frac;
  int32_t layer;
} frac_t;

static int frac_cmp(const void *a, const void *b) {
  const frac_t *x = (const frac_t *)a, *y = (const frac_t *)b;
  if (x->frac > y->frac) return -1; /* larger remainder first */
  if (x->frac < y->frac) return 1;
  return x->layer < y->layer ? -1 : (x->layer > y->layer); /* tie: lower layer */
}

int orc_budget(int32_t L, int32_t n, double rr, int32_t h_param, double m, int32_t schedule, int32_t drop_all,
               int32_t *k, int32_t *n_surv, int32_t *h_out, double *b_out, double *q_out) {
  if (L < 2 || n < 0) return -1;
  if (!(rr > 0.0 && rr <= 1.0) || !(m > 0.0 && m <= 1.0)) return -1;
  /* Truncation layer: h in (1, L]; default three quarters of the depth. */
  int32_t h = h_param ? h_param : (int32_t)floor(0.75 * (double)L + 0.5);
  if (h < 2 || h > L) return -1;

  if (schedule < 0 || schedule > 3) return -1;
  /* Raw proportions, l = 1..h.
   *   0 parabola (Eq. parabolic): b_l = 1 - (l-1)^2 / (2 (h-1)^2), b_1 = 1, b_h = 1/2;
   *   1 fixed (budget ablation, "uniform budget per layer"): b_l = 1;
   *   2 arithmetic (ablation, linear progression; reading: the parabola's
   *     endpoints 1 and 1/2): b_l = 1 - (l-1) / (2 (h-1));
   *   3 geometric (ablation, progression over four layer blocks; reading:
   *     equal depth blocks, ratio 1/2): b_l = 2^-floor(4 (l-1) / h). */
  double *raw = (double *)malloc(sizeof(double) * (size_t)h);
  double *b = (double *)malloc(sizeof(double) * (size_t)h);
  for (int32_t l = 1; l <= h; ++l) {
    if (schedule == 0) {
      double num = (double)(l - 1) * (double)(l - 1);
      double den = 2.0 * (double)(h - 1) * (double)(h - 1);
      raw[l - 1] = 1.0 - num / den;
    } else if (schedule == 1) {
      raw[l - 1] = 1.0;
    } else if (schedule == 2) {
      raw[l - 1] = 1.0 - (double)(l - 1) / (2.0 * (double)(h - 1));
    } else {
      int32_t block = (4 * (l - 1)) / h;
      double v = 1.0;
      for (int32_t j = 0; j < block; ++j) v *= 0.5;
      raw[l - 1] = v;
    }
  }
  /* Normalise so that sum_l b_l = h*m.  Reading: a common scale factor, with
   * any proportion that would exceed 1 held at 1 and the remaining target
   * spread over the other layers by the same rule (water filling). */
  char *clip = (char *)calloc((size_t)h, 1);
  double s = 0.0;
  for (;;) {
    int32_t nclip = 0;
    double free_sum = 0.0;
    for (int32_t i = 0; i < h; ++i) {
      if (clip[i]) ++nclip;
      else free_sum += raw[i];
    }
    if (nclip == h) break;
    s = ((double)h * m - (double)nclip) / free_sum;
    int changed = 0;
    for (int32_t i = 0; i < h; ++i)
      if (!clip[i] && s * raw[i] > 1.0) { clip[i] = 1; changed = 1; }
    if (!changed) break;
  }
  for (int32_t i = 0; i < h; ++i) b[i] = clip[i] ? 1.0 : s * raw[i];

  /* Token-level ratio: RR = p*q*(h/L)*m with p = 1 (no frame filtering). */
  double q = rr / (((double)h / (double)L) * m);
  if (q > 1.0 + 1e-9) { free(raw); free(b); free(clip); return -1; }
  if (q > 1.0) q = 1.0;

  /* Integer budgets: T = round(RR*L*n) tokens in total, apportioned to layers
   * in proportion to b_l by largest remainder (ties to the lower layer). */
  double T = floor(rr * (double)L * (double)n + 0.5);
  double bsum = 0.0;
  for (int32_t i = 0; i < h; ++i) bsum += b[i];
  frac_t *fr = (frac_t *)malloc(sizeof(frac_t) * (size_t)h);
  double assigned = 0.0;
  for (int32_t i = 0; i < h; ++i) {
    double x = T * b[i] / bsum;
    double fl = floor(x);
    k[i] = (int32_t)fl;
    assigned += fl;
    fr[i].frac = x - fl;
    fr[i].layer = i;
  }
  int32_t rem = (int32_t)(T - assigned);
  int bad = rem < 0 || rem > h;
  if (!bad) {
    qsort(fr, (size_t)h, sizeof(frac_t), frac_cmp);
    for (int32_t j = 0; j < rem; ++j) k[fr[j].layer] += 1;
  }
  for (int32_t i = h; i < L; ++i) k[i] = 0; /* layers beyond h are evicted */
  for (int32_t i = 0; i < h; ++i) if (k[i] > n) bad = 1;

  /* Survivors of the top-q cut; never fewer than the largest layer budget.
   * With drop_all every token survives: the values of all non-kept tokens
   * are fused (Eq. (redistribution) read on its own). */
  int32_t ns = (int32_t)floor(q * (double)n + 0.5);
  for (int32_t i = 0; i < h; ++i) if (ns < k[i]) ns = k[i];
  if (ns > n) ns = n;
  if (drop_all) ns = n;
  *n_surv = ns;
  if (h_out) *h_out = h;
  if (q_out) *q_out = q;
  if (b_out) {
    for (int32_t i = 0; i < L; ++i) b_out[i] = i < h ? b[i] : 0.0;
  }
  free(raw); free(b); free(clip); free(fr);
  return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Scores: Eq. (token_score), with the window reading.                       */
/* ------------------------------------------------------------------------ */

void orc_scores_unit(int32_t n, int32_t d, int32_t rows, const uint16_t *K, const float *Q,
                     double *S) {
  double *qd = (double *)malloc(sizeof(double) * (size_t)d);
  double *z = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  for (int32_t v = 0; v < n; ++v) S[v] = 0.0;
  for (int32_t r = 0; r < rows; ++r) {
    /* The query enters the contraction in bf16, the cache's own type. */
    for (int32_t j = 0; j < d; ++j) qd[j] = bf(to_bf16(Q[(int64_t)r * d + j]));
    double zmax = -INFINITY;
    for (int32_t v = 0; v < n; ++v) {
      double acc = 0.0;
      const uint16_t *kv = K + (int64_t)v * d;
      for (int32_t j = 0; j < d; ++j) acc += qd[j] * bf(kv[j]);
      z[v] = acc * inv_sqrt_d; /* scaled dot-product attention logit */
      if (z[v] > zmax) zmax = z[v];
    }
    double sum = 0.0;
    for (int32_t v = 0; v < n; ++v) {
      z[v] = exp(z[v] - zmax);
      sum += z[v];
    }
    /* A_{r,v} = softmax over the visual keys; the score sums it over rows. */
    for (int32_t v = 0; v < n; ++v) S[v] += z[v] / sum;
  }
  free(qd);
  free(z);
}

/* ------------------------------------------------------------------------ */
/* Scores: Eq. (token_score) with every prefill token as a query.            */
/* ------------------------------------------------------------------------ */

void orc_scores_unit_prefill(int32_t n, int32_t T, int32_t d, int32_t G, const uint16_t *K,
                             const uint16_t *Kt, const float *Q, double *S, double *St) {
  const int32_t N = n + T;
  double *qd = (double *)malloc(sizeof(double) * (size_t)d);
  double *z = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
  double inv_sqrt_d = 1.0 / sqrt((double)d);
  for (int32_t v = 0; v < n; ++v) S[v] = 0.0;
  if (St)
    for (int32_t t = 0; t < T; ++t) St[t] = 0.0;
  for (int32_t hh = 0; hh < G; ++hh) {
    for (int32_t i = 0; i < N; ++i) {
      /* Token i of the sequence H = concat[H_v, H_q] (visual tokens first);
       * its query enters the contraction in bf16. */
      const float *qi = Q + ((int64_t)hh * N + i) * d;
      for (int32_t j = 0; j < d; ++j) qd[j] = bf(to_bf16(qi[j]));
      /* Causal self-attention: token i attends tokens 0..i. */
      double zmax = -INFINITY;
      for (int32_t j = 0; j <= i; ++j) {
        const uint16_t *kj = j < n ? K + (int64_t)j * d : Kt + (int64_t)(j - n) * d;
        double acc = 0.0;
        for (int32_t x = 0; x < d; ++x) acc += qd[x] * bf(kj[x]);
        z[j] = acc * inv_sqrt_d;
        if (z[j] > zmax) zmax = z[j];
      }
      double sum = 0.0;
      for (int32_t j = 0; j <= i; ++j) {
        z[j] = exp(z[j] - zmax);
        sum += z[j];
      }
      /* A^l_{i,j}; the visual columns accumulate into the score. */
      for (int32_t j = 0; j <= i; ++j) {
        if (j < n)
          S[j] += z[j] / sum;
        else if (St)
          St[j - n] += z[j] / sum;
      }
    }
  }
  free(qd);
  free(z);
}

/* ------------------------------------------------------------------------ */
/* Selection: top-q survivors and top-b_l keep set share one ranking.        */
/* ------------------------------------------------------------------------ */

typedef struct {
  float s;
  int32_t i;
} rank_t;

static int rank_cmp(const void *a, const void *b) {
  const rank_t *x = (const rank_t *)a, *y = (const rank_t *)b;
  if (x->s > y->s) return -1; /* higher score first */
  if (x->s < y->s) return 1;
  return x->i < y->i ? -1 : (x->i > y->i); /* equal scores: lower index first */
}

static int int_cmp(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return x < y ? -1 : (x > y);
}

void orc_select(int32_t n, const float *score, int32_t k, int32_t n_surv,
                int32_t *kept, int32_t *drop) {
  rank_t *r = (rank_t *)malloc(sizeof(rank_t) * (size_t)(n > 0 ? n : 1));
  for (int32_t v = 0; v < n; ++v) { r[v].s = score[v]; r[v].i = v; }
  qsort(r, (size_t)n, sizeof(rank_t), rank_cmp);
  for (int32_t j = 0; j < k; ++j) kept[j] = r[j].i;
  for (int32_t j = k; j < n_surv; ++j) drop[j - k] = r[j].i;
  qsort(kept, (size_t)k, sizeof(int32_t), int_cmp);
  qsort(drop, (size_t)(n_surv - k), sizeof(int32_t), int_cmp);
  free(r);
}

void orc_gather(int32_t d, int32_t k, const int32_t *kept, const uint16_t *K, uint16_t *K_out) {
  for (int32_t j = 0; j < k; ++j)
    memcpy(K_out + (int64_t)j * d, K + (int64_t)kept[j] * d, sizeof(uint16_t) * (size_t)d);
}

/* ------------------------------------------------------------------------ */
/* Value fusion: Eq. (redistribution), Eq. (weight_fusion).                  */
/* ------------------------------------------------------------------------ */

void orc_fuse(int32_t d, int32_t k, int32_t r, const uint16_t *V, const int32_t *kept,
              const int32_t *drop, double tau, double mu, double *out) {
  if (k <= 0) return;
  if (r <= 0) {
    /* Nothing was dropped: the kept values are returned unchanged. */
    for (int32_t i = 0; i < k; ++i)
      for (int32_t j = 0; j < d; ++j) out[(int64_t)i * d + j] = bf(V[(int64_t)kept[i] * d + j]);
    return;
  }
  double *a = (double *)malloc(sizeof(double) * (size_t)r);
  double *F = (double *)malloc(sizeof(double) * (size_t)d);
  for (int32_t i = 0; i < k; ++i) {
    const uint16_t *vk = V + (int64_t)kept[i] * d;
    /* Row i of Phi: softmax over the dropped tokens of (v_k,i . v_d,j) / tau. */
    double amax = -INFINITY;
    for (int32_t j = 0; j < r; ++j) {
      const uint16_t *vd = V + (int64_t)drop[j] * d;
      double acc = 0.0;
      for (int32_t x = 0; x < d; ++x) acc += bf(vk[x]) * bf(vd[x]);
      a[j] = acc / tau;
      if (a[j] > amax) amax = a[j];
    }
    double sum = 0.0;
    for (int32_t j = 0; j < r; ++j) {
      a[j] = exp(a[j] - amax);
      sum += a[j];
    }
    for (int32_t x = 0; x < d; ++x) F[x] = 0.0;
    for (int32_t j = 0; j < r; ++j) {
      const uint16_t *vd = V + (int64_t)drop[j] * d;
      double w = a[j] / sum;
      for (int32_t x = 0; x < d; ++x) F[x] += w * bf(vd[x]);
    }
    /* V_new = mu V_k + (1 - mu) Phi V_d. */
    for (int32_t x = 0; x < d; ++x) out[(int64_t)i * d + x] = mu * bf(vk[x]) + (1.0 - mu) * F[x];
  }
  free(a);
  free(F);
}

/* ------------------------------------------------------------------------ */
/* Decode attention (Sec. 2): softmax(scale q K^T) V.                         */
/* ------------------------------------------------------------------------ */

void orc_attend(int32_t d, int32_t rows, const uint16_t *q, const uint16_t *K, const uint16_t *V,
                double scale, double *out) {
  double *z = (double *)malloc(sizeof(double) * (size_t)(rows > 0 ? rows : 1));
  double zmax = -INFINITY;
  for (int32_t t = 0; t < rows; ++t) {
    double acc = 0.0;
    for (int32_t x = 0; x < d; ++x) acc += bf(q[x]) * bf(K[(int64_t)t * d + x]);
    z[t] = acc * scale;
    if (z[t] > zmax) zmax = z[t];
  }
  double sum = 0.0;
  for (int32_t t = 0; t < rows; ++t) {
    z[t] = exp(z[t] - zmax);
    sum += z[t];
  }
  for (int32_t x = 0; x < d; ++x) out[x] = 0.0;
  for (int32_t t = 0; t < rows; ++t) {
    double w = z[t] / sum;
    for (int32_t x = 0; x < d; ++x) out[x] += w * bf(V[(int64_t)t * d + x]);
  }
  free(z);
}

/* ------------------------------------------------------------------------ */
/* One unit end to end (layer- and head-specific ranking).                   */
/* ------------------------------------------------------------------------ */

void orc_prune_unit(int32_t n, int32_t d, int32_t rows, const uint16_t *K, const uint16_t *V,
                    const float *Q, int32_t k, int32_t n_surv, double tau, double mu,
                    int32_t *kept, int32_t *drop, uint16_t *K_out, double *V_out, float *S32) {
  double *S = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  float *s32 = (float *)malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  orc_scores_unit(n, d, rows, K, Q, S);
  for (int32_t v = 0; v < n; ++v) s32[v] = (float)S[v]; /* ranking in fp32 */
  orc_select(n, s32, k, n_surv, kept, drop);
  orc_gather(d, k, kept, K, K_out);
  orc_fuse(d, k, n_surv - k, V, kept, drop, tau, mu, V_out);
  if (S32) memcpy(S32, s32, sizeof(float) * (size_t)n);
  free(S);
  free(s32);
}

/* ------------------------------------------------------------------------ */
/* 4-bit cache rows (reading of the quantisation experiments; see header).    */
/* ------------------------------------------------------------------------ */

void orc_quant_rows(int32_t n, int32_t d, const uint16_t *x, uint8_t *codes, float *meta) {
  const int32_t groups = d / 32;
  for (int32_t r = 0; r < n; ++r) {
    memset(codes + (size_t)r * (d / 2), 0, (size_t)(d / 2));
    for (int32_t g = 0; g < groups; ++g) {
      const uint16_t *xg = x + (size_t)r * d + 32 * g;
      float lo = bf32(xg[0]), hi = lo;
      for (int c = 1; c < 32; ++c) {
        const float v = bf32(xg[c]);
        if (v < lo) lo = v;
        if (v > hi) hi = v;
      }
      lo = lo + 0.0f; /* -0 -> +0: the stored offset does not depend on which zero came first */
      const float range = hi - lo;
      const float scale = range / 15.0f;
      meta[((size_t)r * groups + g) * 2] = scale;
      meta[((size_t)r * groups + g) * 2 + 1] = lo;
      for (int c = 0; c < 32; ++c) {
        int code = 0;
        if (scale > 0.0f) {
          const float t = (bf32(xg[c]) - lo) / scale;
          code = (int)rintf(t);
          if (code < 0) code = 0;
          if (code > 15) code = 15;
        }
        const int ch = 32 * g + c;
        codes[(size_t)r * (d / 2) + ch / 2] |= (uint8_t)(code << (4 * (ch & 1)));
      }
    }
  }
}

void orc_dequant_rows(int32_t n, int32_t d, const uint8_t *codes, const float *meta, uint16_t *out) {
  const int32_t groups = d / 32;
  for (int32_t r = 0; r < n; ++r)
    for (int32_t ch = 0; ch < d; ++ch) {
      const int code = (codes[(size_t)r * (d / 2) + ch / 2] >> (4 * (ch & 1))) & 15;
      const float scale = meta[((size_t)r * groups + ch / 32) * 2];
      const float lo = meta[((size_t)r * groups + ch / 32) * 2 + 1];
      out[(size_t)r * d + ch] = to_bf16(fmaf((float)code, scale, lo));
    }
}
