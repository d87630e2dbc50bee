/*
 * synthgen.c -- seeded synthetic inputs for PruneKV (visual KV cache, window
 * queries, decode rows).  This module holds only random-number generation and
 * the data model of the workloads; none of the compression method's arithmetic
 * lives here.  Both the CPU oracle and the GPU path read the buffers it fills.
 *
 * Random numbers: counter-based.  Every value is a pure function of
 * (seed, tensor id, element index), so any subset can be regenerated in any
 * order and on any number of threads.
 *   mix(x)      = the SplitMix64 output function (Steele, Lea, Flood 2014):
 *                 z = x + 0x9E3779B97F4A7C15;
 *                 z = (z ^ z>>30) * 0xBF58476D1CE4E5B9;
 *                 z = (z ^ z>>27) * 0x94D049BB133111EB;  return z ^ z>>31.
 *   key(s, t)   = mix(s ^ mix(t))
 *   U(s, t, i)  = (mix(key(s,t) + i) >> 11) * 2^-53            in [0, 1)
 *   N(s, t, i)  = sqrt(-2 ln(1 - U(s,t,2i))) * cos(2 pi U(s,t,2i+1))
 *                 (Box-Muller, cosine branch only)
 *
 * Data model (one visual token = one row of d values):
 *   token v of sequence b lies in frame f(v) = v / tokens_per_frame;
 *   per (b, layer, kv head) and per role K/V there is one centroid per frame,
 *   c_f ~ N(0, I_d); token x_v = 0.8 c_f(v) + 0.6 eps_v, eps ~ N(0, I_d);
 *   outlier tokens (a per-sequence set shared by all layers, heads, K and V)
 *   are scaled by 8; the result is rounded to bfloat16 (round to nearest even).
 *   Window query (b, layer, q head h, row i) = xi + c^K_{b,l,h/G, rel[i mod R]}
 *   with xi ~ N(0, I_d) and rel[] R distinct "relevant" frames per sequence;
 *   stored as fp32 values that are exactly representable in bfloat16.
 * Prefill scoring (every token of the prefill is a query):
 *   the query of visual token v = xi + c^K_{b,l,h/G, f(v)} (aligned with its
 *   own frame); the queries of the W text tokens are the window queries;
 *   text keys (b, layer, kv head g, token t) ~ N(0, I_d), rounded to bf16.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  uint64_t seed;
  int32_t B, L, Hq, Hkv, d, W;
  int32_t tokens_per_frame; /* N_V */
  int32_t frames;           /* nominal frames per sequence */
  int32_t frame_jitter;     /* frames_b = frames + U{-J..J}; 0 = no jitter */
  int32_t n_relevant;       /* R */
  double outlier_frac;      /* rho */
} sg_config;

enum {
  ROLE_CENT_K = 1, ROLE_CENT_V = 2, ROLE_NOISE_K = 3, ROLE_NOISE_V = 4,
  ROLE_Q = 5, ROLE_OUTLIER = 6, ROLE_RELEVANT = 7, ROLE_JITTER = 8,
  ROLE_NORMAL = 9, ROLE_QVIS = 10, ROLE_KTEXT = 11
};

static inline uint64_t mix(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline uint64_t tensor_id(uint64_t role, uint64_t b, uint64_t l, uint64_t g) {
  return (role << 48) ^ (b << 32) ^ (l << 16) ^ g;
}

static inline uint64_t stream_key(uint64_t seed, uint64_t tid) { return mix(seed ^ mix(tid)); }

static inline double unif(uint64_t key, uint64_t i) {
  return (double)(mix(key + i) >> 11) * 0x1.0p-53;
}

static inline double normal(uint64_t key, uint64_t i) {
  double u1 = unif(key, 2 * i), u2 = unif(key, 2 * i + 1);
  return sqrt(-2.0 * log(1.0 - u1)) * cos(6.283185307179586476925 * u2);
}

static inline uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline float bf16_round_f32(float f) {
  uint32_t u = (uint32_t)bf16_rne(f) << 16;
  float r;
  memcpy(&r, &u, 4);
  return r;
}

/* ---- per-sequence metadata ---------------------------------------------- */

int32_t sg_frames_of(const sg_config *c, int32_t b) {
  if (c->frame_jitter <= 0) return c->frames;
  uint64_t key = stream_key(c->seed, tensor_id(ROLE_JITTER, (uint64_t)b, 0, 0));
  int32_t span = 2 * c->frame_jitter + 1;
  int32_t off = (int32_t)floor(unif(key, 0) * span) - c->frame_jitter;
  int32_t f = c->frames + off;
  return f < 1 ? 1 : f;
}

void sg_n_vis(const sg_config *c, int32_t *n) {
  for (int32_t b = 0; b < c->B; ++b) n[b] = sg_frames_of(c, b) * c->tokens_per_frame;
}

/* Partial Fisher-Yates: the first `cnt` entries of a permutation of [0, total). */
static void pick_distinct(uint64_t key, int32_t total, int32_t cnt, int32_t *out) {
  int32_t *perm = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total > 0 ? total : 1));
  for (int32_t i = 0; i < total; ++i) perm[i] = i;
  for (int32_t i = 0; i < cnt; ++i) {
    int32_t j = i + (int32_t)floor(unif(key, (uint64_t)i) * (double)(total - i));
    if (j >= total) j = total - 1;
    int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
    out[i] = perm[i];
  }
  free(perm);
}

int32_t sg_outlier_count(const sg_config *c, int32_t n_b) {
  return (int32_t)floor(c->outlier_frac * (double)n_b + 0.5);
}

/* flag[v] = 1 for the outlier tokens of sequence b (n_b tokens). */
void sg_outlier_flags(const sg_config *c, int32_t b, int32_t n_b, uint8_t *flag) {
  int32_t cnt = sg_outlier_count(c, n_b);
  memset(flag, 0, (size_t)n_b);
  if (cnt <= 0) return;
  int32_t *pick = (int32_t *)malloc(sizeof(int32_t) * (size_t)cnt);
  pick_distinct(stream_key(c->seed, tensor_id(ROLE_OUTLIER, (uint64_t)b, 0, 0)), n_b, cnt, pick);
  for (int32_t i = 0; i < cnt; ++i) flag[pick[i]] = 1;
  free(pick);
}

void sg_relevant_frames(const sg_config *c, int32_t b, int32_t *rel) {
  int32_t F = sg_frames_of(c, b);
  int32_t R = c->n_relevant < F ? c->n_relevant : F;
  pick_distinct(stream_key(c->seed, tensor_id(ROLE_RELEVANT, (uint64_t)b, 0, 0)), F, R, rel);
}

/* ---- threaded fill helpers ---------------------------------------------- */

typedef struct {
  const sg_config *c;
  int role; /* 0 = K, 1 = V */
  int32_t layer;
  uint16_t *out;
  const int64_t *row_base; /* per (b) packed row offset of sequence b, times Hkv */
  const int32_t *n;
  uint8_t **outl;
  float **cent; /* per (b*Hkv+g): [F_b][d] */
  int64_t rows_total;
  int nthreads, tid;
} kv_job;

static void *kv_worker(void *p) {
  kv_job *j = (kv_job *)p;
  const sg_config *c = j->c;
  const int32_t d = c->d;
  int64_t lo = j->rows_total * j->tid / j->nthreads;
  int64_t hi = j->rows_total * (j->tid + 1) / j->nthreads;
  /* locate (b, g, v) of row lo by walking sequences */
  for (int32_t b = 0; b < c->B; ++b) {
    int64_t base = j->row_base[b];
    int64_t cnt = (int64_t)c->Hkv * j->n[b];
    int64_t a = lo > base ? lo : base, e = hi < base + cnt ? hi : base + cnt;
    for (int64_t r = a; r < e; ++r) {
      int64_t local = r - base;
      int32_t g = (int32_t)(local / j->n[b]);
      int32_t v = (int32_t)(local % j->n[b]);
      int32_t f = v / c->tokens_per_frame;
      uint64_t nkey = stream_key(c->seed, tensor_id(j->role ? ROLE_NOISE_V : ROLE_NOISE_K,
                                                    (uint64_t)b, (uint64_t)j->layer, (uint64_t)g));
      const float *cf = j->cent[(int64_t)b * c->Hkv + g] + (int64_t)f * d;
      double scale = j->outl[b][v] ? 8.0 : 1.0;
      uint16_t *dst = j->out + r * d;
      for (int32_t x = 0; x < d; ++x) {
        double val = 0.8 * (double)cf[x] + 0.6 * normal(nkey, (uint64_t)v * d + x);
        dst[x] = bf16_rne((float)(val * scale));
      }
    }
  }
  return NULL;
}

static float *make_centroids(const sg_config *c, int role, int32_t b, int32_t l, int32_t g, int32_t F) {
  float *cent = (float *)malloc(sizeof(float) * (size_t)F * c->d);
  uint64_t key = stream_key(c->seed, tensor_id(role ? ROLE_CENT_V : ROLE_CENT_K,
                                               (uint64_t)b, (uint64_t)l, (uint64_t)g));
  for (int64_t i = 0; i < (int64_t)F * c->d; ++i) cent[i] = (float)normal(key, (uint64_t)i);
  return cent;
}

/* Fill one layer of K (role 0) or V (role 1) for all sequences:
 * bf16 packed [sum_b Hkv*n_b][d], row (b, g, v) at off_b*Hkv + g*n_b + v. */
int sg_kv_layer(const sg_config *c, int role, int32_t layer, uint16_t *out, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  int32_t *n = (int32_t *)malloc(sizeof(int32_t) * c->B);
  int64_t *row_base = (int64_t *)malloc(sizeof(int64_t) * c->B);
  uint8_t **outl = (uint8_t **)malloc(sizeof(uint8_t *) * c->B);
  float **cent = (float **)malloc(sizeof(float *) * (size_t)c->B * c->Hkv);
  sg_n_vis(c, n);
  int64_t rows = 0;
  for (int32_t b = 0; b < c->B; ++b) {
    row_base[b] = rows;
    rows += (int64_t)c->Hkv * n[b];
    outl[b] = (uint8_t *)malloc((size_t)(n[b] > 0 ? n[b] : 1));
    sg_outlier_flags(c, b, n[b], outl[b]);
    int32_t F = sg_frames_of(c, b);
    for (int32_t g = 0; g < c->Hkv; ++g) cent[(int64_t)b * c->Hkv + g] = make_centroids(c, role, b, layer, g, F);
  }
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * nthreads);
  kv_job *jobs = (kv_job *)malloc(sizeof(kv_job) * nthreads);
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = (kv_job){c, role, layer, out, row_base, n, outl, cent, rows, nthreads, t};
    pthread_create(&th[t], NULL, kv_worker, &jobs[t]);
  }
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  for (int32_t b = 0; b < c->B; ++b) {
    free(outl[b]);
    for (int32_t g = 0; g < c->Hkv; ++g) free(cent[(int64_t)b * c->Hkv + g]);
  }
  free(th); free(jobs); free(n); free(row_base); free(outl); free(cent);
  return 0;
}

/* Window queries of one layer: fp32 [B][Hq][W][d], bf16-representable. */
int sg_q_layer(const sg_config *c, int32_t layer, float *out) {
  const int32_t d = c->d, G = c->Hq / c->Hkv;
  for (int32_t b = 0; b < c->B; ++b) {
    int32_t F = sg_frames_of(c, b);
    int32_t R = c->n_relevant < F ? c->n_relevant : F;
    int32_t rel[64];
    if (R > 64) R = 64;
    sg_relevant_frames(c, b, rel);
    for (int32_t h = 0; h < c->Hq; ++h) {
      int32_t g = h / G;
      float *cent = make_centroids(c, 0, b, layer, g, F);
      uint64_t key = stream_key(c->seed, tensor_id(ROLE_Q, (uint64_t)b, (uint64_t)layer, (uint64_t)h));
      for (int32_t i = 0; i < c->W; ++i) {
        const float *cf = R > 0 ? cent + (int64_t)rel[i % R] * d : NULL;
        float *dst = out + (((int64_t)b * c->Hq + h) * c->W + i) * d;
        for (int32_t x = 0; x < d; ++x) {
          double val = normal(key, (uint64_t)i * d + x) + (cf ? (double)cf[x] : 0.0);
          dst[x] = bf16_round_f32((float)val);
        }
      }
      free(cent);
    }
  }
  return 0;
}

/* Queries of every prefill token, fp32 (bf16-representable), packed over
 * sequences: row (b, h, i) at qoff_b*Hq + h*(n_b + W) + i, with
 * qoff_b = sum_{b' < b} (n_b' + W); i < n_b are the visual tokens, then the
 * W text tokens (the window queries of sg_q_layer). */
int sg_qall_layer(const sg_config *c, int32_t layer, float *out) {
  const int32_t d = c->d, G = c->Hq / c->Hkv;
  int32_t *n = (int32_t *)malloc(sizeof(int32_t) * c->B);
  sg_n_vis(c, n);
  float *win = (float *)malloc(sizeof(float) * (size_t)c->B * c->Hq * c->W * d);
  sg_q_layer(c, layer, win);
  int64_t row = 0;
  for (int32_t b = 0; b < c->B; ++b) {
    const int32_t F = sg_frames_of(c, b);
    const int32_t N = n[b] + c->W;
    for (int32_t h = 0; h < c->Hq; ++h) {
      float *cent = make_centroids(c, 0, b, layer, h / G, F);
      uint64_t key = stream_key(c->seed, tensor_id(ROLE_QVIS, (uint64_t)b, (uint64_t)layer, (uint64_t)h));
      for (int32_t i = 0; i < N; ++i) {
        float *dst = out + (row + (int64_t)h * N + i) * d;
        if (i < n[b]) {
          const float *cf = cent + (int64_t)(i / c->tokens_per_frame) * d;
          for (int32_t x = 0; x < d; ++x) dst[x] = bf16_round_f32((float)(normal(key, (uint64_t)i * d + x) + (double)cf[x]));
        } else {
          memcpy(dst, win + (((int64_t)b * c->Hq + h) * c->W + (i - n[b])) * d, sizeof(float) * (size_t)d);
        }
      }
      free(cent);
    }
    row += (int64_t)c->Hq * N;
  }
  free(win);
  free(n);
  return 0;
}

/* Keys of the W text tokens, bf16 [B][Hkv][W][d]. */
int sg_ktext_layer(const sg_config *c, int32_t layer, uint16_t *out) {
  const int32_t d = c->d;
  for (int32_t b = 0; b < c->B; ++b)
    for (int32_t g = 0; g < c->Hkv; ++g) {
      uint64_t key = stream_key(c->seed, tensor_id(ROLE_KTEXT, (uint64_t)b, (uint64_t)layer, (uint64_t)g));
      uint16_t *dst = out + (((int64_t)b * c->Hkv + g) * c->W) * d;
      for (int64_t i = 0; i < (int64_t)c->W * d; ++i) dst[i] = bf16_rne((float)normal(key, (uint64_t)i));
    }
  return 0;
}

/* Generic N(0,1) bf16 fill for decode rows and decode queries. */
void sg_normal_bf16(uint64_t seed, uint64_t stream, int64_t count, uint16_t *out) {
  uint64_t key = stream_key(seed, tensor_id(ROLE_NORMAL, 0, 0, 0) ^ mix(stream));
  for (int64_t i = 0; i < count; ++i) out[i] = bf16_rne((float)normal(key, (uint64_t)i));
}

/* Uniform doubles, exposed so tests can check the generator's distribution. */
void sg_uniform(uint64_t seed, uint64_t stream, int64_t count, double *out) {
  uint64_t key = stream_key(seed, tensor_id(ROLE_NORMAL, 0, 0, 0) ^ mix(stream));
  for (int64_t i = 0; i < count; ++i) out[i] = unif(key, (uint64_t)i);
}
