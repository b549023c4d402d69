/*
 * synth.c - seeded synthetic multi-vector corpora.  See synth.h for the recipe.
 * Input generation only: nothing in this file scores, probes, quantises or
 * selects.
 */
#include "synth.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GOLDEN_GAMMA 0x9E3779B97F4A7C15ULL

enum {
  STREAM_CENT = 1,
  STREAM_LEN = 2,
  STREAM_TOKCLUSTER = 3,
  STREAM_TOKNOISE = 4,
  STREAM_PERM = 5,
  STREAM_QSRC = 6,
  STREAM_QNOISE = 7,
  STREAM_QSEED = 8
};

struct synth_ctx {
  synth_cfg cfg;
  int16_t *cent;  /* [ncent][dim] */
  double *zipf_cdf; /* [ncent], cumulative unnormalised weights (zipf only) */
  int32_t *perm;  /* [ncent] rank -> centroid id (zipf only) */
  int32_t *zipf_guide; /* [ZIPF_GUIDE + 1]: entry j is the first rank whose
                          cdf exceeds (j / ZIPF_GUIDE) of the total (zipf only) */
};

#define ZIPF_GUIDE 65536
#define SYNTH_MAX_DIM 1024

/* SplitMix64 output function. */
static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* n-th output (0-based) of a SplitMix64 generator whose state starts at s. */
uint64_t synth_splitmix64_at(uint64_t s, uint64_t n) { return sm_mix(s + (n + 1) * GOLDEN_GAMMA); }

/* Stream key for (seed, stream, index): two chained SplitMix64 draws. */
static inline uint64_t stream_key(uint64_t seed, uint64_t stream, uint64_t index) {
  return synth_splitmix64_at(synth_splitmix64_at(seed, stream), index);
}

/* Uniform double in the open interval (0, 1). */
static inline double u01(uint64_t key, uint64_t ctr) {
  uint64_t x = synth_splitmix64_at(key, ctr);
  return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

/* Box-Muller: the two normals of pair p from counters 2p and 2p+1. */
static inline void normal_pair(uint64_t key, uint64_t pair, double *z0, double *z1) {
  double a = u01(key, 2 * pair), b = u01(key, 2 * pair + 1);
  double r = sqrt(-2.0 * log(a));
  double t = 6.283185307179586476925286766559 * b;
  *z0 = r * cos(t);
  *z1 = r * sin(t);
}

/* The Box-Muller normals of pairs base .. base + np - 1 into z[2 np]
 * (vectorised transform in synth_bm.c).  w is scratch of 4 np doubles
 * following z: uniforms a, b, then the transform's r and t. */
void synth_box_muller(const double *restrict a, const double *restrict b, double *restrict r,
                      double *restrict t, double *restrict z, int n);
static void normals(uint64_t key, uint64_t base, int np, double *z, double *w) {
  double *a = w, *b = w + np;
  for (int p = 0; p < np; ++p) {
    a[p] = u01(key, 2 * (base + (uint64_t)p));
    b[p] = u01(key, 2 * (base + (uint64_t)p) + 1);
  }
  synth_box_muller(a, b, w + 2 * np, w + 3 * np, z, np);
}

double synth_to_grid(double x) {
  double a = fabs(x);
  /* below 2^-4 the grid spacing is 2^-11: adding and removing 1.5 * 2^41
   * (whose ulp is 2^-11) rounds to it, ties to even, in the default rounding
   * mode (this file is built without value-changing optimisations) */
  if (a < 0.0625) return (x + 3298534883328.0) - 3298534883328.0;
  /* bf16 spacing: keep 8 significant bits of the normal double x, rounding
   * the 45 dropped significand bits to nearest, ties to even (a carry out of
   * the significand correctly bumps the exponent) */
  uint64_t b;
  memcpy(&b, &x, sizeof b);
  b += ((uint64_t)1 << 44) - 1 + ((b >> 45) & 1);
  b &= ~(((uint64_t)1 << 45) - 1);
  memcpy(&x, &b, sizeof x);
  return x;
}

/* Unit-normalise v[dim] and write its grid integers to out. */
static void normalise_to_grid(const double *v, int dim, int16_t *out) {
  double ss = 0.0;
  for (int i = 0; i < dim; ++i) ss += v[i] * v[i];
  double inv = ss > 0.0 ? 1.0 / sqrt(ss) : 0.0;
  for (int i = 0; i < dim; ++i) {
    double g = synth_to_grid(v[i] * inv);
    out[i] = (int16_t)(g * 2048.0); /* exact: g is a multiple of 2^-11 */
  }
}

synth_ctx *synth_create(const synth_cfg *cfg) {
  if (!cfg || cfg->ncent <= 0 || cfg->dim <= 0 || (cfg->dim & 1) || cfg->dim > SYNTH_MAX_DIM || cfg->ndocs < 0)
    return NULL;
  if (cfg->len_lo < 1 || cfg->len_hi < cfg->len_lo) return NULL;
  synth_ctx *ctx = (synth_ctx *)calloc(1, sizeof(synth_ctx));
  if (!ctx) return NULL;
  ctx->cfg = *cfg;
  int n = cfg->ncent, dim = cfg->dim;
  ctx->cent = (int16_t *)malloc((size_t)n * dim * sizeof(int16_t));
  if (!ctx->cent) { synth_free(ctx); return NULL; }
#pragma omp parallel
  {
    double *v = (double *)malloc((size_t)4 * dim * sizeof(double));
#pragma omp for schedule(static)
    for (int c = 0; c < n; ++c) {
      uint64_t key = stream_key(cfg->seed, STREAM_CENT, (uint64_t)c);
      normals(key, 0, dim / 2, v, v + dim);
      normalise_to_grid(v, dim, ctx->cent + (size_t)c * dim);
    }
    free(v);
  }
  if (cfg->pop_kind == SYNTH_POP_ZIPF) {
    ctx->zipf_cdf = (double *)malloc((size_t)n * sizeof(double));
    ctx->perm = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    ctx->zipf_guide = (int32_t *)malloc((size_t)(ZIPF_GUIDE + 1) * sizeof(int32_t));
    if (!ctx->zipf_cdf || !ctx->perm || !ctx->zipf_guide) { synth_free(ctx); return NULL; }
    double acc = 0.0;
    for (int r = 0; r < n; ++r) {
      acc += pow((double)(r + 1), -cfg->zipf_s);
      ctx->zipf_cdf[r] = acc;
    }
    for (int j = 0, r = 0; j <= ZIPF_GUIDE; ++j) {
      const double x = ((double)j / (double)ZIPF_GUIDE) * acc;
      while (r < n - 1 && !(ctx->zipf_cdf[r] > x)) ++r;
      ctx->zipf_guide[j] = r;
    }
    for (int i = 0; i < n; ++i) ctx->perm[i] = i;
    uint64_t key = stream_key(cfg->seed, STREAM_PERM, 0);
    for (int i = n - 1; i > 0; --i) { /* Fisher-Yates */
      int j = (int)(u01(key, (uint64_t)i) * (double)(i + 1));
      if (j > i) j = i;
      int32_t t = ctx->perm[i];
      ctx->perm[i] = ctx->perm[j];
      ctx->perm[j] = t;
    }
  }
  return ctx;
}

void synth_free(synth_ctx *ctx) {
  if (!ctx) return;
  free(ctx->cent);
  free(ctx->zipf_cdf);
  free(ctx->perm);
  free(ctx->zipf_guide);
  free(ctx);
}

const int16_t *synth_centroids(const synth_ctx *ctx) { return ctx->cent; }

static int32_t doc_length(const synth_ctx *ctx, int64_t d) {
  const synth_cfg *c = &ctx->cfg;
  uint64_t key = stream_key(c->seed, STREAM_LEN, (uint64_t)d);
  if (c->len_kind == SYNTH_LEN_FIXED) return c->len_lo;
  if (c->len_kind == SYNTH_LEN_UNIFORM) {
    int64_t span = (int64_t)c->len_hi - c->len_lo + 1;
    int64_t off = (int64_t)(u01(key, 0) * (double)span);
    if (off >= span) off = span - 1;
    return (int32_t)(c->len_lo + off);
  }
  double z0, z1;
  normal_pair(key, 0, &z0, &z1);
  double mu = log(c->len_mean) - 0.5 * c->len_sigma * c->len_sigma;
  double L = nearbyint(exp(mu + c->len_sigma * z0));
  if (L < c->len_lo) L = c->len_lo;
  if (L > c->len_hi) L = c->len_hi;
  return (int32_t)L;
}

void synth_doc_lengths(const synth_ctx *ctx, int64_t d0, int64_t d1, int32_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t d = d0; d < d1; ++d) out[d - d0] = doc_length(ctx, d);
}

/* First rank r with zipf_cdf[r] > x (the last rank if there is none),
 * searched between lo and hi, which must bracket that rank. */
static int zipf_search(const synth_ctx *ctx, double x, int lo, int hi) {
  while (lo < hi) {
    int mid = lo + (hi - lo) / 2;
    if (ctx->zipf_cdf[mid] > x) hi = mid; else lo = mid + 1;
  }
  return lo;
}

static int32_t cluster_of(const synth_ctx *ctx, uint64_t key, int64_t t) {
  const synth_cfg *c = &ctx->cfg;
  double u = u01(key, (uint64_t)t);
  if (c->pop_kind == SYNTH_POP_ZIPF) {
    double x = u * ctx->zipf_cdf[c->ncent - 1];
    /* u in [j/G, (j+1)/G) and rounding is monotone, so x lies between the
     * guide's thresholds j and j+1 and the rank between their entries */
    int j = (int)(u * (double)ZIPF_GUIDE);
    if (j >= ZIPF_GUIDE) j = ZIPF_GUIDE - 1;
    return ctx->perm[zipf_search(ctx, x, ctx->zipf_guide[j], ctx->zipf_guide[j + 1])];
  }
  int32_t k = (int32_t)(u * (double)c->ncent);
  return k >= c->ncent ? c->ncent - 1 : k;
}

/* Per-thread scratch of a block of up to GEN_BLOCK tokens. */
#define GEN_BLOCK 8
typedef struct {
  double a[GEN_BLOCK * SYNTH_MAX_DIM / 2], b[GEN_BLOCK * SYNTH_MAX_DIM / 2];
  double r[GEN_BLOCK * SYNTH_MAX_DIM / 2], t[GEN_BLOCK * SYNTH_MAX_DIM / 2];
  double z[GEN_BLOCK * SYNTH_MAX_DIM], v[GEN_BLOCK * SYNTH_MAX_DIM];
  const int16_t *base[GEN_BLOCK];
} gen_scratch;

/* n (<= GEN_BLOCK) noisy unit vectors: token i is
 * G(normalise(base[i] / 2^11 + sigma * z_i)), where z_i takes the normals of
 * pairs pair0 + i * dim/2 .. of the stream key.  Outputs (each may be NULL):
 * grid integers out_k [n][dim], bf16 bits out_bf16 [n][dim].
 * The arithmetic is exactly that of the per-token recipe in synth.h (the
 * same IEEE operations in the same order per token, no contraction); the
 * loops run over the block so that they vectorise. */
__attribute__((target_clones("arch=skylake-avx512", "arch=haswell", "default")))
static void noisy_unit_block(gen_scratch *w, int n, int dim, uint64_t key, uint64_t pair0, double sigma,
                             int16_t *out_k, uint16_t *out_bf16) {
  const int np = n * dim / 2, nv = n * dim;
  for (int p = 0; p < np; ++p) {
    const uint64_t c = 2 * (pair0 + (uint64_t)p);
    uint64_t x0 = synth_splitmix64_at(key, c), x1 = synth_splitmix64_at(key, c + 1);
    w->a[p] = ((double)(x0 >> 11) + 0.5) * (1.0 / 9007199254740992.0);
    w->b[p] = ((double)(x1 >> 11) + 0.5) * (1.0 / 9007199254740992.0);
  }
  synth_box_muller(w->a, w->b, w->r, w->t, w->z, np);
  for (int i = 0; i < n; ++i) {
    const int16_t *base = w->base[i];
    double *v = w->v + (size_t)i * dim;
    const double *z = w->z + (size_t)i * dim;
    for (int d = 0; d < dim; ++d) v[d] = base[d] * (1.0 / 2048.0) + sigma * z[d]; /* exact scaling */
  }
  double ss[GEN_BLOCK], inv[GEN_BLOCK];
  for (int i = 0; i < n; ++i) ss[i] = 0.0;
  for (int d = 0; d < dim; ++d) /* each token's sum in dimension order */
    for (int i = 0; i < n; ++i) ss[i] += w->v[(size_t)i * dim + d] * w->v[(size_t)i * dim + d];
  for (int i = 0; i < n; ++i) inv[i] = ss[i] > 0.0 ? 1.0 / sqrt(ss[i]) : 0.0;
  for (int i = 0; i < n; ++i) {
    const double s = inv[i];
    double *v = w->v + (size_t)i * dim;
    for (int d = 0; d < dim; ++d) {
      const double x = v[d] * s;
      /* synth_to_grid without the branch: both roundings, then a select */
      const double small = (x + 3298534883328.0) - 3298534883328.0;
      uint64_t bits;
      memcpy(&bits, &x, sizeof bits);
      bits += ((uint64_t)1 << 44) - 1 + ((bits >> 45) & 1);
      bits &= ~(((uint64_t)1 << 45) - 1);
      double big;
      memcpy(&big, &bits, sizeof big);
      v[d] = fabs(x) < 0.0625 ? small : big;
    }
  }
  if (out_k)
    for (int e = 0; e < nv; ++e) out_k[e] = (int16_t)(w->v[e] * 2048.0); /* exact: a multiple of 2^-11 */
  if (out_bf16)
    for (int e = 0; e < nv; ++e) {
      float f = (float)w->v[e]; /* exact: a bf16 value */
      uint32_t u;
      memcpy(&u, &f, sizeof u);
      out_bf16[e] = (uint16_t)(u >> 16);
    }
}

/* Tokens t0 .. t0+n-1 (n <= GEN_BLOCK) of doc d. */
static void doc_token_block(const synth_ctx *ctx, gen_scratch *w, int64_t d, int64_t t0, int n, int16_t *out_k,
                            uint16_t *out_bf16, int32_t *out_cl) {
  const synth_cfg *c = &ctx->cfg;
  const int dim = c->dim;
  const uint64_t ckey = stream_key(c->seed, STREAM_TOKCLUSTER, (uint64_t)d);
  for (int i = 0; i < n; ++i) {
    int32_t cl = cluster_of(ctx, ckey, t0 + i);
    if (out_cl) out_cl[i] = cl;
    w->base[i] = ctx->cent + (size_t)cl * dim;
  }
  if (!out_k && !out_bf16) return;
  const uint64_t key = stream_key(c->seed, STREAM_TOKNOISE, (uint64_t)d);
  noisy_unit_block(w, n, dim, key, (uint64_t)t0 * (uint64_t)(dim / 2), c->tok_sigma, out_k, out_bf16);
}

/* All L tokens of doc d to rows starting at row. */
static void gen_doc(const synth_ctx *ctx, gen_scratch *w, int64_t d, int32_t L, int64_t row, int16_t *out_k,
                    uint16_t *out_bf16, int32_t *out_cl) {
  const size_t dim = (size_t)ctx->cfg.dim;
  for (int32_t t = 0; t < L; t += GEN_BLOCK) {
    const int n = L - t < GEN_BLOCK ? L - t : GEN_BLOCK;
    const int64_t r = row + t;
    doc_token_block(ctx, w, d, t, n, out_k ? out_k + (size_t)r * dim : NULL,
                    out_bf16 ? out_bf16 + (size_t)r * dim : NULL, out_cl ? out_cl + r : NULL);
  }
}

void synth_doc_tokens_ex(const synth_ctx *ctx, int64_t d0, int64_t d1, const int64_t *tok_off,
                         const int32_t *lens, int16_t *out_k, uint16_t *out_bf16, int32_t *out_cluster,
                         int nthreads) {
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel num_threads(nthreads)
  {
    gen_scratch *w = (gen_scratch *)malloc(sizeof(gen_scratch));
#pragma omp for schedule(dynamic, 64)
    for (int64_t d = d0; d < d1; ++d)
      gen_doc(ctx, w, d, lens[d - d0], tok_off[d - d0], out_k, out_bf16, out_cluster);
    free(w);
  }
}

void synth_doc_tokens(const synth_ctx *ctx, int64_t d0, int64_t d1, const int64_t *tok_off,
                      const int32_t *lens, int16_t *out_k, int32_t *out_cluster, int nthreads) {
  synth_doc_tokens_ex(ctx, d0, d1, tok_off, lens, out_k, NULL, out_cluster, nthreads);
}

void synth_docs_tokens(const synth_ctx *ctx, const int64_t *docs, int64_t n, const int64_t *row_off,
                       int16_t *out_k, int32_t *out_cluster, int nthreads) {
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel num_threads(nthreads)
  {
    gen_scratch *w = (gen_scratch *)malloc(sizeof(gen_scratch));
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i)
      gen_doc(ctx, w, docs[i], doc_length(ctx, docs[i]), row_off[i], out_k, NULL, out_cluster);
    free(w);
  }
}

void synth_queries(const synth_ctx *ctx, uint64_t query_seed, int64_t q0, int64_t q1, int32_t Tq,
                   int16_t *out_k, int64_t *out_src, int nthreads) {
  const synth_cfg *c = &ctx->cfg;
  int dim = c->dim;
  uint64_t qseed = stream_key(c->seed, STREAM_QSEED, query_seed);
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel num_threads(nthreads)
  {
    gen_scratch *w = (gen_scratch *)malloc(sizeof(gen_scratch));
    int16_t *src_tok = (int16_t *)malloc((size_t)GEN_BLOCK * dim * sizeof(int16_t));
#pragma omp for schedule(dynamic, 4)
    for (int64_t q = q0; q < q1; ++q) {
      uint64_t skey = stream_key(qseed, STREAM_QSRC, (uint64_t)q);
      int64_t src = (int64_t)(u01(skey, 0) * (double)c->ndocs);
      if (src >= c->ndocs) src = c->ndocs - 1;
      if (out_src) out_src[q - q0] = src;
      int32_t L = doc_length(ctx, src);
      uint64_t nkey = stream_key(qseed, STREAM_QNOISE, (uint64_t)q);
      for (int32_t j0 = 0; j0 < Tq; j0 += GEN_BLOCK) {
        const int n = Tq - j0 < GEN_BLOCK ? Tq - j0 : GEN_BLOCK;
        /* query token j is the noised source token j mod L */
        for (int i = 0; i < n; ++i)
          doc_token_block(ctx, w, src, (j0 + i) % L, 1, src_tok + (size_t)i * dim, NULL, NULL);
        for (int i = 0; i < n; ++i) w->base[i] = src_tok + (size_t)i * dim;
        noisy_unit_block(w, n, dim, nkey, (uint64_t)j0 * (uint64_t)(dim / 2), c->q_sigma,
                         out_k + ((size_t)(q - q0) * Tq + j0) * dim, NULL);
      }
    }
    free(w);
    free(src_tok);
  }
}
