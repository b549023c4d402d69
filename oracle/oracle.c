/*
 * oracle.c - plain, slow CPU reference of the GPU query path.
 *
 * TEST INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's CPU
 * baseline leg).  See oracle.h for the arithmetic convention: everything is
 * exact int64 on grid integers.
 */
#include "oracle.h"

#include <limits.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ grid */

int32_t orc_grid_k(double x) {
  /* Nearest multiple of max(2^-11, bf16 spacing at |x|), ties to even. */
  double a = fabs(x);
  if (a < 0.0625) return (int32_t)nearbyint(x * 2048.0);
  int e;
  frexp(a, &e);
  double q = ldexp(1.0, e - 8);
  double g = nearbyint(x / q) * q;
  return (int32_t)nearbyint(g * 2048.0);
}

void orc_grid_f32(const float *x, int64_t n, int16_t *k_out) {
  for (int64_t i = 0; i < n; ++i) k_out[i] = (int16_t)orc_grid_k((double)x[i]);
}

void orc_grid_bf16(const uint16_t *bits, int64_t n, int16_t *k_out) {
  for (int64_t i = 0; i < n; ++i) {
    uint32_t u = (uint32_t)bits[i] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    k_out[i] = (int16_t)orc_grid_k((double)f);
  }
}

static int64_t dot_k(const int16_t *a, const int16_t *b, int dim) {
  int64_t s = 0;
  for (int d = 0; d < dim; ++d) s += (int64_t)a[d] * (int64_t)b[d];
  return s;
}

/* ------------------------------------------------------------ assignment */

void orc_assign(const int16_t *tok_k, int64_t ntok, const int16_t *cent_k, int32_t ncent, int32_t dim,
                int32_t *cid, int nthreads) {
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel for schedule(dynamic, 256) num_threads(nthreads)
  for (int64_t t = 0; t < ntok; ++t) {
    int64_t best = LLONG_MIN;
    int32_t arg = 0;
    for (int32_t c = 0; c < ncent; ++c) {
      int64_t s = dot_k(tok_k + t * dim, cent_k + (int64_t)c * dim, dim);
      if (s > best) { best = s; arg = c; } /* strict: ties keep the lowest c */
    }
    cid[t] = arg;
  }
}

/* ---------------------------------------------------------- posting lists */

int64_t orc_ivf_docs(const int32_t *cid, const int64_t *doc_off, int64_t ndocs, int32_t ncent,
                     int64_t *ivf_off, int32_t *ivf_doc) {
  /* last[c] = last doc appended to list c, so each doc enters a list once;
   * docs are visited in ascending order, so every list is ascending. */
  int64_t *last = (int64_t *)malloc((size_t)ncent * sizeof(int64_t));
  int64_t *fill = (int64_t *)calloc((size_t)ncent + 1, sizeof(int64_t));
  for (int32_t c = 0; c < ncent; ++c) last[c] = -1;
  for (int64_t v = 0; v < ndocs; ++v)
    for (int64_t t = doc_off[v]; t < doc_off[v + 1]; ++t) {
      int32_t c = cid[t];
      if (last[c] != v) { last[c] = v; fill[c + 1]++; }
    }
  for (int32_t c = 0; c < ncent; ++c) fill[c + 1] += fill[c];
  int64_t nnz = fill[ncent];
  if (ivf_off) memcpy(ivf_off, fill, ((size_t)ncent + 1) * sizeof(int64_t));
  if (ivf_doc) {
    for (int32_t c = 0; c < ncent; ++c) last[c] = -1;
    for (int64_t v = 0; v < ndocs; ++v)
      for (int64_t t = doc_off[v]; t < doc_off[v + 1]; ++t) {
        int32_t c = cid[t];
        if (last[c] != v) { last[c] = v; ivf_doc[fill[c]++] = (int32_t)v; }
      }
  }
  free(last);
  free(fill);
  return nnz;
}

void orc_ivf_tokens(const int32_t *cid, int64_t ntok, int32_t ncent, int64_t *tok_off, int32_t *ivf_tok) {
  int64_t *fill = (int64_t *)calloc((size_t)ncent + 1, sizeof(int64_t));
  for (int64_t t = 0; t < ntok; ++t) fill[cid[t] + 1]++;
  for (int32_t c = 0; c < ncent; ++c) fill[c + 1] += fill[c];
  memcpy(tok_off, fill, ((size_t)ncent + 1) * sizeof(int64_t));
  for (int64_t t = 0; t < ntok; ++t) ivf_tok[fill[cid[t]]++] = (int32_t)t; /* ascending t */
  free(fill);
}

/* ------------------------------------------------------------- quantiser */

void orc_residual_hist(const int16_t *tok_k, const int32_t *cid, int64_t ntok, const int16_t *cent_k,
                       int32_t dim, int64_t *hist) {
  for (int64_t t = 0; t < ntok; ++t) {
    const int16_t *c = cent_k + (int64_t)cid[t] * dim;
    for (int d = 0; d < dim; ++d) hist[(int)tok_k[t * dim + d] - (int)c[d] + 4096]++;
  }
}

/* floor(num * n / den)-th smallest value (0-based, clamped to n - 1). */
static int32_t hist_quantile(const int64_t *hist, int64_t n, int64_t num, int64_t den) {
  int64_t idx = (num * n) / den;
  if (idx > n - 1) idx = n - 1;
  int64_t seen = 0;
  for (int b = 0; b < 8193; ++b) {
    seen += hist[b];
    if (seen > idx) return b - 4096;
  }
  return 4096;
}

int orc_quantizer(const int64_t *hist, int nbits, int32_t *cut_k, int32_t *w_k) {
  int64_t n = 0;
  for (int b = 0; b < 8193; ++b) n += hist[b];
  if (n == 0) return -1;
  int B = 1 << nbits;
  for (int i = 1; i < B; ++i) cut_k[i - 1] = hist_quantile(hist, n, i, B);
  for (int u = 0; u < B; ++u) {
    int32_t r = hist_quantile(hist, n, 2 * u + 1, 2 * B);
    w_k[u] = orc_grid_k((double)r / 2048.0);
  }
  return 0;
}

void orc_encode(const int16_t *tok_k, const int32_t *cid, int64_t ntok, const int16_t *cent_k, int32_t dim,
                const int32_t *cut_k, int nbits, uint8_t *codes) {
  int B = 1 << nbits;
  for (int64_t t = 0; t < ntok; ++t) {
    const int16_t *c = cent_k + (int64_t)cid[t] * dim;
    for (int d = 0; d < dim; ++d) {
      int32_t r = (int32_t)tok_k[t * dim + d] - (int32_t)c[d];
      int code = 0;
      for (int i = 0; i < B - 1; ++i)
        if (cut_k[i] < r) code++;
      codes[t * dim + d] = (uint8_t)code;
    }
  }
}

void orc_pack(const uint8_t *codes, int64_t ntok, int32_t dim, int nbits, uint8_t *packed) {
  int per = 8 / nbits;                 /* codes per byte */
  int64_t bpt = (int64_t)dim / per;    /* bytes per token */
  for (int64_t t = 0; t < ntok; ++t)
    for (int64_t i = 0; i < bpt; ++i) {
      uint32_t byte = 0;
      for (int s = 0; s < per; ++s) byte |= (uint32_t)codes[t * dim + i * per + s] << (nbits * s);
      packed[t * bpt + i] = (uint8_t)byte;
    }
}

void orc_unpack(const uint8_t *packed, int64_t ntok, int32_t dim, int nbits, uint8_t *codes) {
  int per = 8 / nbits;
  int64_t bpt = (int64_t)dim / per;
  uint32_t mask = (1u << nbits) - 1u;
  for (int64_t t = 0; t < ntok; ++t)
    for (int64_t i = 0; i < bpt; ++i)
      for (int s = 0; s < per; ++s)
        codes[t * dim + i * per + s] = (uint8_t)((packed[t * bpt + i] >> (nbits * s)) & mask);
}

/* ------------------------------------------------------------ query path */

void orc_centroid_scores(const int16_t *q_k, int32_t Tq, const int16_t *cent_k, int32_t ncent, int32_t dim,
                         int64_t *S) {
  for (int32_t j = 0; j < Tq; ++j)
    for (int32_t c = 0; c < ncent; ++c)
      S[(int64_t)j * ncent + c] = dot_k(q_k + (int64_t)j * dim, cent_k + (int64_t)c * dim, dim);
}

/* (key desc, id asc) ordering: does (ka, ia) come before (kb, ib)? */
static int before(int64_t ka, int64_t ia, int64_t kb, int64_t ib) {
  return ka > kb || (ka == kb && ia < ib);
}

void orc_probe(const int64_t *S, int32_t Tq, int32_t ncent, int32_t nprobe, int32_t *cent_ids,
               int64_t *cent_keys) {
  /* Insertion into a sorted list of the nprobe best so far. */
  for (int32_t j = 0; j < Tq; ++j) {
    int32_t *ids = cent_ids + (int64_t)j * nprobe;
    int64_t *keys = cent_keys + (int64_t)j * nprobe;
    int32_t n = 0;
    for (int32_t c = 0; c < ncent; ++c) {
      int64_t s = S[(int64_t)j * ncent + c];
      if (n == nprobe && !before(s, c, keys[n - 1], ids[n - 1])) continue;
      int32_t p = n < nprobe ? n++ : nprobe - 1;
      while (p > 0 && before(s, c, keys[p - 1], ids[p - 1])) {
        keys[p] = keys[p - 1];
        ids[p] = ids[p - 1];
        --p;
      }
      keys[p] = s;
      ids[p] = c;
    }
  }
}

int64_t orc_candidates(const int32_t *cent_ids, int32_t Tq, int32_t nprobe, const int64_t *ivf_off,
                       const int32_t *ivf_doc, int64_t ndocs, int32_t *out) {
  uint8_t *in = (uint8_t *)calloc((size_t)ndocs, 1);
  for (int64_t e = 0; e < (int64_t)Tq * nprobe; ++e) {
    int32_t c = cent_ids[e];
    for (int64_t p = ivf_off[c]; p < ivf_off[c + 1]; ++p) in[ivf_doc[p]] = 1;
  }
  int64_t n = 0;
  for (int64_t v = 0; v < ndocs; ++v)
    if (in[v]) out[n++] = (int32_t)v;
  free(in);
  return n;
}

int64_t orc_partial_scores(const int64_t *S, const int32_t *cent_ids, int32_t Tq, int32_t ncent,
                           int32_t nprobe, const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs,
                           int32_t *docs, int64_t *fprime) {
  int64_t *best = (int64_t *)malloc((size_t)ndocs * sizeof(int64_t));
  int64_t *acc = (int64_t *)calloc((size_t)ndocs, sizeof(int64_t));
  uint8_t *has = (uint8_t *)calloc((size_t)ndocs, 1);
  uint8_t *in = (uint8_t *)calloc((size_t)ndocs, 1);
  int32_t *touched = (int32_t *)malloc((size_t)ndocs * sizeof(int32_t));
  for (int32_t j = 0; j < Tq; ++j) {
    int64_t nt = 0;
    for (int32_t r = 0; r < nprobe; ++r) {
      int32_t c = cent_ids[(int64_t)j * nprobe + r];
      int64_t s = S[(int64_t)j * ncent + c];
      for (int64_t p = ivf_off[c]; p < ivf_off[c + 1]; ++p) {
        int32_t v = ivf_doc[p];
        in[v] = 1;
        if (!has[v]) { has[v] = 1; best[v] = s; touched[nt++] = v; }
        else if (s > best[v]) best[v] = s;
      }
    }
    /* V with no retrieved token for this j contributes 0 (not touched). */
    for (int64_t i = 0; i < nt; ++i) { acc[touched[i]] += best[touched[i]]; has[touched[i]] = 0; }
  }
  int64_t n = 0;
  for (int64_t v = 0; v < ndocs; ++v)
    if (in[v]) { docs[n] = (int32_t)v; fprime[n] = acc[v]; ++n; }
  free(best); free(acc); free(has); free(in); free(touched);
  return n;
}

int64_t orc_partial_scores_res(const int64_t *S, const int32_t *cent_ids, int32_t Tq, int32_t ncent,
                               int32_t nprobe, const int16_t *q_k, int32_t dim, const int32_t *w_k,
                               const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                               const uint8_t *codes, int64_t ndocs, int32_t *docs, int64_t *fprime) {
  int64_t *best = (int64_t *)malloc((size_t)ndocs * sizeof(int64_t));
  int64_t *acc = (int64_t *)calloc((size_t)ndocs, sizeof(int64_t));
  uint8_t *has = (uint8_t *)calloc((size_t)ndocs, 1);
  uint8_t *in = (uint8_t *)calloc((size_t)ndocs, 1);
  int32_t *touched = (int32_t *)malloc((size_t)ndocs * sizeof(int32_t));
  for (int32_t j = 0; j < Tq; ++j) {
    const int16_t *q = q_k + (int64_t)j * dim;
    int64_t nt = 0;
    for (int32_t r = 0; r < nprobe; ++r) {
      int32_t c = cent_ids[(int64_t)j * nprobe + r];
      for (int64_t p = tok_off[c]; p < tok_off[c + 1]; ++p) {
        int64_t t = ivf_tok[p];
        int64_t s = S[(int64_t)j * ncent + c];
        for (int d = 0; d < dim; ++d) s += (int64_t)q[d] * (int64_t)w_k[codes[t * dim + d]];
        int32_t v = tok_doc[t];
        in[v] = 1;
        if (!has[v]) { has[v] = 1; best[v] = s; touched[nt++] = v; }
        else if (s > best[v]) best[v] = s;
      }
    }
    /* V with no retrieved token for this j contributes 0 (not touched). */
    for (int64_t i = 0; i < nt; ++i) { acc[touched[i]] += best[touched[i]]; has[touched[i]] = 0; }
  }
  int64_t n = 0;
  for (int64_t v = 0; v < ndocs; ++v)
    if (in[v]) { docs[n] = (int32_t)v; fprime[n] = acc[v]; ++n; }
  free(best); free(acc); free(has); free(in); free(touched);
  return n;
}

typedef struct { int64_t key; int32_t id; } kid;

static int cmp_kid(const void *a, const void *b) {
  const kid *x = (const kid *)a, *y = (const kid *)b;
  if (x->key != y->key) return x->key > y->key ? -1 : 1;
  return (x->id > y->id) - (x->id < y->id);
}

int64_t orc_topk(const int32_t *ids, const int64_t *keys, int64_t n, int64_t k, int32_t *out_ids,
                 int64_t *out_keys) {
  kid *a = (kid *)malloc((size_t)(n > 0 ? n : 1) * sizeof(kid));
  for (int64_t i = 0; i < n; ++i) { a[i].key = keys[i]; a[i].id = ids[i]; }
  qsort(a, (size_t)n, sizeof(kid), cmp_kid);
  int64_t m = n < k ? n : k;
  for (int64_t i = 0; i < m; ++i) { out_ids[i] = a[i].id; out_keys[i] = a[i].key; }
  free(a);
  return m;
}

void orc_doc_scores(const int64_t *S, int32_t Tq, int32_t ncent, const int16_t *q_k, int32_t dim,
                    const int32_t *w_k, int64_t ndocs_r, const int64_t *tok_begin, const int32_t *tok_len,
                    const int32_t *cid, const uint8_t *codes, int64_t *fhat) {
  for (int64_t i = 0; i < ndocs_r; ++i) {
    int64_t total = 0;
    for (int32_t j = 0; j < Tq; ++j) {
      const int16_t *q = q_k + (int64_t)j * dim;
      int64_t m = LLONG_MIN;
      for (int32_t u = 0; u < tok_len[i]; ++u) {
        int64_t t = tok_begin[i] + u;
        int64_t s = S[(int64_t)j * ncent + cid[t]];
        for (int d = 0; d < dim; ++d) s += (int64_t)q[d] * (int64_t)w_k[codes[t * dim + d]];
        if (s > m) m = s;
      }
      total += m;
    }
    fhat[i] = total;
  }
}

float orc_key_to_score(int64_t key) { return (float)key * (1.0f / 4194304.0f); }

void orc_exact_chamfer(const int16_t *q_k, int32_t Tq, int32_t dim, const int16_t *tok_k,
                       const int64_t *doc_off, int64_t ndocs, int64_t *F) {
  for (int64_t v = 0; v < ndocs; ++v) {
    int64_t total = 0;
    for (int32_t j = 0; j < Tq; ++j) {
      int64_t m = LLONG_MIN;
      for (int64_t t = doc_off[v]; t < doc_off[v + 1]; ++t) {
        int64_t s = dot_k(q_k + (int64_t)j * dim, tok_k + t * dim, dim);
        if (s > m) m = s;
      }
      total += m;
    }
    F[v] = total;
  }
}

/* ---------------------------------------------------------- batch drivers */

/* Probe, candidates, F' and top-ncand of one query; S is [Tq][ncent]. */
/* What refine 1 needs besides the doc-level lists. */
typedef struct {
  int refine;
  const int32_t *w_k;
  const uint8_t *codes;
  const int64_t *tok_off;
  const int32_t *ivf_tok;
  const int32_t *tok_doc;
} refine_in;

static int64_t prune_one(const int16_t *cent_k, int32_t ncent, int32_t dim, int64_t ndocs, const int64_t *ivf_off,
                         const int32_t *ivf_doc, const int16_t *q, int32_t Tq, int32_t nprobe, int32_t ncand,
                         const refine_in *rf, int64_t *S, int32_t *ci, int64_t *ck, int64_t *n_sq, int32_t *cand,
                         int64_t *cand_keys, int32_t *docs, int64_t *fp) {
  orc_centroid_scores(q, Tq, cent_k, ncent, dim, S);
  orc_probe(S, Tq, ncent, nprobe, ci, ck);
  int64_t nsq = rf->refine ? orc_partial_scores_res(S, ci, Tq, ncent, nprobe, q, dim, rf->w_k, rf->tok_off,
                                                    rf->ivf_tok, rf->tok_doc, rf->codes, ndocs, docs, fp)
                           : orc_partial_scores(S, ci, Tq, ncent, nprobe, ivf_off, ivf_doc, ndocs, docs, fp);
  if (n_sq) *n_sq = nsq;
  return orc_topk(docs, fp, nsq, ncand, cand, cand_keys);
}

int orc_prune_batch(const int16_t *cent_k, int32_t ncent, int32_t dim, int64_t ndocs, const int64_t *ivf_off,
                    const int32_t *ivf_doc, const int16_t *q_k, int64_t nq, int32_t Tq, int32_t nprobe,
                    int32_t ncand, int32_t *cent_ids, int64_t *cent_keys, int64_t *n_sq, int32_t *cand,
                    int64_t *cand_keys, int64_t *n_cand, int refine, const int32_t *w_k, const uint8_t *codes,
                    const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc, int nthreads) {
  const refine_in rf = {refine, w_k, codes, tok_off, ivf_tok, tok_doc};
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel num_threads(nthreads)
  {
    int64_t *S = (int64_t *)malloc((size_t)Tq * ncent * sizeof(int64_t));
    int32_t *ci = (int32_t *)malloc((size_t)Tq * nprobe * sizeof(int32_t));
    int64_t *ck = (int64_t *)malloc((size_t)Tq * nprobe * sizeof(int64_t));
    int32_t *docs = (int32_t *)malloc((size_t)(ndocs > 0 ? ndocs : 1) * sizeof(int32_t));
    int64_t *fp = (int64_t *)malloc((size_t)(ndocs > 0 ? ndocs : 1) * sizeof(int64_t));
#pragma omp for schedule(dynamic, 1)
    for (int64_t qi = 0; qi < nq; ++qi) {
      int64_t nsq = 0;
      int64_t nc = prune_one(cent_k, ncent, dim, ndocs, ivf_off, ivf_doc, q_k + qi * Tq * dim, Tq, nprobe, ncand,
                             &rf, S, ci, ck, &nsq, cand + qi * ncand, cand_keys + qi * ncand, docs, fp);
      if (cent_ids) memcpy(cent_ids + qi * Tq * nprobe, ci, (size_t)Tq * nprobe * sizeof(int32_t));
      if (cent_keys) memcpy(cent_keys + qi * Tq * nprobe, ck, (size_t)Tq * nprobe * sizeof(int64_t));
      if (n_sq) n_sq[qi] = nsq;
      n_cand[qi] = nc;
    }
    free(S); free(ci); free(ck); free(docs); free(fp);
  }
  return 0;
}

int orc_search(const int16_t *cent_k, int32_t ncent, int32_t dim, const int64_t *doc_off, int64_t ndocs,
               const int32_t *cid, const uint8_t *codes, const int32_t *w_k, const int64_t *ivf_off,
               const int32_t *ivf_doc, const int16_t *q_k, int64_t nq, int32_t Tq, int32_t nprobe,
               int32_t ncand, int32_t k, int32_t *cent_ids, int64_t *cent_keys, int64_t *n_sq,
               int32_t *cand, int64_t *cand_keys, int64_t *n_cand, int32_t *ids, int64_t *keys,
               int refine, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
               int nthreads) {
  const refine_in rf = {refine, w_k, codes, tok_off, ivf_tok, tok_doc};
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#endif
#pragma omp parallel num_threads(nthreads)
  {
    int64_t *S = (int64_t *)malloc((size_t)Tq * ncent * sizeof(int64_t));
    int32_t *ci = (int32_t *)malloc((size_t)Tq * nprobe * sizeof(int32_t));
    int64_t *ck = (int64_t *)malloc((size_t)Tq * nprobe * sizeof(int64_t));
    int32_t *docs = (int32_t *)malloc((size_t)(ndocs > 0 ? ndocs : 1) * sizeof(int32_t));
    int64_t *fp = (int64_t *)malloc((size_t)(ndocs > 0 ? ndocs : 1) * sizeof(int64_t));
    int32_t *r = (int32_t *)malloc((size_t)ncand * sizeof(int32_t));
    int64_t *rk = (int64_t *)malloc((size_t)ncand * sizeof(int64_t));
    int64_t *tb = (int64_t *)malloc((size_t)ncand * sizeof(int64_t));
    int32_t *tl = (int32_t *)malloc((size_t)ncand * sizeof(int32_t));
    int64_t *fh = (int64_t *)malloc((size_t)ncand * sizeof(int64_t));
#pragma omp for schedule(dynamic, 1)
    for (int64_t qi = 0; qi < nq; ++qi) {
      const int16_t *q = q_k + qi * Tq * dim;
      int64_t nsq = 0;
      int64_t nc = prune_one(cent_k, ncent, dim, ndocs, ivf_off, ivf_doc, q, Tq, nprobe, ncand, &rf, S, ci, ck,
                             &nsq, r, rk, docs, fp);
      if (cent_ids) memcpy(cent_ids + qi * Tq * nprobe, ci, (size_t)Tq * nprobe * sizeof(int32_t));
      if (cent_keys) memcpy(cent_keys + qi * Tq * nprobe, ck, (size_t)Tq * nprobe * sizeof(int64_t));
      if (n_sq) n_sq[qi] = nsq;
      if (n_cand) n_cand[qi] = nc;
      if (cand) memcpy(cand + qi * ncand, r, (size_t)nc * sizeof(int32_t));
      if (cand_keys) memcpy(cand_keys + qi * ncand, rk, (size_t)nc * sizeof(int64_t));
      for (int64_t i = 0; i < nc; ++i) { tb[i] = doc_off[r[i]]; tl[i] = (int32_t)(doc_off[r[i] + 1] - doc_off[r[i]]); }
      orc_doc_scores(S, Tq, ncent, q, dim, w_k, nc, tb, tl, cid, codes, fh);
      int64_t m = orc_topk(r, fh, nc, k, ids + qi * k, keys + qi * k);
      for (int64_t i = m; i < k; ++i) { ids[qi * k + i] = -1; keys[qi * k + i] = LLONG_MIN; }
    }
    free(S); free(ci); free(ck); free(docs); free(fp); free(r); free(rk); free(tb); free(tl); free(fh);
  }
  return 0;
}

/* ------------------------------------------------------------- RaBitQ */

void orc_rabitq_rotate(const int16_t *x_k, int64_t n, int32_t D, const int8_t *signs, int64_t *xp) {
  for (int64_t r = 0; r < n; ++r)
    for (int32_t i = 0; i < D; ++i) {
      int64_t s = 0;
      for (int32_t j = 0; j < D; ++j) {
        const int64_t h = (__builtin_popcount((unsigned)(i & j)) & 1) ? -1 : 1;
        s += h * (int64_t)signs[j] * (int64_t)x_k[r * D + j];
      }
      xp[r * D + i] = s;
    }
}

/* t = num / den at which coordinate i of the rounding path steps up */
typedef struct {
  int64_t num, den;
  int32_t i;
} rq_event;

static int rq_event_cmp(const void *pa, const void *pb) {
  const rq_event *a = (const rq_event *)pa, *b = (const rq_event *)pb;
  const int64_t l = a->num * b->den, r = b->num * a->den;
  if (l != r) return l < r ? -1 : 1;
  return a->i < b->i ? -1 : (a->i > b->i ? 1 : 0);
}

/* The nearest codeword of one vector.  As t grows, rounding t * xp to the
 * nearest point of the half-integer grid (clamped to |y| <= (2^B-1)/2) visits
 * a sequence of codewords; the codeword of largest cosine lies on it (it is a
 * nearest grid point of some t * xp, and of the points tied at a step of
 * several coordinates at once the cosine is largest at the two ends, since
 * every stepping coordinate adds the same ratio of <xp, 2y> to |2y|^2).  So
 * the candidates are the codewords between consecutive distinct step values
 * of t, compared exactly: A / sqrt(N) with A = <xp, 2y>, N = |2y|^2. */
static void rq_quantize_one(const int64_t *xp, int32_t D, int B, uint8_t *code, int64_t *az, rq_event *ev,
                            int32_t *level, int32_t *best) {
  const int32_t half = 1 << (B - 1);
  int64_t A = 0, N = D;
  int64_t ne = 0;
  for (int32_t i = 0; i < D; ++i) {
    level[i] = 0;
    best[i] = 0;
    const int64_t a = xp[i] < 0 ? -xp[i] : xp[i];
    A += a;
    if (a == 0) continue;
    for (int32_t m = 1; m < half; ++m) {
      ev[ne].num = m;
      ev[ne].den = a;
      ev[ne].i = i;
      ++ne;
    }
  }
  qsort(ev, (size_t)ne, sizeof(rq_event), rq_event_cmp);
  int64_t bestA = A, bestN = N;
  for (int64_t e = 0; e < ne;) {
    int64_t f = e;
    while (f < ne && ev[f].num * ev[e].den == ev[e].num * ev[f].den) {
      const int32_t i = ev[f].i;
      const int64_t a = xp[i] < 0 ? -xp[i] : xp[i];
      A += 2 * a;
      N += 8 * (int64_t)level[i] + 8;
      level[i] += 1;
      ++f;
    }
    e = f;
    /* A / sqrt(N) > bestA / sqrt(bestN), both A > 0 */
    if ((__int128)A * A * bestN > (__int128)bestA * bestA * N) {
      bestA = A;
      bestN = N;
      memcpy(best, level, sizeof(int32_t) * (size_t)D);
    }
  }
  for (int32_t i = 0; i < D; ++i) code[i] = (uint8_t)(xp[i] < 0 ? half - 1 - best[i] : half + best[i]);
  *az = bestA;
}

void orc_rabitq_quantize(const int64_t *xp, int64_t n, int32_t D, int B, uint8_t *codes, int64_t *az) {
  rq_event *ev = (rq_event *)malloc(sizeof(rq_event) * (size_t)D * (size_t)(1 << (B - 1)));
  int32_t *level = (int32_t *)malloc(sizeof(int32_t) * (size_t)D);
  int32_t *best = (int32_t *)malloc(sizeof(int32_t) * (size_t)D);
  for (int64_t r = 0; r < n; ++r) rq_quantize_one(xp + r * D, D, B, codes + r * D, az + r, ev, level, best);
  free(ev);
  free(level);
  free(best);
}

static float rq_factor(int64_t k2, int64_t a) {
  return a == 0 ? 0.0f : (float)((double)k2 / ((double)a * 1024.0));
}

void orc_rabitq_encode(const int16_t *x_k, int64_t n, int32_t D, const int8_t *signs, int B, uint8_t *codes,
                       float *gB, float *g1) {
  int64_t *xp = (int64_t *)malloc(sizeof(int64_t) * (size_t)D);
  for (int64_t r = 0; r < n; ++r) {
    orc_rabitq_rotate(x_k + r * D, 1, D, signs, xp);
    int64_t az = 0;
    orc_rabitq_quantize(xp, 1, D, B, codes + r * D, &az);
    int64_t k2 = 0, a1 = 0;
    for (int32_t i = 0; i < D; ++i) {
      k2 += (int64_t)x_k[r * D + i] * x_k[r * D + i];
      a1 += xp[i] < 0 ? -xp[i] : xp[i]; /* <xp, 2 y1> with y1 = msb - 1/2 */
    }
    gB[r] = rq_factor(k2, az);
    g1[r] = rq_factor(k2, a1);
  }
  free(xp);
}

void orc_rabitq_pack1(const uint8_t *codes, int64_t n, int32_t D, int B, uint8_t *bits) {
  memset(bits, 0, (size_t)(n * D / 8));
  for (int64_t r = 0; r < n; ++r)
    for (int32_t i = 0; i < D; ++i)
      if (codes[r * D + i] >> (B - 1)) bits[r * (D / 8) + i / 8] |= (uint8_t)(1u << (i % 8));
}

int64_t orc_lut_ip(const int64_t *xq, const uint8_t *bits, int32_t D) {
  int64_t s = 0;
  for (int32_t j = 0; j < D / 4; ++j) {
    int64_t T[16];
    for (int u = 0; u < 16; ++u) {
      T[u] = 0;
      for (int t = 0; t < 4; ++t)
        if ((u >> t) & 1) T[u] += xq[4 * j + t];
    }
    const int u = (bits[(4 * j) / 8] >> ((4 * j) % 8)) & 15;
    s += T[u];
  }
  return s;
}

/* est = g * float(<xq, 2y> * 2^-12) */
static float rq_est(const int64_t *xq, const uint8_t *code, int32_t D, int B, int bits, float g) {
  int64_t ip = 0;
  for (int32_t i = 0; i < D; ++i) {
    const int64_t z = bits == 1 ? (code[i] >> (B - 1) ? 1 : -1) : 2 * (int64_t)code[i] - ((1 << B) - 1);
    ip += xq[i] * z;
  }
  const float x = (float)ldexp((double)ip, -12);
  return g * x;
}

void orc_rabitq_doc_scores(const int16_t *q_k, int32_t Tq, int32_t D, const int8_t *signs, int B, int bits,
                           int64_t n, const int64_t *tok_begin, const int32_t *tok_len, const uint8_t *codes,
                           const float *g, int64_t *out) {
  int64_t *xq = (int64_t *)malloc(sizeof(int64_t) * (size_t)Tq * D);
  orc_rabitq_rotate(q_k, Tq, D, signs, xq);
  for (int64_t i = 0; i < n; ++i) {
    if (tok_len[i] <= 0) {
      out[i] = LLONG_MIN;
      continue;
    }
    int64_t f = 0;
    for (int32_t j = 0; j < Tq; ++j) {
      float m = -INFINITY;
      for (int32_t t = 0; t < tok_len[i]; ++t) {
        const int64_t tok = tok_begin[i] + t;
        const float e = rq_est(xq + (int64_t)j * D, codes + tok * D, D, B, bits, g[tok]);
        if (e > m) m = e;
      }
      f += (int64_t)nearbyint((double)m * 4194304.0);
    }
    out[i] = f;
  }
  free(xq);
}
