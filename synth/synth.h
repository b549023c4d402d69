/*
 * synth.h - seeded synthetic multi-vector corpora (input generator only).
 *
 * This module produces the *inputs* of the retrieval method: centroid
 * vectors, document token vectors, the centroid each token was drawn around,
 * document lengths and query token vectors.  It holds none of the method's
 * arithmetic (no scoring, probing, quantisation or selection); both the CPU
 * oracle and the GPU library consume what it produces.
 *
 * Randomness is counter based: every value is a pure function of
 * (seed, stream id, object index, counter), using the SplitMix64 output
 * function (Steele, Lea & Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014) on the state  key + (counter + 1) * golden_gamma,
 * and Box-Muller normals (Box & Muller, 1958).  Any document or query can
 * therefore be regenerated on its own, in any order and on any thread.
 *
 * Every emitted vector component lies on the value grid G: bf16 numbers that
 * are integer multiples of 2^-11.  Components are returned as the int16
 * integer k = x * 2^11 (|k| <= 2048).
 *
 * Recipe (one corpus):
 *   centroid c       = G(normalise(z)),            z ~ N(0, I_dim)
 *   doc length L_d   = fixed | clip(round(exp(mu + s*z)), lo, hi) | uniform[lo, hi]
 *   token cluster    = uniform over ncent, or Zipf(s) rank mapped through a
 *                      seeded permutation of centroid ids
 *   token vector     = G(normalise(c_cluster + tok_sigma * z))
 *   query source doc = uniform over docs
 *   query token j    = G(normalise(v_{src, j mod L_src} + q_sigma * z))
 */
#ifndef CHIMERA_SYNTH_H
#define CHIMERA_SYNTH_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { SYNTH_LEN_FIXED = 0, SYNTH_LEN_LOGNORMAL = 1, SYNTH_LEN_UNIFORM = 2 };
enum { SYNTH_POP_UNIFORM = 0, SYNTH_POP_ZIPF = 1 };

typedef struct {
  uint64_t seed;
  int64_t ndocs;
  int32_t ncent;
  int32_t dim;
  int32_t len_kind;      /* SYNTH_LEN_* */
  int32_t len_lo, len_hi;/* fixed: len_lo; lognormal: clip range; uniform: inclusive range */
  double len_mean;       /* lognormal arithmetic mean before clipping */
  double len_sigma;      /* lognormal sigma in log space */
  int32_t pop_kind;      /* SYNTH_POP_* */
  double zipf_s;         /* Zipf exponent */
  double tok_sigma;      /* per-dimension noise of doc tokens */
  double q_sigma;        /* per-dimension noise of query tokens */
} synth_cfg;

typedef struct synth_ctx synth_ctx;

/* Builds the context: centroids, the Zipf table and the rank->id permutation.
 * Returns NULL on bad configuration or allocation failure. */
synth_ctx *synth_create(const synth_cfg *cfg);  /* dim even and at most 1024 */
void synth_free(synth_ctx *ctx);

/* Centroids as grid integers, [ncent][dim]. The pointer is owned by ctx. */
const int16_t *synth_centroids(const synth_ctx *ctx);

/* Document lengths for docs [d0, d1) into out[d1-d0]. */
void synth_doc_lengths(const synth_ctx *ctx, int64_t d0, int64_t d1, int32_t *out);

/* Tokens of docs [d0, d1).  tok_off[i] is the row of doc d0+i inside out_k /
 * out_cluster (rows are contiguous, doc after doc); lens[i] its length.
 * out_k is [rows][dim] int16, out_cluster is [rows] int32 (the centroid each
 * token was drawn around).  Either output may be NULL.  Uses nthreads
 * OpenMP threads (<= 0: library default). */
void synth_doc_tokens(const synth_ctx *ctx, int64_t d0, int64_t d1,
                      const int64_t *tok_off, const int32_t *lens,
                      int16_t *out_k, int32_t *out_cluster, int nthreads);

/* As synth_doc_tokens, with the components also (or only) as bf16 bit
 * patterns out_bf16 [rows][dim] (every grid value is a bf16 value).  Any
 * output may be NULL. */
void synth_doc_tokens_ex(const synth_ctx *ctx, int64_t d0, int64_t d1, const int64_t *tok_off,
                         const int32_t *lens, int16_t *out_k, uint16_t *out_bf16, int32_t *out_cluster,
                         int nthreads);

/* Queries [q0, q1) with Tq tokens each: out_k is [q1-q0][Tq][dim] int16,
 * out_src[q1-q0] the source document (may be NULL).  query_seed separates
 * query sets drawn from one corpus. */
/* Tokens of an arbitrary list of docs: doc docs[i] goes to rows
 * row_off[i] .. row_off[i] + len - 1 of out_k [rows][dim] / out_cluster. */
void synth_docs_tokens(const synth_ctx *ctx, const int64_t *docs, int64_t n, const int64_t *row_off,
                       int16_t *out_k, int32_t *out_cluster, int nthreads);
void synth_queries(const synth_ctx *ctx, uint64_t query_seed, int64_t q0, int64_t q1,
                   int32_t Tq, int16_t *out_k, int64_t *out_src, int nthreads);

/* Exposed for tests of the generator itself. */
uint64_t synth_splitmix64_at(uint64_t state, uint64_t n);
double synth_to_grid(double x);

#ifdef __cplusplus
}
#endif
#endif
