/*
 * oracle.h - plain, slow CPU reference of the GPU query path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or helper with the GPU library; the two meet only at the
 * seeded input generator (synth/) and at the documented index layout.
 *
 * Paper: "Chimera: Efficient Multi-Vector Retrieval via GPU-CPU
 * Co-Processing".  Every function names the passage it follows.
 *
 * Arithmetic.  Every vector component is on the grid G (bf16 values that
 * are multiples of 2^-11) and is carried as the integer k = x * 2^11.  An
 * inner product is then the exact integer sum of k_a * k_b, in units of
 * 2^-22; every score, partial score and document score below is such an
 * int64 "key".  No floating point is used anywhere in the search; a score
 * leaves the oracle only through orc_key_to_score.
 *
 * Parity status: every function is pinned by the CPU tests (brute force,
 * closed forms, library routines, invariants); none is "parity unpinned".
 */
#ifndef CHIMERA_ORACLE_H
#define CHIMERA_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- Value grid G (the fixed-point reading of the paper's fp32 sums). ---- */
/* Nearest grid value of x, ties to even, as k = x * 2^11. */
int32_t orc_grid_k(double x);
void orc_grid_f32(const float *x, int64_t n, int16_t *k_out);
void orc_grid_bf16(const uint16_t *bits, int64_t n, int16_t *k_out);

/* ---- IVF assignment (Sec. 2.3, inverted file: nearest centroid). ----
 * cid[t] = argmax_c <v_t, c>, ties to the lowest c. */
void orc_assign(const int16_t *tok_k, int64_t ntok, const int16_t *cent_k, int32_t ncent, int32_t dim,
                int32_t *cid, int nthreads);

/* ---- Posting lists (Sec. 2.3; Sec. 3.2 candidate generation). ----
 * Doc-level list of centroid c: ascending distinct docs that own a token
 * assigned to c.  Call with ivf_doc == NULL to get nnz; ivf_off is
 * [ncent+1]. Returns nnz. */
int64_t orc_ivf_docs(const int32_t *cid, const int64_t *doc_off, int64_t ndocs, int32_t ncent,
                     int64_t *ivf_off, int32_t *ivf_doc);
/* Token-level list of centroid c (Sec. 2.3, the IVF over token vectors): the
 * tokens assigned to c in ascending token order.  tok_off is [ncent+1],
 * ivf_tok [ntok]. */
void orc_ivf_tokens(const int32_t *cid, int64_t ntok, int32_t ncent, int64_t *tok_off, int32_t *ivf_tok);

/* ---- Residual quantiser (bucketed residual codes; the paper only names
 * residual compression among related systems, so this is the build's
 * reading: pooled empirical quantiles). ---- */
/* Adds the residual r = v - c_cid of every component to hist[r + 4096]
 * (hist has 8193 int64 bins). */
void orc_residual_hist(const int16_t *tok_k, const int32_t *cid, int64_t ntok, const int16_t *cent_k,
                       int32_t dim, int64_t *hist);
/* B = 2^nbits buckets: cutoffs cut_k[i-1] = Q(i/B), i = 1..B-1; weights
 * w_k[u] = G(Q((2u+1)/(2B))), where Q(a) is the floor(a*n)-th smallest
 * residual (0-based, clamped to n-1).  Returns 0, or -1 if hist is empty. */
int orc_quantizer(const int64_t *hist, int nbits, int32_t *cut_k, int32_t *w_k);
/* code[t][d] = #{i : cut_i < r_{t,d}} (a residual equal to a cutoff goes to
 * the lower bucket). */
void orc_encode(const int16_t *tok_k, const int32_t *cid, int64_t ntok, const int16_t *cent_k, int32_t dim,
                const int32_t *cut_k, int nbits, uint8_t *codes);
/* Packed layout: 2-bit puts dim 4i+s in bits [2s, 2s+1] of byte i; 4-bit puts
 * dim 2i in the low nibble and 2i+1 in the high nibble of byte i. */
void orc_pack(const uint8_t *codes, int64_t ntok, int32_t dim, int nbits, uint8_t *packed);
void orc_unpack(const uint8_t *packed, int64_t ntok, int32_t dim, int nbits, uint8_t *codes);

/* ---- Query path (Alg. 1). ---- */
/* S[j][c] = <Q_j, c> as keys; S is [Tq][ncent]. (Sec. 2.3: a query vector is
 * compared against all centroids.) */
void orc_centroid_scores(const int16_t *q_k, int32_t Tq, const int16_t *cent_k, int32_t ncent, int32_t dim,
                         int64_t *S);
/* C_j = first nprobe centroids in the order (S[j][c] desc, c asc)
 * (Sec. 3.2, candidate generation). Outputs are [Tq][nprobe]. */
void orc_probe(const int64_t *S, int32_t Tq, int32_t ncent, int32_t nprobe, int32_t *cent_ids,
               int64_t *cent_keys);
/* S_Q: ascending docs with a token in a probed list (Sec. 3.2 candidate
 * generation).  out needs ndocs entries; returns |S_Q|. */
int64_t orc_candidates(const int32_t *cent_ids, int32_t Tq, int32_t nprobe, const int64_t *ivf_off,
                       const int32_t *ivf_doc, int64_t ndocs, int32_t *out);
/* Partial Chamfer score F'(V) of every V in S_Q (Sec. 3.2 candidate
 * refinement, the F' definition; S[j][c] stands in for the 1-bit token
 * distance): per query token the max over its probed lists that hold V, 0
 * if none, summed over query tokens.  docs/fprime need ndocs entries;
 * returns |S_Q| with docs ascending. */
int64_t orc_partial_scores(const int64_t *S, const int32_t *cent_ids, int32_t Tq, int32_t ncent,
                           int32_t nprobe, const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs,
                           int32_t *docs, int64_t *fprime);
/* F'(V) of Sec. 3.2 (candidate refinement, Alg. 2) with each retrieved
 * token's own score instead of its centroid's: the tokens L_j retrieved for
 * query token j are those assigned to one of its probed centroids, and a
 * retrieved token t scores as in document scoring, S[j][cid t] +
 * sum_d q_jd w[code_td].  Per query token the max over V's retrieved tokens,
 * 0 if V has none, summed over query tokens.  tok_doc[t] is t's document;
 * codes are unpacked ([ntok][dim]).  docs/fprime need ndocs entries; returns
 * |S_Q| with docs ascending (the same S_Q as orc_partial_scores). */
int64_t orc_partial_scores_res(const int64_t *S, const int32_t *cent_ids, int32_t Tq, int32_t ncent,
                               int32_t nprobe, const int16_t *q_k, int32_t dim, const int32_t *w_k,
                               const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                               const uint8_t *codes, int64_t ndocs, int32_t *docs, int64_t *fprime);
/* First min(k, n) of (key desc, id asc) (Alg. 1 topK; Alg. 2 last step).
 * Returns the count written. */
int64_t orc_topk(const int32_t *ids, const int64_t *keys, int64_t n, int64_t k, int32_t *out_ids,
                 int64_t *out_keys);
/* Complete document score over all tokens of each listed doc (Sec. 3.2
 * document scoring on the GPU; Chamfer, Def. 1) with dequantised tokens
 * c_cid + w[code]: F^(V) = sum_j max_t (S[j][cid t] + sum_d q_jd w[code_td]).
 * Tokens of doc i are rows tok_begin[i] .. tok_begin[i]+tok_len[i]-1 of
 * cid/codes ([rows][dim] unpacked codes). */
void orc_doc_scores(const int64_t *S, int32_t Tq, int32_t ncent, const int16_t *q_k, int32_t dim,
                    const int32_t *w_k, int64_t ndocs_r, const int64_t *tok_begin, const int32_t *tok_len,
                    const int32_t *cid, const uint8_t *codes, int64_t *fhat);
/* Score value of a key: the int64 rounded once to float, times 2^-22. */
float orc_key_to_score(int64_t key);

/* Exact Chamfer similarity (Def. 1) of one query against every doc, over
 * the raw grid tokens. F is [ndocs]. */
void orc_exact_chamfer(const int16_t *q_k, int32_t Tq, int32_t dim, const int16_t *tok_k,
                       const int64_t *doc_off, int64_t ndocs, int64_t *F);

/* Whole path for a batch of queries, in memory (Alg. 1 without the CPU
 * full-bit re-rank), OpenMP over queries only.  refine 0 takes F' from the
 * probed centroids' scores (orc_partial_scores), refine 1 from the retrieved
 * tokens' decoded scores (orc_partial_scores_res, which needs tok_off,
 * ivf_tok and tok_doc; they may be NULL otherwise).  Per query q:
 *   cent_ids/cent_keys [Tq][nprobe]   (may be NULL)
 *   n_sq[q] = |S_Q|                    (may be NULL)
 *   cand/cand_keys [ncand], n_cand[q]  (order: F' desc, doc asc; may be NULL)
 *   ids [k], keys [k]                  (order: F^ desc, doc asc; padded -1 / INT64_MIN)
 * codes are the unpacked codes of every token ([ntok][dim]).  Returns 0. */
int orc_search(const int16_t *cent_k, int32_t ncent, int32_t dim, const int64_t *doc_off, int64_t ndocs,
               const int32_t *cid, const uint8_t *codes, const int32_t *w_k, const int64_t *ivf_off,
               const int32_t *ivf_doc, const int16_t *q_k, int64_t nq, int32_t Tq, int32_t nprobe,
               int32_t ncand, int32_t k, int32_t *cent_ids, int64_t *cent_keys, int64_t *n_sq,
               int32_t *cand, int64_t *cand_keys, int64_t *n_cand, int32_t *ids, int64_t *keys,
               int refine, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
               int nthreads);

/* Only the prune half of orc_search (probe, candidates, F', top-ncand), for
 * corpora whose codes are produced on demand (refine 0; w_k, codes and the
 * token lists may then be NULL). */
int orc_prune_batch(const int16_t *cent_k, int32_t ncent, int32_t dim, int64_t ndocs, const int64_t *ivf_off,
                    const int32_t *ivf_doc, const int16_t *q_k, int64_t nq, int32_t Tq, int32_t nprobe,
                    int32_t ncand, int32_t *cent_ids, int64_t *cent_keys, int64_t *n_sq, int32_t *cand,
                    int64_t *cand_keys, int64_t *n_cand, int refine, const int32_t *w_k, const uint8_t *codes,
                    const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc, int nthreads);

/* ---- RaBitQ codes (Sec. 2.2, Eqs. 2-6, extended to B bits; Sec. 3.1, the
 * 1-bit most significant part; Sec. 4.1, the LUT binary inner product).
 *
 * Readings.  The random orthonormal P is P = H diag(s) / sqrt(D): H the
 * Sylvester Hadamard matrix of order D (H[i][j] = (-1)^popcount(i & j)), s
 * random signs (an input).  Every quantity below is a ratio in which the
 * factor 1/sqrt(D) and the norms of Eq. 2 cancel, so the oracle works with
 * xp = H diag(s) x on grid integers, exactly.  The codeword of Eq. 4 is the
 * y in {-(2^B-1)/2 + u}^D of largest cosine with xp, ties to the smallest
 * |y| (a zero coordinate of xp takes y = +1/2).  The estimate of <q_r, o_r> (Eq. 5, with Eq. 2's norms and Eq. 6's
 * code form) is |o_r|^2 <P q_r, y> / <P o_r, y>, carried as
 *   est = g * float(<xq, 2y> * 2^-12),   g = float(K2 / (A * 1024.0)),
 * xq = H diag(s) q_k, K2 = sum_d o_k[d]^2, A = <xp, 2y> (integers; the last
 * multiply is one fp32 rounding).  The 1-bit part uses y1 = msb - 1/2 and its
 * own factor g1. ---- */
/* xp [n][D] = H diag(s) x for each of the n rows of x_k [n][D]. */
void orc_rabitq_rotate(const int16_t *x_k, int64_t n, int32_t D, const int8_t *signs, int64_t *xp);
/* codes [n][D] in 0..2^B-1 (B <= 8) of the nearest codewords of the rows of
 * xp, and az [n] = <xp, 2y> of each. */
void orc_rabitq_quantize(const int64_t *xp, int64_t n, int32_t D, int B, uint8_t *codes, int64_t *az);
/* Rotation, quantisation and the factors gB (B-bit code) and g1 (its most
 * significant bits) of n tokens; g = 0 for a zero token. */
void orc_rabitq_encode(const int16_t *x_k, int64_t n, int32_t D, const int8_t *signs, int B, uint8_t *codes,
                       float *gB, float *g1);
/* The most significant bits of B-bit codes [n][D], packed: bit i of a token
 * in byte i / 8, bit i % 8. */
void orc_rabitq_pack1(const uint8_t *codes, int64_t n, int32_t D, int B, uint8_t *bits);
/* <xq, b> of a packed 1-bit code through the table of Sec. 4.1:
 * T[j][u] = sum_{t<4} u_t xq[4j+t], summed over the D/4 nibbles. */
int64_t orc_lut_ip(const int64_t *xq, const uint8_t *bits, int32_t D);
/* RaBitQ document scores: for doc i (tokens tok_begin[i] .. + tok_len[i] of
 * codes [..][D] with factors g [..]) F^ = sum_{j<Tq} key(max_t est(q_j, t)),
 * key(x) = rint(x * 2^22) (ties to even); est from the whole code (bits == B)
 * or from its most significant bits (bits == 1).  INT64_MIN for an empty doc. */
void orc_rabitq_doc_scores(const int16_t *q_k, int32_t Tq, int32_t D, const int8_t *signs, int B, int bits,
                           int64_t n, const int64_t *tok_begin, const int32_t *tok_len, const uint8_t *codes,
                           const float *g, int64_t *out);

#ifdef __cplusplus
}
#endif
#endif
