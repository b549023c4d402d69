/*
 * chimera.h - C ABI of the MI355X (gfx950) multi-vector query path.
 *
 * Method: "Chimera: Efficient Multi-Vector Retrieval via GPU-CPU
 * Co-Processing".  The library implements the GPU-resident part of the
 * query pipeline of Alg. 1: candidate generation (Sec. 3.2), candidate
 * refinement with a partial Chamfer score (Sec. 3.2, Alg. 2) and document
 * scoring of the refined candidates over compressed codes (Sec. 3.2, the
 * GPU half of Alg. 3), returning the top-k documents by Chamfer similarity
 * (Def. 1) as the MVR problem asks (Def. 2, Eq. 1).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every call returns an int status: CHIMERA_OK (0) or a CHIMERA_E_* code.
 *    chimera_last_error() then holds a message for the calling thread.
 *  - Arguments are validated on the host before anything is launched; a call
 *    that fails validation leaves every output untouched.
 *  - "device pointer" means memory on the index's HIP device (hipMalloc or a
 *    torch CUDA tensor).  The caller owns every pointer it passes in; the
 *    index handle owns all device memory of the index and its scratch.
 *  - Search calls are asynchronous on `hip_stream` (a hipStream_t; NULL is
 *    the null stream); outputs are valid after that stream synchronises.
 *    Successive calls on one index may use different streams: the library
 *    orders them on its scratch.  Concurrent host calls on one index return
 *    CHIMERA_E_BUSY.
 *  - Scratch: a search runs its batch in sub-batches of as many queries as
 *    fit a scratch budget of CHIMERA_SCRATCH_MB MiB (environment, read at
 *    each call; default 131072, at least 16), allocated on the index's
 *    device on first need (at most 9/8 of what the batch needs) and kept with
 *    the index.  At 8.8M documents a query needs about 72 MB (its S^T table
 *    and F' row), so the default takes about 1,900 queries per sub-batch, and
 *    a 4096-query batch runs in 3 sub-batches of 1,366 (about 110 GB).  If
 *    the device cannot hold the arena (other allocations on it), the
 *    sub-batches are halved until it fits; CHIMERA_E_NOMEM only when the
 *    scratch of a single query does not fit.  A sub-batch also holds at
 *    most 2^28 / ncand queries, so that each launch's work-item count fits
 *    in 32 bits.
 *  - Value grid G: all vector values are used as bf16 numbers that are
 *    integer multiples of 2^-11.  Inputs are rounded onto G (nearest, ties to
 *    even), which leaves grid values unchanged.  On G every product is an
 *    exact multiple of 2^-22, and float32 holds every such multiple below 4
 *    in magnitude, so a sum of products is exact in any order while its
 *    partial sums stay below 4.  A query token q is scored against centroid
 *    c plus decoded residual w, so by Cauchy-Schwarz the scores are exact
 *    and independent of the summation order when
 *        ||q|| * (max_c ||c|| + sqrt(dim) * max_u |w_u|) < 4,
 *    i.e. every query token's L2 norm (after rounding) is below
 *    chimera_index_info.q_norm_limit; for unit centroids and the workloads'
 *    residual weights that is about 2.4 (unit query tokens in the intended
 *    use).  Each query token then contributes less than 2^24 units of 2^-22
 *    to a score, so the integer sum over up to 64 tokens cannot overflow.
 *    With CHIMERA_CHECK_QUERIES=1 in the environment when the index is
 *    loaded, every search and stage tap first checks this bound on the
 *    device (the call synchronises its stream) and returns CHIMERA_E_INVAL,
 *    outputs untouched, for a query token at or above the limit or with a
 *    value that is not finite.
 *  - Orders: every "top" list is ordered by (score descending, id
 *    ascending); equal scores are broken by the lowest id.
 */
#ifndef CHIMERA_H
#define CHIMERA_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CHIMERA_ABI_VERSION 1

enum {
  CHIMERA_OK = 0,
  CHIMERA_E_INVAL = 1,       /* bad argument */
  CHIMERA_E_NOMEM = 2,       /* host or device allocation failed / would not fit */
  CHIMERA_E_IO = 3,          /* file could not be opened, read or written */
  CHIMERA_E_FORMAT = 4,      /* index file malformed, truncated, wrong version or checksum */
  CHIMERA_E_DEVICE = 5,      /* HIP runtime error; the index must be freed */
  CHIMERA_E_UNSUPPORTED = 6, /* valid but outside this build's limits (dim != 128, Tq > 64, nprobe > 64 ...) */
  CHIMERA_E_BUSY = 7         /* another host thread is inside a call on this index */
};

/* Element type of a query tensor. */
enum { CHIMERA_F32 = 0, CHIMERA_BF16 = 1 };

/* Score used by the candidate refinement (Sec. 3.2, the partial score F').
 *   CHIMERA_REFINE_CENTROID: a retrieved token scores as its centroid,
 *     S[j][c]; what chimera_search and chimera_prune do.
 *   CHIMERA_REFINE_TOKEN: a retrieved token scores as document scoring
 *     scores it, S[j][c] + <Q_j, w(code_t)> (centroid score plus its decoded
 *     residual), the paper's use of the retrieved tokens' codes. */
enum { CHIMERA_REFINE_CENTROID = 0, CHIMERA_REFINE_TOKEN = 1 };

/* Limits of this build.  Besides these, the candidate walk keeps per-list
 * state for all Tq x nprobe probed lists of a query on chip: with more than
 * 32 query tokens, Tq * nprobe up to 2304 always fits (e.g. 64 x 32), and
 * larger products may return CHIMERA_E_UNSUPPORTED. */
#define CHIMERA_DIM 128
#define CHIMERA_MAX_TQ 64
#define CHIMERA_MAX_NPROBE 64
#define CHIMERA_MAX_NCAND (1 << 20)
#define CHIMERA_MAX_K 8192

typedef struct chimera_index chimera_index;
typedef struct chimera_builder chimera_builder;

typedef struct {
  int64_t ndocs;         /* documents */
  int64_t ntokens;       /* document tokens */
  int64_t nnz;           /* entries of all posting lists */
  int32_t ncent;         /* IVF centroids */
  int32_t dim;           /* vector dimension (128) */
  int32_t nbits;         /* residual code bits per dimension (2 or 4) */
  int32_t max_doc_len;   /* longest document, tokens */
  int64_t device_bytes;  /* device memory held by the index data */
  int32_t device;        /* HIP device ordinal */
  double q_norm_limit;   /* query tokens of smaller L2 norm get exact scores
                            (see "Value grid"); 0 for a builder */
  int64_t ndeleted;      /* documents deleted (chimera_index_delete); 0 for a builder */
} chimera_index_info;

/* Last error message of the calling thread; never NULL. */
const char *chimera_last_error(void);

/* ===================================================================== *
 * Offline index building (Sec. 3.1): IVF posting lists over the
 * centroids and per-token compressed codes, stored document-major so that
 * each document's tokens are contiguous (the doc-reordered copy of the
 * codes in Sec. 4.1).  Host only, no GPU needed.
 *
 * Compression: each token t with centroid c = cid[t] stores the residual
 * r = v_t - c per dimension as a b-bit bucket code (b = nbits, 2 or 4).
 * The 2^b buckets are cut at the pooled empirical quantiles i/2^b
 * (i = 1 .. 2^b-1) of all residual components of the corpus; bucket u is
 * represented by the grid value of the (2u+1)/2^(b+1) quantile.  A residual
 * equal to a cutoff falls in the lower bucket.  (The paper compresses with
 * RaBitQ codes; this residual-bucket reading is the library's code family.)
 *
 * Two passes over the same token stream, in document order:
 *   1. chimera_builder_add_residuals for every token (any chunking);
 *   2. chimera_builder_freeze_quantizer;
 *   3. chimera_builder_add_docs for every document, in document order.
 * The IVF assignment cid[] is an input: the caller gives, for each token,
 * its centroid (normally its nearest centroid by inner product, Sec. 2.3).
 * ===================================================================== */

/* centroids_bf16: host [ncent][dim] bf16 bit patterns (copied).  dim must be
 * 128; nbits 2 or 4; ncent >= 1.  *out receives the builder. */
int chimera_builder_create(const uint16_t *centroids_bf16, int32_t ncent, int32_t dim, int32_t nbits,
                           chimera_builder **out);
/* Pass 1: tokens_bf16 host [ntok][dim], cids host [ntok] in [0, ncent).
 * Token and centroid components must lie in [-1, 1] (unit vectors satisfy
 * it), else E_INVAL. */
int chimera_builder_add_residuals(chimera_builder *b, const uint16_t *tokens_bf16, const int32_t *cids,
                                  int64_t ntok);
/* Ends pass 1: fixes cutoffs and bucket weights.  E_INVAL if no residual. */
int chimera_builder_freeze_quantizer(chimera_builder *b);
/* Pass 2: ndocs documents; doc_lens host [ndocs] (>= 1 each), tokens and cids
 * hold sum(doc_lens) rows in document order.  A call that fails (E_INVAL,
 * E_NOMEM) leaves the builder as it was before the call, so later calls
 * continue from the last accepted document; the same holds for
 * chimera_builder_add_residuals. */
int chimera_builder_add_docs(chimera_builder *b, const uint16_t *tokens_bf16, const int32_t *cids,
                             const int32_t *doc_lens, int64_t ndocs);
/* Optional, before pass 2: reserves host memory for ndocs documents and ntok
 * tokens, so that add_docs never reallocates (a 2-bit index of 600M tokens
 * holds about 20 GB of codes).  E_NOMEM if the memory cannot be reserved. */
int chimera_builder_reserve(chimera_builder *b, int64_t ndocs, int64_t ntok);
/* Optional, before pass 2: also encode every document token with RaBitQ
 * (Sec. 2.2, the extended-bits quantiser, with B = 4 as Sec. 3.1 uses),
 * for chimera_search_rabitq.  The random orthonormal rotation is
 * P = H diag(signs) / sqrt(dim), H the Sylvester Hadamard matrix of order dim
 * (H[i][j] = (-1)^popcount(i & j)), signs host [dim] int8, each +1 or -1
 * (drawn at random by the caller).  A token o (grid values) gets the code
 * y in {-7.5, -6.5, .., 7.5}^dim of largest cosine with P o (ties to the
 * smallest |y|; a zero coordinate takes +1/2), and the factors
 *     g = |o|^2 / <P o, y>   (rounded once to float32)
 * of its 4-bit code and of its most significant bits (y1 = msb - 1/2).  The
 * most significant bits (16 bytes a token) and their factor go to the GPU
 * with the index (Sec. 3.1: 1-bit codes on the GPU); the 4-bit codes stay
 * in host memory.  E_INVAL if documents were already added or a sign is not
 * +-1.  Index files do not hold these codes: chimera_builder_save then
 * returns E_UNSUPPORTED. */
int chimera_builder_rabitq(chimera_builder *b, const int8_t *signs);
/* Quantiser as fixed by freeze: cut_k [2^b - 1] cutoffs in units of 2^-11,
 * weights_bf16 [2^b] bucket values.  Either pointer may be NULL. */
int chimera_builder_quantizer(const chimera_builder *b, int32_t *cut_k, uint16_t *weights_bf16);
/* Writes the index file (format "CHIMIDX1", little-endian, 256-byte aligned
 * sections, each with a 64-bit FNV-1a checksum). */
int chimera_builder_save(const chimera_builder *b, const char *path);
/* Copies the built index to HIP device `hip_device`; *out receives a handle
 * equivalent to chimera_index_load of the saved file. */
int chimera_builder_upload(const chimera_builder *b, int hip_device, chimera_index **out);
/* Host copies of built sections (for inspection and tests).  Sizes:
 * doc_off [ndocs+1] i64, cid [ntok] i32, codes [ntok][dim*nbits/8] u8,
 * ivf_off [ncent+1] i64, ivf_doc [nnz] i32.  Any pointer may be NULL. */
int chimera_builder_sections(const chimera_builder *b, int64_t *doc_off, int32_t *cid, uint8_t *codes,
                             int64_t *ivf_off, int32_t *ivf_doc);
/* Host copies of the RaBitQ sections (chimera_builder_rabitq), per token:
 * bits1 [ntok][dim / 8] the most significant bits (bit d in byte d / 8, bit
 * d % 8), g1 [ntok] their factor, codes4 [ntok][dim / 2] the 4-bit codes
 * (dimension 2i in the low nibble of byte i, 2i + 1 in the high nibble), g4
 * [ntok] their factor.  Any pointer may be NULL; E_INVAL if the builder has
 * no RaBitQ codes. */
int chimera_builder_rabitq_sections(const chimera_builder *b, uint8_t *bits1, float *g1, uint8_t *codes4,
                                    float *g4);
int chimera_builder_info(const chimera_builder *b, chimera_index_info *out);
void chimera_builder_free(chimera_builder *b); /* NULL-safe */

/* ===================================================================== *
 * Device-resident index (Sec. 3: every GPU-side structure is preloaded,
 * only queries move at run time).
 * ===================================================================== */

/* Reads and verifies an index file and copies it to HIP device `hip_device`.
 * E_IO (open/read), E_FORMAT (magic, version, sizes, checksums), E_NOMEM. */
int chimera_index_load(const char *path, int hip_device, chimera_index **out);
void chimera_index_free(chimera_index *idx); /* NULL-safe; waits for pending work */
int chimera_index_info_get(const chimera_index *idx, chimera_index_info *out);

/* Deletion (Sec. 3.3, handling updates: a deletion bitmap over document ids
 * that retrieval skips, with periodic compaction).
 *
 * chimera_index_delete sets the bits of doc_ids [n] (host memory; repeats
 * and ids deleted before are allowed) in the index's bitmap.  From then on
 * every search treats those documents as outside S_Q: they get no F', are
 * never candidates, and never appear in any result; every other document's
 * F', scores and order are unchanged.  E_INVAL (nothing changes) if an id is
 * outside [0, ndocs) or n < 0.  It waits for all work on the index's device
 * to finish before it updates the device copy of the bitmap, so it must not
 * overlap a search of this index on another thread.
 *
 * chimera_index_compact rebuilds the device index without the deleted
 * documents' tokens and posting-list entries, so retrieval no longer walks
 * them.  Document ids do not change: a deleted document keeps its id and has
 * no tokens.  Every search returns the same as before the call.  A store
 * attached with chimera_fullbit_attach is compacted with it.  The old and the
 * new device arrays are held at once while it runs; on failure (E_NOMEM,
 * E_DEVICE) the index is left as it was. */
int chimera_index_delete(chimera_index *idx, const int64_t *doc_ids, int64_t n);
int chimera_index_compact(chimera_index *idx);

/* ===================================================================== *
 * Search (Alg. 1 without the CPU full-bit stage).
 *
 *   Q       device [nq][Tq][d], q_dtype CHIMERA_F32 or CHIMERA_BF16, row-major
 *   nq      >= 0 queries (0: no-op)
 *   Tq      1 .. 64 tokens per query
 *   d       must equal the index dimension (128)
 *   nprobe  1 .. min(ncent, 64): centroids probed per query token
 *   ncand   >= k: documents kept by the refinement (k_refine of Alg. 1);
 *           values above ndocs are clamped to ndocs
 *   k       1 .. min(ncand, CHIMERA_MAX_K) results per query
 *   ids     device [nq][k] int32, scores device [nq][k] float32
 *
 * Steps, per query:
 *  1. S[j][c] = <Q_j, c> for every centroid c, and C_j = the nprobe best
 *     centroids of query token j (Sec. 2.3 IVF probe; Sec. 3.2 candidate
 *     generation).
 *  2. S_Q = documents with a token in some probed posting list (Sec. 3.2,
 *     the candidate set S).
 *  3. F'(V) = sum_j max{S[j][c] : c in C_j, V has a token in list c}, a term
 *     being 0 when no probed list of Q_j holds V (Sec. 3.2, the partial score
 *     F'; the centroid score stands in for the per-token distance); keep the
 *     ncand best of S_Q (Alg. 2).
 *  4. For each kept V: F^(V) = sum_j max_{t in V} <Q_j, c_cid(t) + w(code_t)>,
 *     the complete score over all of V's tokens from their decoded residual
 *     codes (Sec. 3.2 document scoring; Sec. 4.2 aggregation).
 *  5. ids/scores = the k best by F^, padded with (-1, -INFINITY) when fewer
 *     than k documents were kept.
 * Scores are exact multiples of 2^-22, rounded once to float32.
 * ===================================================================== */
int chimera_search(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                   int32_t nprobe, int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream);

/* chimera_search with a choice of refinement score (Sec. 3.2 candidate
 * refinement; Alg. 2).  refine CHIMERA_REFINE_CENTROID is chimera_search.
 * refine CHIMERA_REFINE_TOKEN replaces step 3's F' by
 *   F'(V) = sum_j max{ S[j][cid t] + <Q_j, w(code_t)> : t in V, cid t in C_j },
 * a term being 0 when V has no such token: every token of a probed list is
 * scored from its code (the index's token-level posting lists), so the work
 * grows with the probed lists' token counts.  Other refine values return
 * CHIMERA_E_INVAL; a Tq x nprobe whose per-list state exceeds the
 * refinement's local memory (64 x 64) returns CHIMERA_E_UNSUPPORTED. */
int chimera_search_refine(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t k, int32_t refine, int32_t *ids, float *scores,
                          void *hip_stream);

/* chimera_search with step 4 scored from the RaBitQ 1-bit codes (index built
 * with chimera_builder_rabitq, else E_UNSUPPORTED): Sec. 3.2 document
 * scoring on the GPU, the complete 1-bit score over every token of each
 * kept document,
 *   F^(V) = sum_j key(max_{t in V} est_1(Q_j, t)),
 *   est_1(q, t) = g1_t * <P' q, 2 y1_t> * 2^-12,   key(x) = rint(x * 2^22),
 * with P' = H diag(signs) and y1_t = msb_t - 1/2 (Eq. 5 with Eq. 2's norms,
 * through Eq. 6; <P' q, 2 y1> is the binary inner product of Sec. 4.1 less
 * the sum of P' q, computed exactly); key rounds ties to even.  Scores are
 * F^ * 2^-22 in float32.  Exact (equal to the reference formula) for query
 * tokens of L2 norm below 2.8; F^ saturates at +-(2^31 - 1).  Steps 1-3 and
 * 5 are chimera_search's; the probe writes no centroid-score table. */
int chimera_search_rabitq(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream);

/* chimera_search for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * the same arguments, results and validation as chimera_search, but its
 * scratch is a fixed device array of CHIMERA_NOALLOC_SCRATCH_MB MiB built
 * into the library (one per GPU, reserved while the library's code is loaded
 * on that GPU, until the process ends), so the call allocates no device or
 * host memory.  The batch runs in as many sub-batches as that array needs.
 * CHIMERA_E_UNSUPPORTED if a single query needs more scratch than the array
 * holds (a query needs about 4 (ncent + 1) * 32 bytes of centroid scores
 * plus 4 ndocs bytes of partial scores: about 70 MB at 262,144 centroids
 * and 8.8M documents).  Every call on one GPU shares its array: calls that
 * overlap on a GPU, from any index or stream, race and must be serialised
 * by the caller.  The array keeps the last call's contents; each call
 * clears what must start at zero (its histograms) itself.
 * Stage timing (chimera_stage_times) does not record these calls. */
#define CHIMERA_NOALLOC_SCRATCH_MB 256
int chimera_search_noalloc(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                           int32_t nprobe, int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream);

/* ===================================================================== *
 * CPU-GPU collaborative scoring (Sec. 4, document scoring; Alg. 3).
 *
 * The index keeps compressed codes in HBM; the full-precision token
 * vectors stay in host memory and only the host scores them, so no
 * document data crosses PCIe at query time.
 *
 * chimera_fullbit_attach: tokens is a HOST array [ntok][dim] of bf16 bit
 * patterns, in the index's token order (document-major, the order the
 * builder was given).  The library reads every value onto the value grid,
 * as the builder does, into a host copy that the index owns (2 bytes per
 * value, the size of the input), so the caller may free its array after
 * the call; tokens == NULL drops the copy.  With the builder's own input
 * the full-precision scores are the exact Chamfer scores of the indexed
 * tokens.  Every value must lie in [-1, 1], as for the builder: with query
 * tokens of L2 norm <= 2 that keeps each full-precision dot product exact in
 * 32-bit integers.  E_INVAL if ntok differs from the index's token count or a
 * value breaks that bound (the message names the first such token; the
 * previous copy, if any, is kept), E_NOMEM if the copy cannot be allocated,
 * E_BUSY during another call on the index.
 *
 * chimera_fullbit_attach_range: the same store, attached in consecutive
 * token ranges, so that the caller never holds the whole array (at 600M
 * tokens it is 150 GB): tokens is a HOST array [n][dim] holding tokens
 * t0 .. t0+n-1 of the index's token order.  t0 = 0 drops any previous
 * store and allocates the new one (ntok tokens); each later call must start
 * where the previous one ended.  The store is complete, and collaborative
 * searches accept it, once its ranges reach ntok; until then they fail with
 * E_INVAL.  E_INVAL for a range outside [0, ntok), a range that does not
 * start where the store ends, or a value outside [-1, 1] (the message names
 * the first such token; the range is not counted and may be sent again),
 * E_NOMEM if the store cannot be allocated, E_BUSY during another call on
 * the index.  Compaction keeps a complete store and drops an incomplete one.
 *
 * chimera_search_collab: steps 1-3 of chimera_search, then Alg. 3 over each
 * query's kept candidates S_refine, taken in ascending document id:
 *  - chunk i (0 <= i < chunks) is candidates floor(i*ncand/chunks) ..
 *    floor((i+1)*ncand/chunks) - 1 (those below n_valid); the GPU computes
 *    F^ (step 4) chunk by chunk and copies each chunk's scores to pinned
 *    host memory as it finishes;
 *  - after chunk i arrives, host threads rank every candidate seen so far
 *    by (F^ desc, id asc) and compute the full-precision score
 *       F(V) = sum_j max_{t in V} <Q_j, v_t>
 *    of each of the first ceil((i+1) * kfb / chunks) that has none yet,
 *    while the GPU scores the later chunks;
 *  - ids/scores = the k best of the documents with a full-precision score,
 *    by (F desc, id asc), padded with (-1, -INFINITY).
 *   kfb      k <= kfb: the full-precision budget (k_full-bit)
 *   chunks   1 .. 64 (c of Alg. 3; 1 is the non-concurrent strategy)
 *   ids, scores, n_full   HOST arrays [nq][k], [nq][k], [nq]; n_full[q] is
 *            the number of full-precision scores computed for query q
 *            (k-hat_full-bit): at least min(kfb, n_valid), at most the sum
 *            of the chunk quotas, kfb (chunks + 1) / 2 when chunks divides
 *            kfb (Sec. 4)
 *   nthreads host threads for the full-precision scores (0: all cores)
 * Returns when the results are written (the stream is synchronised).
 * E_INVAL without an attached store (when nq > 0), for k > kfb, chunks
 * out of range, or a query component that is not finite or lies outside
 * [-2, 2] (implied by the L2 norm <= 2 that exact scores assume; the host's
 * 32-bit sums rely on it; found after the GPU has run, the stream is
 * synchronised first and the outputs are undefined);
 * other arguments as chimera_search.  Environment, read at each call:
 * CHIMERA_COLLAB_ISA caps the host instruction set (plain, avx2, vnni; the
 * results are the same), CHIMERA_COLLAB_TRACE=1 prints the host's waiting
 * and working time per sub-batch to stderr.
 * ===================================================================== */
int chimera_fullbit_attach(chimera_index *idx, const uint16_t *tokens, int64_t ntok);
int chimera_fullbit_attach_range(chimera_index *idx, const uint16_t *tokens, int64_t t0, int64_t n);
int chimera_search_collab(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t kfb, int32_t chunks, int32_t k, int32_t *ids,
                          float *scores, int32_t *n_full, int32_t nthreads, void *hip_stream);

/* chimera_search_collab with the paper's code split (Sec. 3.1): the GPU
 * scores each chunk from the RaBitQ 1-bit codes (the F^ of
 * chimera_search_rabitq) and the host's score of a document is its score
 * from the 4-bit RaBitQ codes held in host memory,
 *   F(V) = sum_j key(max_{t in V} g4_t * <P' Q_j, 2 y_t> * 2^-12),
 * (y_t the token's 4-bit codeword, key as in chimera_search_rabitq),
 * instead of the full-precision score; no store needs attaching.
 * E_UNSUPPORTED without RaBitQ codes (chimera_builder_rabitq). */
int chimera_search_collab_rabitq(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                                 int32_t nprobe, int32_t ncand, int32_t kfb, int32_t chunks, int32_t k, int32_t *ids,
                                 float *scores, int32_t *n_full, int32_t nthreads, void *hip_stream);

/* Stage taps: the same inputs as chimera_search, stopping after a stage.
 * They exist so that each stage can be compared with an independent
 * reference; they cost as much as the stages they run. */

/* After step 1: cent_ids device [nq][Tq][nprobe] int32, ordered; cent_keys
 * device [nq][Tq][nprobe] int32, S in units of 2^-22. */
int chimera_probe(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                  int32_t nprobe, int32_t *cent_ids, int32_t *cent_keys, void *hip_stream);

/* After step 2: offsets device [nq+1] int64 (CSR), doc_ids device
 * [capacity] int32, each query's S_Q ascending.  Synchronises the stream.
 * E_INVAL if sum |S_Q| > capacity; offsets are still written then. */
int chimera_candidates(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                       int32_t nprobe, int64_t *offsets, int32_t *doc_ids, int64_t capacity, void *hip_stream);

/* After step 3: cand_ids device [nq][ncand] int32 holding the kept documents
 * in ascending id order, cand_keys device [nq][ncand] int32 their F' in units
 * of 2^-22, n_valid device [nq] int32 the number kept (min(ncand, |S_Q|));
 * entries past n_valid are -1 / 0.  ncand is clamped to ndocs. */
int chimera_prune(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                  int32_t nprobe, int32_t ncand, int32_t *cand_ids, int32_t *cand_keys, int32_t *n_valid,
                  void *hip_stream);

/* chimera_prune with the refinement score chosen as in chimera_search_refine. */
int chimera_prune_refine(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                         int32_t nprobe, int32_t ncand, int32_t refine, int32_t *cand_ids, int32_t *cand_keys,
                         int32_t *n_valid, void *hip_stream);

/* Per-stage device time of the searches run on this index since the last
 * call, in ms, measured with HIP events recorded on the search stream when
 * the environment variable CHIMERA_STAGE_TIMING=1 was set at load time.
 * ms7 receives [0] query rounding, [1] probe (GEMM + top-nprobe), [2]
 * candidate walk, [3] refinement select, [4] residual scoring, [5] final
 * top-k, each summed over searches and sub-batches, and [6] the number of
 * sub-batches (one launch of each kernel per sub-batch).  Synchronises on
 * the last recorded event, then clears the record.  E_INVAL if timing is
 * off or nothing was recorded. */
int chimera_stage_times(chimera_index *idx, float *ms7);

#ifdef __cplusplus
}
#endif
#endif
