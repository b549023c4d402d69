// internal.h - shared declarations of the gfx950 query-path library.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/chimera.h"

namespace chimera {

// ---- errors -------------------------------------------------------------
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int hip_fail(hipError_t e, const char *what);
#define CHIMERA_HIP(call)                                   \
  do {                                                      \
    hipError_t e_ = (call);                                 \
    if (e_ != hipSuccess) return ::chimera::hip_fail(e_, #call); \
  } while (0)

// ---- value grid (host side) ----------------------------------------------
// Nearest multiple of max(2^-11, bf16 spacing), ties to even, of a bf16 or
// float value; returned as the integer k = x * 2^11.
int32_t grid_k_of_float(float x);
uint16_t bf16_of_grid_k(int32_t k);
float float_of_bf16(uint16_t b);

// ---- host index (what the builder produces and the file stores) ---------
struct HostIndex {
  int32_t ncent = 0, dim = 0, nbits = 0, max_doc_len = 0;
  int64_t ndocs = 0, ntok = 0, nnz = 0;
  std::vector<uint16_t> cent;     // bf16 [ncent][dim]
  std::vector<int64_t> doc_off;   // [ndocs+1]
  std::vector<int32_t> cid;       // [ntok]
  std::vector<uint8_t> codes;     // [ntok][dim*nbits/8]
  std::vector<int32_t> cut_k;     // [2^nbits - 1]
  std::vector<uint16_t> weights;  // bf16 [2^nbits]
  std::vector<int64_t> ivf_off;   // [ncent+1]
  std::vector<int32_t> ivf_doc;   // [nnz]
  // RaBitQ codes (optional, see rabitq_encode_rows): the signs of the
  // rotation [dim], per token the packed most significant bits [dim / 8]
  // and their factor, the packed 4-bit codes [dim / 2] and their factor
  bool rq = false;
  std::vector<int8_t> rq_signs;
  std::vector<uint8_t> rq_bits, rq_codes;
  std::vector<float> rq_g1, rq_g4;
  int64_t code_bytes() const { return (int64_t)dim * nbits / 8; }
};

// RaBitQ codes with B = 4 of n tokens (grid integers k [n][dim]) under the
// rotation H diag(signs): bits1 [n][dim / 8] the most significant bits (bit d
// of a token in byte d / 8, bit d % 8) and g1 [n] their factor; codes4
// [n][dim / 2] the 4-bit codes (dim 2i in the low nibble of byte i, 2i + 1 in
// the high nibble) and g4 [n] their factor.  rabitq.cpp states the reading.
void rabitq_encode_rows(const int16_t *k, int64_t n, int dim, const int8_t *signs, uint8_t *bits1, float *g1,
                        uint8_t *codes4, float *g4);

int save_index(const HostIndex &h, const char *path);
// Dense posting lists: up to kMaxDense centroids whose doc-level list holds
// more than ndocs / 16 documents (the longest first, ties to the lower id).
// slot[c] is the centroid's bit (or -1) and doc_mask[v] has bit slot[c] set
// iff document v has a token assigned to c.  Returns E_FORMAT if a mask
// disagrees with the list lengths.
constexpr int kMaxDense = 64;
int dense_lists(const HostIndex &h, std::vector<int8_t> &slot, std::vector<uint64_t> &doc_mask, int &ndense);
// Token-level posting lists (refinement from decoded token scores): tok_off
// [ncent+1], ivf_tok [ntok] the tokens of each centroid in ascending order,
// tok_doc [ntok] each token's document.
void token_lists(const HostIndex &h, std::vector<int64_t> &tok_off, std::vector<int32_t> &ivf_tok,
                 std::vector<int32_t> &tok_doc);
const HostIndex *builder_host(const chimera_builder *b);  // builds the lists on first use
int load_index(const char *path, HostIndex &h);

// Posting lists ivf_off, ivf_doc and nnz from doc_off and cid (each list
// ascending, one entry per document).
void ivf_lists(HostIndex &h);

// Zeroed tokens appended to the device copies of cid and codes.
constexpr int kTokenPad = 64;

// ---- kernel launchers (one translation unit per pipeline step) -----------
// Rounds Q [nq][Tq][128] (f32 or bf16) onto the grid as bf16, padding each
// query to TQP rows with zeros: Qs [nq][TQP][128].
void launch_round_queries(const void *Q, int q_dtype, int64_t nq, int Tq, int TQP, uint16_t *Qs,
                          hipStream_t s);

// Squared-norm check of the nq*Tq query tokens (rounded onto the grid, grid
// units): *first_bad = min token index with norm^2 >= lim2 (or non-finite);
// *first_bad must be set to ~0 before.
void launch_check_queries(const void *Q, int q_dtype, int64_t ntokens, double lim2, unsigned long long *first_bad,
                          hipStream_t s);

// Probe: S = Qs * cent^T on MFMA, top-nprobe per row.  rows = nq*TQP.
// part: [nsplit][rows][pmax] u64 partial lists.  ST (optional): [nq][ncent][TQP] f32.
struct ProbePlan {
  int pmax = 0, nsplit = 0, tiles_per_split = 0;
  int sample = 0, s_nsplit = 0, s_tiles_per_split = 0;  // centroid sample for the row bounds (0: none)
};
ProbePlan plan_probe(int64_t rows, int ncent, int nprobe);
size_t probe_part_bytes(const ProbePlan &p, int64_t rows);
void launch_probe(const uint16_t *Qs, int64_t rows, int TQP, const uint16_t *cent, int ncent,
                  const ProbePlan &p, int nprobe, uint64_t *part, float *ST, hipStream_t s);
// Merge partial lists into cent_ids/cent_keys [nq][TQP][nprobe] (rows j < Tq).
void launch_probe_merge(const uint64_t *part, int64_t nq, int Tq, int TQP, const ProbePlan &p, int nprobe,
                        int32_t *cent_ids, int32_t *cent_keys, hipStream_t s);

// Candidate walk: fp [nq][ndocs] i32 receives F' of every document, or
// INT32_MIN for documents outside S_Q and for documents whose bit is set in
// deleted [ceil(ndocs / 64)] (optional; every entry is written); hist
// [nq][4096] u32, zero on entry, receives the histogram of the top 12 bits of
// F' ^ 0x80000000 over S_Q.
void launch_fill_zero(void *p, size_t bytes, hipStream_t s);
// LDS the candidate walk needs for Tq query tokens and nprobe ranks; a
// workgroup can use at most kWalkMaxLds.
size_t walk_lds_bytes(int TQP, int nprobe, int Tq);
constexpr size_t kWalkMaxLds = 160 * 1024;
// The walk for an index without dense lists (k_walk_lists.hip; the same
// outputs); launch_cand_walk picks it when ndense == 0.
size_t list_walk_lds_bytes(int TQP, int nprobe, int Tq);
void launch_list_walk(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                      const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent,
                      const uint64_t *deleted, int32_t *fp, uint32_t *hist, hipStream_t s);
void launch_cand_walk(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                      const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent, int ndense,
                      const int8_t *dense_slot, const uint64_t *doc_dense, const uint64_t *deleted, int32_t *fp,
                      uint32_t *hist, hipStream_t s);

// Refinement select: per query, the ncand best of S_Q by (F' desc, V asc),
// written in ascending V order; n_valid [nq].  scratch holds
// select_scratch_bytes(nq, ndocs) bytes (no initial contents needed).
int select_chunks(int64_t nq, int64_t ndocs);
size_t select_scratch_bytes(int64_t nq, int64_t ndocs, int ncand);
void launch_select(const int32_t *fp, const uint32_t *hist, int64_t nq, int64_t ndocs, int ncand, void *scratch,
                   int32_t *cand_ids, int32_t *cand_keys, int32_t *n_valid, hipStream_t s);
// Candidate-set tap: counts [nq] of S_Q; then each S_Q in ascending order.
void launch_count_hits(const int32_t *fp, int64_t nq, int64_t ndocs, int64_t *counts, hipStream_t s);
void launch_list_hits(const int32_t *fp, int64_t nq, int64_t ndocs, const int64_t *offsets, int32_t *doc_ids,
                      hipStream_t s);

// Refinement from the retrieved tokens' decoded scores: the same outputs as
// launch_cand_walk (fp, hist added to), from token-level lists, the rounded
// queries Qs [nq][TQP][128] and the probe's ids and keys.  The workgroup's
// LDS is refine_lds_bytes (at most kWalkMaxLds).
size_t refine_lds_bytes(int TQP, int nprobe, int Tq);
void launch_refine_walk(const int32_t *cent_ids, const int32_t *cent_keys, const uint16_t *Qs, int64_t nq, int Tq,
                        int TQP, int nprobe, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                        const int64_t *doc_off, const uint8_t *codes, int nbits, const uint16_t *weights_host,
                        int64_t ndocs, const uint64_t *deleted, int32_t *fp, uint32_t *hist, hipStream_t s);

// Residual scoring of candidates lo .. hi-1 of each query (those below
// n_valid): fhat [nq][ncand] i32 keys; ST is [nq][ncent + 1][TQP] (row ncent
// all -inf).
void launch_residual_score(const uint16_t *Qs, int64_t nq, int Tq, int TQP, const float *ST, int ncent,
                           const int64_t *doc_off, const int32_t *cid, const uint8_t *codes, int nbits,
                           const uint16_t *weights_host, const int32_t *cand_ids, const int32_t *n_valid,
                           int ncand, int lo, int hi, int32_t *fhat, hipStream_t s);

// RaBitQ document scoring (k_rabitq.hip).  Query preparation: for each of
// the rows rounded query rows Qs [rows][128], X = 2048 H diag(signs) q as
// three int8 limbs Qi8 [rows][RQ_ROW_BYTES] (a, b, c with X = a 2^14 + b 2^7
// + c, 128 bytes each) and qsum [rows] = sum(x).  Scoring: fhat [nq][ncand]
// i32 keys of candidates lo .. hi-1 of each query (those below n_valid) from
// the 1-bit codes bits [ntok][16] and factors g1 [ntok] (both padded by
// kTokenPad tokens).
constexpr int RQ_ROW_BYTES = 384;
void launch_rq_prep(const uint16_t *Qs, int64_t rows, const int8_t *signs, uint8_t *Qi8, float *qsum, hipStream_t s);
void launch_rq_score(const uint8_t *Qi8, const float *qsum, int64_t nq, int TQP,
                     const int64_t *doc_off, const uint8_t *bits, const float *g1, const int32_t *cand_ids,
                     const int32_t *n_valid, int ncand, int lo, int hi, int32_t *fhat, hipStream_t s);

// Collaborative scoring of one sub-batch (collab.cpp): ids, scores, n_full
// are host arrays for the whole batch, written at query q0 onwards.
struct CollabOut {
  int kfb = 0, chunks = 1, k = 1, nthreads = 0;
  bool rabitq = false;  // GPU scores from the RaBitQ bits, host scores from the 4-bit codes
  int32_t *ids = nullptr;
  float *scores = nullptr;
  int32_t *n_full = nullptr;
};
// The rotated queries of a sub-batch for RaBitQ scoring (launch_rq_prep).
struct RqQuery {
  uint8_t *Qi8 = nullptr;  // [rows][RQ_ROW_BYTES]
  float *qsum = nullptr;
};
int collab_subbatch(chimera_index *idx, hipStream_t s, const uint16_t *Qs, int64_t nb, int64_t q0, int Tq, int TQP,
                    const float *ST, const RqQuery *rq, const int32_t *cand, const int32_t *nval, int ncand,
                    int32_t *fhat, const CollabOut &o);
void collab_free(chimera_index *idx);

// The fixed scratch of chimera_search_noalloc (noalloc.hip): its device
// address on `device`, which must be current; looked up on the first call
// per device and kept.
constexpr size_t kFixedScratchBytes = (size_t)CHIMERA_NOALLOC_SCRATCH_MB << 20;
// kept unused at the array's end, as the grown arena keeps 1/8 spare
constexpr size_t kFixedScratchGuard = (size_t)1 << 20;
int fixed_scratch(int device, void **ptr);

// Final top-k: ids/scores [nq][k].
void launch_topk(const int32_t *fhat, const int32_t *cand_ids, const int32_t *n_valid, int64_t nq, int ncand,
                 int k, int32_t *ids, float *scores, hipStream_t s);

}  // namespace chimera

// ---- the opaque handle -----------------------------------------------------
namespace chimera {
struct Collab;
}

struct chimera_index {
  int device = 0;
  int32_t ncent = 0, dim = 0, nbits = 0, max_doc_len = 0;
  int64_t ndocs = 0, ntok = 0, nnz = 0;
  int64_t device_bytes = 0;
  uint16_t *d_cent = nullptr;
  int64_t *d_doc_off = nullptr;
  int32_t *d_cid = nullptr;
  uint8_t *d_codes = nullptr;
  int64_t *d_ivf_off = nullptr;
  int32_t *d_ivf_doc = nullptr;
  int ndense = 0;                  // dense posting lists (see dense_lists)
  int8_t *d_dense_slot = nullptr;  // [ncent]
  uint64_t *d_doc_dense = nullptr;  // [ndocs] dense-list masks (see dense_lists)
  // RaBitQ codes (chimera_builder_rabitq): on the device the most
  // significant bits [ntok][16] and their factors [ntok] (both padded by
  // kTokenPad tokens) and the rotation's signs [dim]; in host memory the
  // 4-bit codes [ntok][dim / 2] and their factors
  bool rq = false;
  uint8_t *d_rq_bits = nullptr;
  float *d_rq_g1 = nullptr;
  int8_t *d_rq_signs = nullptr;
  std::vector<int8_t> rq_signs;
  std::vector<uint8_t> rq_codes;
  std::vector<float> rq_g4;
  int64_t *d_tok_off = nullptr;     // token-level lists (see token_lists)
  int32_t *d_ivf_tok = nullptr;
  int32_t *d_tok_doc = nullptr;
  // deletion bitmap over document ids (bit v of word v / 64), host copy and
  // device copy (allocated on the first deletion)
  std::vector<uint64_t> h_deleted;
  uint64_t *d_deleted = nullptr;
  int64_t ndeleted = 0;
  uint16_t h_weights[16] = {0};
  int32_t h_cut[15] = {0};
  // exact scores need every query token's L2 norm below this (see upload)
  double q_norm_limit = 0.0;
  bool check_queries = false;              // CHIMERA_CHECK_QUERIES=1 at load
  unsigned long long *d_check = nullptr;  // the check's result word
  // scratch arena, grown on demand, ordered across streams by scratch_done
  void *scratch = nullptr;
  size_t scratch_bytes = 0;
  hipEvent_t scratch_done = nullptr;
  bool scratch_pending = false;
  std::atomic<int> busy{0};
  // CPU-GPU collaborative scoring (collab.cpp)
  std::vector<int64_t> h_doc_off;      // host copy of doc_off [ndocs + 1]
  std::vector<int16_t> fullbit;        // full-precision tokens [ntok][dim], grid integers
  int64_t fullbit_filled = 0;          // tokens of fullbit written; complete at ntok
  chimera::Collab *collab = nullptr;   // pinned staging, events, host threads
  // per-stage timing
  bool timing = false;
  std::vector<hipEvent_t> ev;  // 7 events per sub-batch
  int ev_used = 0;
};
