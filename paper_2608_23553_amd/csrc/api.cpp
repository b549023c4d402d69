// api.cpp - the C ABI: errors, device index, validation and the per-batch
// orchestration of the query path (Alg. 1 without the CPU full-bit stage).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>

#include "internal.h"

namespace chimera {

static thread_local char g_err[512] = "no error";

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char *what) {
  if (e == hipErrorOutOfMemory) return fail(CHIMERA_E_NOMEM, "%s: %s", what, hipGetErrorString(e));
  return fail(CHIMERA_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess) ok = true;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

// Marks the index busy for the duration of a host call.
struct BusyGuard {
  chimera_index *idx;
  bool ok;
  explicit BusyGuard(chimera_index *i) : idx(i), ok(i->busy.exchange(1) == 0) {}
  ~BusyGuard() {
    if (ok) idx->busy.store(0);
  }
};

static int upload(const HostIndex &h, int device, chimera_index **out) {
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0) return fail(CHIMERA_E_DEVICE, "no HIP device available");
  if (device < 0 || device >= ndev) return fail(CHIMERA_E_INVAL, "device %d out of range (%d devices)", device, ndev);
  DeviceGuard dg(device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", device);
  chimera_index *idx = new (std::nothrow) chimera_index;
  if (!idx) return fail(CHIMERA_E_NOMEM, "handle allocation");
  idx->device = device;
  idx->ncent = h.ncent; idx->dim = h.dim; idx->nbits = h.nbits; idx->max_doc_len = h.max_doc_len;
  idx->ndocs = h.ndocs; idx->ntok = h.ntok; idx->nnz = h.nnz;
  idx->h_doc_off = h.doc_off;
  std::memcpy(idx->h_weights, h.weights.data(), h.weights.size() * 2);
  std::memcpy(idx->h_cut, h.cut_k.data(), h.cut_k.size() * 4);
  {
    // Exactness bound (header, "Value grid"): a query token q scores
    // <q, c> + <q, w(code)>; every partial sum is at most
    // ||q|| (max_c ||c|| + sqrt(dim) max_u |w_u|) in magnitude and must stay
    // below 4.  Norms from the grid integers, rounded up slightly.
    int64_t c2max = 0;
    for (int32_t c = 0; c < h.ncent; ++c) {
      int64_t c2 = 0;
      for (int d = 0; d < h.dim; ++d) {
        const int64_t k = (int64_t)(float_of_bf16(h.cent[(size_t)c * h.dim + d]) * 2048.0f);
        c2 += k * k;
      }
      c2max = std::max(c2max, c2);
    }
    double wmax = 0.0;
    for (uint16_t w : h.weights) wmax = std::max(wmax, (double)std::fabs(float_of_bf16(w)));
    const double bound = std::sqrt((double)c2max) / 2048.0 + std::sqrt((double)h.dim) * wmax;
    idx->q_norm_limit = bound > 0.0 ? 4.0 / (bound * (1.0 + 1e-9)) : 1e30;
  }
  std::vector<int8_t> dense_slot;
  std::vector<uint64_t> doc_dense;
  if (int rc = dense_lists(h, dense_slot, doc_dense, idx->ndense)) {
    delete idx;
    return rc;
  }
  std::vector<int64_t> tok_off;
  std::vector<int32_t> ivf_tok, tok_doc;
  token_lists(h, tok_off, ivf_tok, tok_doc);
  struct Sec { void **dst; const void *src; size_t bytes; size_t pad; };
  std::vector<Sec> secs = {
      {(void **)&idx->d_cent, h.cent.data(), h.cent.size() * 2},
      {(void **)&idx->d_doc_off, h.doc_off.data(), h.doc_off.size() * 8},
      {(void **)&idx->d_cid, h.cid.data(), h.cid.size() * 4},
      {(void **)&idx->d_codes, h.codes.data(), h.codes.size()},
      {(void **)&idx->d_ivf_off, h.ivf_off.data(), h.ivf_off.size() * 8},
      {(void **)&idx->d_ivf_doc, h.ivf_doc.data(), h.ivf_doc.size() * 4},
      {(void **)&idx->d_dense_slot, dense_slot.data(), dense_slot.size()},
      {(void **)&idx->d_doc_dense, doc_dense.data(), doc_dense.size() * 8},
      {(void **)&idx->d_tok_off, tok_off.data(), tok_off.size() * 8},
      {(void **)&idx->d_ivf_tok, ivf_tok.data(), ivf_tok.size() * 4},
      {(void **)&idx->d_tok_doc, tok_doc.data(), tok_doc.size() * 4},
  };
  // Token arrays (cid, codes, RaBitQ bits and factors) are followed by
  // kTokenPad zeroed tokens: the scorers read whole 16- or 32-token tiles
  // and may run up to 31 tokens past the last document.  Every section gets
  // at least 256 spare bytes.
  const size_t pad_bytes[] = {256, 256, kTokenPad * 4 + 256, (size_t)kTokenPad * h.code_bytes() + 256, 256, 256, 256,
                              256, 256, 256, 256};
  static_assert(sizeof(pad_bytes) / sizeof(pad_bytes[0]) == 11, "one pad per section");
  for (size_t i = 0; i < secs.size(); ++i) secs[i].pad = pad_bytes[i];
  if (h.rq) {
    idx->rq = true;
    idx->rq_signs = h.rq_signs;
    idx->rq_codes = h.rq_codes;
    idx->rq_g4 = h.rq_g4;
    secs.push_back({(void **)&idx->d_rq_bits, h.rq_bits.data(), h.rq_bits.size(), (size_t)kTokenPad * 16 + 256});
    secs.push_back({(void **)&idx->d_rq_g1, h.rq_g1.data(), h.rq_g1.size() * 4, (size_t)kTokenPad * 4 + 256});
    secs.push_back({(void **)&idx->d_rq_signs, h.rq_signs.data(), h.rq_signs.size(), 256});
  }
  size_t need = 0;
  for (auto &s : secs) need += s.bytes;
  size_t free_b = 0, total_b = 0;
  if (hipMemGetInfo(&free_b, &total_b) == hipSuccess && need > free_b) {
    delete idx;
    return fail(CHIMERA_E_NOMEM, "index needs %zu bytes, %zu free on device %d", need, free_b, device);
  }
  for (auto &s : secs) {
    const size_t pad = s.pad;
    hipError_t e = hipMalloc(s.dst, s.bytes + pad);
    if (e == hipSuccess) e = hipMemset((char *)*s.dst + s.bytes, 0, pad);
    if (e == hipSuccess && s.bytes) e = hipMemcpy(*s.dst, s.src, s.bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      int rc = hip_fail(e, "index upload");
      chimera_index_free(idx);
      return rc;
    }
    idx->device_bytes += (int64_t)s.bytes;
  }
  if (hipEventCreateWithFlags(&idx->scratch_done, hipEventDisableTiming) != hipSuccess) {
    chimera_index_free(idx);
    return fail(CHIMERA_E_DEVICE, "event creation failed");
  }
  const char *t = std::getenv("CHIMERA_STAGE_TIMING");
  idx->timing = t && t[0] == '1';
  const char *cq = std::getenv("CHIMERA_CHECK_QUERIES");
  idx->check_queries = cq && cq[0] == '1';
  if (idx->check_queries && hipMalloc(&idx->d_check, sizeof(unsigned long long)) != hipSuccess) {
    idx->d_check = nullptr;
    chimera_index_free(idx);
    return fail(CHIMERA_E_NOMEM, "query check word");
  }
  *out = idx;
  return CHIMERA_OK;
}

// ----------------------------------------------------------- validation
static int check_query_args(const chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                            int32_t nprobe, int refine = CHIMERA_REFINE_CENTROID) {
  if (!idx) return fail(CHIMERA_E_INVAL, "null index");
  if (nq < 0) return fail(CHIMERA_E_INVAL, "nq must be >= 0");
  if (nq > 0 && !Q) return fail(CHIMERA_E_INVAL, "null query pointer");
  if (q_dtype != CHIMERA_F32 && q_dtype != CHIMERA_BF16) return fail(CHIMERA_E_INVAL, "q_dtype must be F32 or BF16");
  if (d != idx->dim) return fail(CHIMERA_E_INVAL, "query dim %d != index dim %d", d, idx->dim);
  if (Tq < 1) return fail(CHIMERA_E_INVAL, "Tq must be >= 1");
  if (Tq > CHIMERA_MAX_TQ) return fail(CHIMERA_E_UNSUPPORTED, "Tq %d > %d", Tq, CHIMERA_MAX_TQ);
  if (nprobe < 1 || nprobe > idx->ncent) return fail(CHIMERA_E_INVAL, "nprobe must be in [1, ncent=%d]", idx->ncent);
  if (nprobe > CHIMERA_MAX_NPROBE) return fail(CHIMERA_E_UNSUPPORTED, "nprobe %d > %d", nprobe, CHIMERA_MAX_NPROBE);
  if (walk_lds_bytes(Tq <= 32 ? 32 : 64, nprobe, Tq) > kWalkMaxLds)
    return fail(CHIMERA_E_UNSUPPORTED, "Tq %d x nprobe %d exceeds the candidate walk's local memory", Tq, nprobe);
  if (refine != CHIMERA_REFINE_CENTROID && refine != CHIMERA_REFINE_TOKEN)
    return fail(CHIMERA_E_INVAL, "refine must be CHIMERA_REFINE_CENTROID or CHIMERA_REFINE_TOKEN");
  if (refine == CHIMERA_REFINE_TOKEN && refine_lds_bytes(Tq <= 32 ? 32 : 64, nprobe, Tq) > kWalkMaxLds)
    return fail(CHIMERA_E_UNSUPPORTED, "Tq %d x nprobe %d exceeds the token refinement's local memory", Tq, nprobe);
  return CHIMERA_OK;
}

static const int kMaxK = CHIMERA_MAX_K;

// No C++ exception leaves the C ABI: host allocations inside a call that fail
// report E_NOMEM.
template <class F>
static int guarded(F &&f) {
  try {
    return f();
  } catch (const std::bad_alloc &) {
    return fail(CHIMERA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(CHIMERA_E_INVAL, "internal error");
  }
}

// ------------------------------------------------------------- pipeline
enum Stop { STOP_PROBE = 1, STOP_CANDIDATES = 2, STOP_PRUNE = 3, STOP_FULL = 4, STOP_COLLAB = 5 };

struct Outs {
  int32_t *cent_ids = nullptr, *cent_keys = nullptr;            // probe tap [nq][Tq][nprobe]
  int64_t *offsets = nullptr; int32_t *doc_ids = nullptr; int64_t capacity = 0;  // candidates tap
  int32_t *cand_ids = nullptr, *cand_keys = nullptr, *n_valid = nullptr;         // prune tap
  int32_t *ids = nullptr; float *scores = nullptr;                               // search
  const CollabOut *collab = nullptr;                                             // collaborative scoring
  bool rabitq = false;                                                           // score from RaBitQ bits
};

static size_t align_up(size_t x) { return (x + 255) / 256 * 256; }

struct Carve {
  char *base;
  size_t off = 0;
  template <class T>
  T *take(size_t n) {
    T *p = (T *)(base + off);
    off += align_up(n * sizeof(T));
    return p;
  }
};

// Exact bytes the sub-batch loop below carves for nb queries.
static size_t carve_bytes(const chimera_index *idx, int64_t nb, int TQP, int nprobe, int ncand, Stop stop,
                          bool rq) {
  const int64_t rows = nb * TQP;
  const ProbePlan plan = plan_probe(rows, idx->ncent, nprobe);
  size_t b = 0;
  b += align_up((size_t)rows * 128 * 2);                       // Qs
  b += align_up(probe_part_bytes(plan, rows));                 // partial lists
  b += 2 * align_up((size_t)rows * nprobe * 4);                // cent ids / keys
  if (stop >= STOP_FULL && !rq) b += align_up((size_t)nb * (idx->ncent + 1) * TQP * 4);  // S^T + sentinel rows
  if (rq) b += align_up((size_t)rows * RQ_ROW_BYTES) + align_up((size_t)rows * 4);  // query limbs, qsum
  if (stop >= STOP_CANDIDATES) {
    b += align_up((size_t)nb * idx->ndocs * 4);  // F'
    b += align_up((size_t)nb * 4096 * 4);        // select histogram
  }
  if (stop == STOP_CANDIDATES) b += align_up((size_t)(nb + 1) * 8);  // counts
  if (stop >= STOP_PRUNE)  // cand, keys, F^, n, select state
    b += 3 * align_up((size_t)nb * ncand * 4) + align_up((size_t)nb * 4) + align_up(select_scratch_bytes(nb, idx->ndocs, ncand));
  return b;
}

// CHIMERA_SCRATCH_DEVICE_MB (environment, for tests): an arena larger than
// this is refused as if the device were out of memory.
static size_t scratch_device_cap() {
  const char *s = std::getenv("CHIMERA_SCRATCH_DEVICE_MB");
  return s ? (size_t)std::strtoull(s, nullptr, 10) << 20 : SIZE_MAX;
}

static int ensure_scratch(chimera_index *idx, size_t bytes) {
  if (bytes <= idx->scratch_bytes) return CHIMERA_OK;
  if (bytes + bytes / 8 > scratch_device_cap())
    return fail(CHIMERA_E_NOMEM, "scratch allocation of %zu bytes: above CHIMERA_SCRATCH_DEVICE_MB",
                bytes + bytes / 8);
  if (idx->scratch) {
    CHIMERA_HIP(hipDeviceSynchronize());
    CHIMERA_HIP(hipFree(idx->scratch));
    idx->scratch = nullptr;
    idx->scratch_bytes = 0;
    idx->scratch_pending = false;
  }
  size_t want = bytes + bytes / 8;
  hipError_t e = hipMalloc(&idx->scratch, want);
  if (e != hipSuccess) {
    idx->scratch = nullptr;
    (void)hipGetLastError();  // reported here; not to be seen again by a later launch check
    return hip_fail(e, "scratch allocation");
  }
  idx->scratch_bytes = want;
  return CHIMERA_OK;
}

static size_t scratch_budget() {
  const char *s = std::getenv("CHIMERA_SCRATCH_MB");
  // larger sub-batches amortise each launch's tail: at 8.8M documents a
  // query needs about 72 MB, and a 4096-query batch takes 6,862 QPS in 9
  // sub-batches (32 GiB), 6,898 in 5 (64 GiB) and 6,990 in 3 (128 GiB);
  // the arena is sized to the batch, so small batches take little of it
  size_t mb = s ? (size_t)std::strtoull(s, nullptr, 10) : 131072;
  if (mb < 16) mb = 16;
  return mb << 20;
}

static void stage_mark(chimera_index *idx, hipStream_t s, bool on) {
  if (!idx->timing || !on) return;
  if (idx->ev_used >= (int)idx->ev.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return;
    idx->ev.push_back(e);
  }
  (void)hipEventRecord(idx->ev[idx->ev_used++], s);
}

// The on-request query check (CHIMERA_CHECK_QUERIES): E_INVAL, before
// anything else is launched, if a query token's norm breaks the limit.
static int check_queries(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int Tq, hipStream_t s) {
  const unsigned long long none = ~0ull;
  unsigned long long bad = none;
  const double lim = idx->q_norm_limit * 2048.0;
  CHIMERA_HIP(hipMemcpyAsync(idx->d_check, &none, sizeof none, hipMemcpyHostToDevice, s));
  launch_check_queries(Q, q_dtype, nq * Tq, lim * lim, idx->d_check, s);
  CHIMERA_HIP(hipGetLastError());
  CHIMERA_HIP(hipMemcpyAsync(&bad, idx->d_check, sizeof bad, hipMemcpyDeviceToHost, s));
  CHIMERA_HIP(hipStreamSynchronize(s));
  if (bad != none)
    return fail(CHIMERA_E_INVAL, "query %lld token %lld: L2 norm not below %.6g (the limit for exact scores on this "
                "index) or a value that is not finite", (long long)(bad / Tq), (long long)(bad % Tq),
                idx->q_norm_limit);
  return CHIMERA_OK;
}

// A caller-provided scratch region instead of the index's own arena (the
// search that allocates nothing): nothing is allocated, no stage events are
// recorded, and the sub-batches are sized to fit `bytes`.
struct FixedScratch {
  char *base = nullptr;
  size_t bytes = 0;
};

static int run(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int Tq, int nprobe, int ncand, int k,
               Stop stop, Outs o, hipStream_t s, int refine = CHIMERA_REFINE_CENTROID, FixedScratch fixed = {}) {
  const int TQP = Tq <= 32 ? 32 : 64;
  const bool own = fixed.base == nullptr;
  if (idx->check_queries)
    if (int rc = check_queries(idx, Q, q_dtype, nq, Tq, s)) return rc;
  // sub-batch size: the largest that fits the scratch budget (carve_bytes
  // grows with nb, but not in proportion: the select's chunking depends on nb)
  const size_t budget = own ? scratch_budget() : fixed.bytes;
  int64_t lo = 1, hi = std::min<int64_t>(nq, 65535);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (carve_bytes(idx, mid, TQP, nprobe, ncand, stop, o.rabitq) <= budget) lo = mid;
    else hi = mid - 1;
  }
  int64_t B = lo;
  // a launch counts its work-items in 32 bits; the scorer runs about 8 per
  // (query, candidate) (its grid rounds queries up to 8 and candidates up to
  // 32), so a sub-batch keeps nb * ncand at most 2^28
  B = std::min<int64_t>(B, std::max<int64_t>(1, ((int64_t)1 << 28) / std::max(1, ncand)));
  // equal sub-batches: the same number of passes, without a short last one
  const int64_t npass = (nq + B - 1) / B;
  B = (nq + npass - 1) / npass;
  auto need_for = [&](int64_t b) {
    size_t n = carve_bytes(idx, b, TQP, nprobe, ncand, stop, o.rabitq);
    if (nq % b) n = std::max(n, carve_bytes(idx, nq % b, TQP, nprobe, ncand, stop, o.rabitq));
    return n;
  };
  size_t need = need_for(B);
  if (!own) {
    while (need > fixed.bytes && B > 1) need = need_for(--B);
    if (need > fixed.bytes)
      return fail(CHIMERA_E_UNSUPPORTED, "one query of this search needs %zu bytes of scratch, more than the "
                  "fixed scratch's %zu", need, fixed.bytes);
  } else {
    int rc = ensure_scratch(idx, need);
    // the device cannot hold that much now (other allocations on it): halve
    // the sub-batches until their scratch fits, down to one query
    while (rc == CHIMERA_E_NOMEM && B > 1) {
      B = (B + 1) / 2;
      need = need_for(B);
      rc = ensure_scratch(idx, need);
    }
    if (rc) return rc;
    if (idx->scratch_pending) CHIMERA_HIP(hipStreamWaitEvent(s, idx->scratch_done, 0));
  }
  char *const scratch = own ? (char *)idx->scratch : fixed.base;
  const size_t scratch_cap = own ? idx->scratch_bytes : fixed.bytes;
  // Every exit from here on, error returns included, marks the index's
  // scratch as in use by the work queued on s, so a later call on another
  // stream waits for that work before it reuses the scratch.
  struct ScratchDone {
    chimera_index *idx;
    hipStream_t s;
    bool on;
    ~ScratchDone() {
      if (on && hipEventRecord(idx->scratch_done, s) == hipSuccess) idx->scratch_pending = true;
    }
  } scratch_done_on_exit{idx, s, own};
  const bool mark = stop == STOP_FULL && own;
  int rc = CHIMERA_OK;

  std::vector<int64_t> host_counts;
  int64_t total_hits = 0;

  for (int64_t q0 = 0; q0 < nq; q0 += B) {
    const int64_t nb = std::min<int64_t>(B, nq - q0);
    const int64_t rows = nb * TQP;
    const ProbePlan plan = plan_probe(rows, idx->ncent, nprobe);
    Carve cv{scratch};
    uint16_t *Qs = cv.take<uint16_t>((size_t)rows * 128);
    uint64_t *part = cv.take<uint64_t>(probe_part_bytes(plan, rows) / 8);
    int32_t *ci = cv.take<int32_t>((size_t)rows * nprobe);
    int32_t *ck = cv.take<int32_t>((size_t)rows * nprobe);
    float *ST = stop >= STOP_FULL && !o.rabitq ? cv.take<float>((size_t)nb * (idx->ncent + 1) * TQP) : nullptr;
    if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
    const size_t qbytes = (size_t)Tq * 128 * (q_dtype == CHIMERA_F32 ? 4 : 2);
    const void *Qb = (const char *)Q + (size_t)q0 * qbytes;

    stage_mark(idx, s, mark);
    launch_round_queries(Qb, q_dtype, nb, Tq, TQP, Qs, s);
    stage_mark(idx, s, mark);
    launch_probe(Qs, rows, TQP, idx->d_cent, idx->ncent, plan, nprobe, part, ST, s);
    launch_probe_merge(part, nb, Tq, TQP, plan, nprobe, ci, ck, s);
    CHIMERA_HIP(hipGetLastError());
    if (stop == STOP_PROBE) {
      CHIMERA_HIP(hipMemcpy2DAsync(o.cent_ids + q0 * Tq * nprobe, (size_t)Tq * nprobe * 4, ci,
                                   (size_t)TQP * nprobe * 4, (size_t)Tq * nprobe * 4, nb, hipMemcpyDeviceToDevice, s));
      CHIMERA_HIP(hipMemcpy2DAsync(o.cent_keys + q0 * Tq * nprobe, (size_t)Tq * nprobe * 4, ck,
                                   (size_t)TQP * nprobe * 4, (size_t)Tq * nprobe * 4, nb, hipMemcpyDeviceToDevice, s));
      continue;
    }
    int32_t *fp = cv.take<int32_t>((size_t)nb * idx->ndocs);
    uint32_t *hist = cv.take<uint32_t>((size_t)nb * 4096);
    if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
    stage_mark(idx, s, mark);
    launch_fill_zero(hist, (size_t)nb * 4096 * 4, s);
    if (refine == CHIMERA_REFINE_TOKEN)
      launch_refine_walk(ci, ck, Qs, nb, Tq, TQP, nprobe, idx->d_tok_off, idx->d_ivf_tok, idx->d_tok_doc,
                         idx->d_doc_off, idx->d_codes, idx->nbits, idx->h_weights, idx->ndocs,
                         idx->ndeleted ? idx->d_deleted : nullptr, fp, hist, s);
    else
      launch_cand_walk(ci, ck, nb, Tq, TQP, nprobe, idx->d_ivf_off, idx->d_ivf_doc, idx->ndocs, idx->ncent,
                       idx->ndense, idx->d_dense_slot, idx->d_doc_dense, idx->ndeleted ? idx->d_deleted : nullptr, fp,
                       hist, s);
    CHIMERA_HIP(hipGetLastError());
    if (stop == STOP_CANDIDATES) {
      int64_t *cnt = cv.take<int64_t>((size_t)nb + 1);
      if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
      launch_count_hits(fp, nb, idx->ndocs, cnt, s);
      std::vector<int64_t> hc(nb);
      CHIMERA_HIP(hipMemcpyAsync(hc.data(), cnt, nb * 8, hipMemcpyDeviceToHost, s));
      CHIMERA_HIP(hipStreamSynchronize(s));
      std::vector<int64_t> offs(nb + 1);
      offs[0] = total_hits;
      for (int64_t i = 0; i < nb; ++i) offs[i + 1] = offs[i] + hc[i];
      bool fits = offs[nb] <= o.capacity;
      if (fits && offs[nb] > total_hits) {
        CHIMERA_HIP(hipMemcpyAsync(cnt, offs.data(), (nb + 1) * 8, hipMemcpyHostToDevice, s));
        launch_list_hits(fp, nb, idx->ndocs, cnt, o.doc_ids, s);
        CHIMERA_HIP(hipStreamSynchronize(s));
      }
      for (int64_t i = 0; i < nb; ++i) host_counts.push_back(hc[i]);
      total_hits = offs[nb];
      continue;
    }
    int32_t *cand = o.cand_ids ? o.cand_ids + q0 * ncand : cv.take<int32_t>((size_t)nb * ncand);
    int32_t *candk = o.cand_keys ? o.cand_keys + q0 * ncand : cv.take<int32_t>((size_t)nb * ncand);
    int32_t *nval = o.n_valid ? o.n_valid + q0 : cv.take<int32_t>((size_t)nb);
    int32_t *fhat = stop >= STOP_FULL ? cv.take<int32_t>((size_t)nb * ncand) : nullptr;
    if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
    stage_mark(idx, s, mark);
    char *selw = cv.take<char>(select_scratch_bytes(nb, idx->ndocs, ncand));
    if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
    launch_select(fp, hist, nb, idx->ndocs, ncand, selw, cand, candk, nval, s);
    CHIMERA_HIP(hipGetLastError());
    if (stop == STOP_PRUNE) continue;
    // RaBitQ scoring: the rotated queries as int8 limbs
    RqQuery rq;
    if (o.rabitq) {
      rq.Qi8 = cv.take<uint8_t>((size_t)rows * RQ_ROW_BYTES);
      rq.qsum = cv.take<float>((size_t)rows);
      if (cv.off > scratch_cap) return fail(CHIMERA_E_NOMEM, "internal: scratch plan overflow");
      launch_rq_prep(Qs, rows, idx->d_rq_signs, rq.Qi8, rq.qsum, s);
    }
    if (stop == STOP_COLLAB) {
      rc = collab_subbatch(idx, s, Qs, nb, q0, Tq, TQP, ST, o.rabitq ? &rq : nullptr, cand, nval, ncand, fhat,
                           *o.collab);
      if (rc) return rc;
      continue;
    }
    stage_mark(idx, s, mark);
    if (o.rabitq) {
      launch_rq_score(rq.Qi8, rq.qsum, nb, TQP, idx->d_doc_off, idx->d_rq_bits, idx->d_rq_g1, cand, nval,
                      ncand, 0, ncand, fhat, s);
    } else {
      launch_residual_score(Qs, nb, Tq, TQP, ST, idx->ncent, idx->d_doc_off, idx->d_cid, idx->d_codes, idx->nbits,
                            idx->h_weights, cand, nval, ncand, 0, ncand, fhat, s);
    }
    stage_mark(idx, s, mark);
    launch_topk(fhat, cand, nval, nb, ncand, k, o.ids + q0 * k, o.scores + q0 * k, s);
    stage_mark(idx, s, mark);
    CHIMERA_HIP(hipGetLastError());
  }
  if (stop == STOP_CANDIDATES) {
    std::vector<int64_t> offs(nq + 1, 0);
    for (int64_t i = 0; i < nq; ++i) offs[i + 1] = offs[i] + host_counts[i];
    CHIMERA_HIP(hipMemcpyAsync(o.offsets, offs.data(), (nq + 1) * 8, hipMemcpyHostToDevice, s));
    CHIMERA_HIP(hipStreamSynchronize(s));
    if (offs[nq] > o.capacity)
      return fail(CHIMERA_E_INVAL, "candidate sets hold %lld ids, capacity is %lld", (long long)offs[nq],
                  (long long)o.capacity);
  }
  return CHIMERA_OK;
}

}  // namespace chimera

using namespace chimera;

extern "C" {

const char *chimera_last_error(void) { return g_err; }

int chimera_builder_upload(const chimera_builder *b, int hip_device, chimera_index **out) {
  if (!b || !out) return fail(CHIMERA_E_INVAL, "null argument");
  const HostIndex *h = builder_host(b);
  if (h->weights.empty()) return fail(CHIMERA_E_INVAL, "quantiser not frozen");
  return upload(*h, hip_device, out);
}

int chimera_index_load(const char *path, int hip_device, chimera_index **out) {
  if (!path || !out) return fail(CHIMERA_E_INVAL, "null argument");
  HostIndex h;
  int rc = load_index(path, h);
  if (rc) return rc;
  return upload(h, hip_device, out);
}

void chimera_index_free(chimera_index *idx) {
  if (!idx) return;
  DeviceGuard dg(idx->device);
  (void)hipDeviceSynchronize();
  void *ptrs[] = {idx->d_cent,    idx->d_doc_off,    idx->d_cid,       idx->d_codes,     idx->d_ivf_off,
                  idx->d_ivf_doc, idx->d_dense_slot, idx->d_doc_dense, idx->d_tok_off,   idx->d_ivf_tok,
                  idx->d_tok_doc, idx->scratch,      idx->d_check,     idx->d_deleted,   idx->d_rq_bits,
                  idx->d_rq_g1,   idx->d_rq_signs};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  collab_free(idx);
  if (idx->scratch_done) (void)hipEventDestroy(idx->scratch_done);
  for (hipEvent_t e : idx->ev) (void)hipEventDestroy(e);
  delete idx;
}

int chimera_index_info_get(const chimera_index *idx, chimera_index_info *out) {
  if (!idx || !out) return fail(CHIMERA_E_INVAL, "null argument");
  out->ndocs = idx->ndocs; out->ntokens = idx->ntok; out->nnz = idx->nnz; out->ncent = idx->ncent;
  out->dim = idx->dim; out->nbits = idx->nbits; out->max_doc_len = idx->max_doc_len;
  out->device_bytes = idx->device_bytes; out->device = idx->device;
  out->q_norm_limit = idx->q_norm_limit;
  out->ndeleted = idx->ndeleted;
  return CHIMERA_OK;
}

int chimera_index_delete(chimera_index *idx, const int64_t *doc_ids, int64_t n) {
  if (!idx || n < 0 || (n > 0 && !doc_ids)) return fail(CHIMERA_E_INVAL, "null index, null ids or n < 0");
  for (int64_t i = 0; i < n; ++i)
    if (doc_ids[i] < 0 || doc_ids[i] >= idx->ndocs)
      return fail(CHIMERA_E_INVAL, "document id %lld (entry %lld) outside [0, %lld)", (long long)doc_ids[i],
                  (long long)i, (long long)idx->ndocs);
  if (n == 0) return CHIMERA_OK;
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  return guarded([&]() -> int {
    const size_t words = (size_t)(idx->ndocs + 63) / 64;
    std::vector<uint64_t> bits = idx->h_deleted;
    bits.resize(words, 0);
    int64_t added = 0;
    for (int64_t i = 0; i < n; ++i) {
      uint64_t &w = bits[(size_t)doc_ids[i] >> 6];
      const uint64_t b = 1ull << (doc_ids[i] & 63);
      added += (w & b) ? 0 : 1;
      w |= b;
    }
    if (!idx->d_deleted) CHIMERA_HIP(hipMalloc(&idx->d_deleted, words * 8));
    // searches already queued read the bitmap as it was
    CHIMERA_HIP(hipDeviceSynchronize());
    CHIMERA_HIP(hipMemcpy(idx->d_deleted, bits.data(), words * 8, hipMemcpyHostToDevice));
    idx->h_deleted.swap(bits);
    idx->ndeleted += added;
    return CHIMERA_OK;
  });
}

int chimera_index_compact(chimera_index *idx) {
  if (!idx) return fail(CHIMERA_E_INVAL, "null index");
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  if (idx->ndeleted == 0) return CHIMERA_OK;
  return guarded([&]() -> int {
    CHIMERA_HIP(hipDeviceSynchronize());
    // the index as the host builder holds it, without the deleted
    // documents' tokens: the same centroids and quantiser, lists rebuilt
    HostIndex h;
    h.ncent = idx->ncent;
    h.dim = idx->dim;
    h.nbits = idx->nbits;
    h.ndocs = idx->ndocs;
    const int64_t cb = (int64_t)idx->dim * idx->nbits / 8;
    h.cent.resize((size_t)idx->ncent * idx->dim);
    CHIMERA_HIP(hipMemcpy(h.cent.data(), idx->d_cent, h.cent.size() * 2, hipMemcpyDeviceToHost));
    h.cut_k.assign(idx->h_cut, idx->h_cut + (1 << idx->nbits) - 1);
    h.weights.assign(idx->h_weights, idx->h_weights + (1 << idx->nbits));
    std::vector<int32_t> cid((size_t)idx->ntok);
    std::vector<uint8_t> codes((size_t)(idx->ntok * cb));
    CHIMERA_HIP(hipMemcpy(cid.data(), idx->d_cid, cid.size() * 4, hipMemcpyDeviceToHost));
    CHIMERA_HIP(hipMemcpy(codes.data(), idx->d_codes, codes.size(), hipMemcpyDeviceToHost));
    const std::vector<int64_t> &off = idx->h_doc_off;
    auto gone = [&](int64_t v) { return (idx->h_deleted[(size_t)v >> 6] >> (v & 63)) & 1; };
    h.doc_off.assign((size_t)idx->ndocs + 1, 0);
    for (int64_t v = 0; v < idx->ndocs; ++v) {
      const int64_t len = gone(v) ? 0 : off[v + 1] - off[v];
      h.doc_off[v + 1] = h.doc_off[v] + len;
      h.max_doc_len = std::max<int32_t>(h.max_doc_len, (int32_t)len);
    }
    h.ntok = h.doc_off[idx->ndocs];
    h.cid.resize((size_t)h.ntok);
    h.codes.resize((size_t)(h.ntok * cb));
    std::vector<int16_t> fullbit;
    // a complete store is compacted with the index; one still being attached
    // range by range is dropped
    if (!idx->fullbit.empty() && idx->fullbit_filled == idx->ntok) fullbit.resize((size_t)h.ntok * idx->dim);
    // RaBitQ codes: bits and factors from the device, 4-bit codes from host
    const int64_t b1 = idx->dim / 8, b4 = idx->dim / 2;
    std::vector<uint8_t> rq_bits;
    std::vector<float> rq_g1;
    if (idx->rq) {
      rq_bits.resize((size_t)(idx->ntok * b1));
      rq_g1.resize((size_t)idx->ntok);
      CHIMERA_HIP(hipMemcpy(rq_bits.data(), idx->d_rq_bits, rq_bits.size(), hipMemcpyDeviceToHost));
      CHIMERA_HIP(hipMemcpy(rq_g1.data(), idx->d_rq_g1, rq_g1.size() * 4, hipMemcpyDeviceToHost));
      h.rq = true;
      h.rq_signs = idx->rq_signs;
      h.rq_bits.resize((size_t)(h.ntok * b1));
      h.rq_g1.resize((size_t)h.ntok);
      h.rq_codes.resize((size_t)(h.ntok * b4));
      h.rq_g4.resize((size_t)h.ntok);
    }
    for (int64_t v = 0; v < idx->ndocs; ++v) {
      const int64_t len = h.doc_off[v + 1] - h.doc_off[v];
      if (!len) continue;
      const int64_t to = h.doc_off[v], from = off[v];
      std::memcpy(&h.cid[to], &cid[from], len * 4);
      std::memcpy(&h.codes[to * cb], &codes[from * cb], len * cb);
      if (!fullbit.empty()) std::memcpy(&fullbit[to * idx->dim], &idx->fullbit[from * idx->dim], len * idx->dim * 2);
      if (idx->rq) {
        std::memcpy(&h.rq_bits[to * b1], &rq_bits[from * b1], len * b1);
        std::memcpy(&h.rq_g1[to], &rq_g1[from], len * 4);
        std::memcpy(&h.rq_codes[to * b4], &idx->rq_codes[from * b4], len * b4);
        std::memcpy(&h.rq_g4[to], &idx->rq_g4[from], len * 4);
      }
    }
    std::vector<int32_t>().swap(cid);
    std::vector<uint8_t>().swap(codes);
    ivf_lists(h);
    chimera_index *fresh = nullptr;
    if (int rc = upload(h, idx->device, &fresh)) return rc;
    // the new arrays replace the old ones; the handle, its scratch, events,
    // bitmap and host state stay
    void **mine[] = {(void **)&idx->d_cent,      (void **)&idx->d_doc_off,    (void **)&idx->d_cid,
                     (void **)&idx->d_codes,     (void **)&idx->d_ivf_off,    (void **)&idx->d_ivf_doc,
                     (void **)&idx->d_dense_slot, (void **)&idx->d_doc_dense, (void **)&idx->d_tok_off,
                     (void **)&idx->d_ivf_tok,   (void **)&idx->d_tok_doc,    (void **)&idx->d_rq_bits,
                     (void **)&idx->d_rq_g1,     (void **)&idx->d_rq_signs};
    void **theirs[] = {(void **)&fresh->d_cent,      (void **)&fresh->d_doc_off,    (void **)&fresh->d_cid,
                       (void **)&fresh->d_codes,     (void **)&fresh->d_ivf_off,    (void **)&fresh->d_ivf_doc,
                       (void **)&fresh->d_dense_slot, (void **)&fresh->d_doc_dense, (void **)&fresh->d_tok_off,
                       (void **)&fresh->d_ivf_tok,   (void **)&fresh->d_tok_doc,    (void **)&fresh->d_rq_bits,
                       (void **)&fresh->d_rq_g1,     (void **)&fresh->d_rq_signs};
    for (size_t i = 0; i < sizeof(mine) / sizeof(mine[0]); ++i) {
      if (*mine[i]) (void)hipFree(*mine[i]);
      *mine[i] = *theirs[i];
      *theirs[i] = nullptr;
    }
    idx->ntok = fresh->ntok;
    idx->nnz = fresh->nnz;
    idx->max_doc_len = fresh->max_doc_len;
    idx->ndense = fresh->ndense;
    idx->device_bytes = fresh->device_bytes;
    idx->h_doc_off.swap(fresh->h_doc_off);
    idx->fullbit.swap(fullbit);
    idx->fullbit_filled = idx->fullbit.empty() ? 0 : idx->ntok;
    idx->rq_codes.swap(fresh->rq_codes);
    idx->rq_g4.swap(fresh->rq_g4);
    chimera_index_free(fresh);
    return CHIMERA_OK;
  });
}

int chimera_search(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d, int32_t nprobe,
                   int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream) {
  return chimera_search_refine(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, k, CHIMERA_REFINE_CENTROID, ids, scores,
                               hip_stream);
}

// Validation and set-up shared by the searches; `fixed` selects the fixed
// scratch (chimera_search_noalloc).
static int search_common(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                         int32_t nprobe, int32_t ncand, int32_t k, int32_t refine, int32_t *ids, float *scores,
                         void *hip_stream, bool fixed, bool rabitq = false) {
  int rc = check_query_args(idx, Q, q_dtype, nq, Tq, d, nprobe, refine);
  if (rc) return rc;
  if (k < 1) return fail(CHIMERA_E_INVAL, "k must be >= 1");
  if (ncand < k) return fail(CHIMERA_E_INVAL, "ncand (%d) must be >= k (%d)", ncand, k);
  if (k > kMaxK) return fail(CHIMERA_E_UNSUPPORTED, "k %d > %d", k, kMaxK);
  if (ncand > CHIMERA_MAX_NCAND) return fail(CHIMERA_E_UNSUPPORTED, "ncand %d > %d", ncand, CHIMERA_MAX_NCAND);
  if (nq > 0 && (!ids || !scores)) return fail(CHIMERA_E_INVAL, "null output pointer");
  if (rabitq && !idx->rq) return fail(CHIMERA_E_UNSUPPORTED, "the index holds no RaBitQ codes");
  if (nq == 0) return CHIMERA_OK;
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  FixedScratch fs;
  if (fixed) {
    void *p = nullptr;
    if ((rc = fixed_scratch(idx->device, &p))) return rc;
    fs.base = (char *)p;
    fs.bytes = kFixedScratchBytes - kFixedScratchGuard;
  }
  int nc = (int)std::min<int64_t>(ncand, idx->ndocs);
  Outs o;
  o.ids = ids;
  o.scores = scores;
  o.rabitq = rabitq;
  return guarded([&] {
    return run(idx, Q, q_dtype, nq, Tq, nprobe, nc, k, STOP_FULL, o, (hipStream_t)hip_stream, refine, fs);
  });
}

int chimera_search_refine(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t k, int32_t refine, int32_t *ids, float *scores,
                          void *hip_stream) {
  return search_common(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, k, refine, ids, scores, hip_stream, false);
}

int chimera_search_noalloc(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                           int32_t nprobe, int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream) {
  return search_common(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, k, CHIMERA_REFINE_CENTROID, ids, scores,
                       hip_stream, true);
}

int chimera_search_rabitq(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t k, int32_t *ids, float *scores, void *hip_stream) {
  return search_common(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, k, CHIMERA_REFINE_CENTROID, ids, scores,
                       hip_stream, false, true);
}

static int collab_common(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                         int32_t nprobe, int32_t ncand, int32_t kfb, int32_t chunks, int32_t k, int32_t *ids,
                         float *scores, int32_t *n_full, int32_t nthreads, void *hip_stream, bool rabitq) {
  int rc = check_query_args(idx, Q, q_dtype, nq, Tq, d, nprobe);
  if (rc) return rc;
  if (k < 1) return fail(CHIMERA_E_INVAL, "k must be >= 1");
  if (kfb < k) return fail(CHIMERA_E_INVAL, "kfb (%d) must be >= k (%d)", kfb, k);
  if (ncand < 1) return fail(CHIMERA_E_INVAL, "ncand must be >= 1");
  if (chunks < 1 || chunks > 64) return fail(CHIMERA_E_INVAL, "chunks must be in [1, 64]");
  if (nthreads < 0) return fail(CHIMERA_E_INVAL, "nthreads must be >= 0");
  if (ncand > CHIMERA_MAX_NCAND) return fail(CHIMERA_E_UNSUPPORTED, "ncand %d > %d", ncand, CHIMERA_MAX_NCAND);
  if (nq > 0 && (!ids || !scores || !n_full)) return fail(CHIMERA_E_INVAL, "null output pointer");
  if (nq == 0) return CHIMERA_OK;
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  // read under the guard: attach swaps the store while it holds it
  if (rabitq && !idx->rq) return fail(CHIMERA_E_UNSUPPORTED, "the index holds no RaBitQ codes");
  if (!rabitq && idx->fullbit.empty())
    return fail(CHIMERA_E_INVAL, "no full-precision store attached (chimera_fullbit_attach)");
  if (!rabitq && idx->fullbit_filled != idx->ntok)
    return fail(CHIMERA_E_INVAL, "full-precision store incomplete: %lld of %lld tokens attached",
                (long long)idx->fullbit_filled, (long long)idx->ntok);
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  int nc = (int)std::min<int64_t>(ncand, idx->ndocs);
  if (nc == 0) return fail(CHIMERA_E_INVAL, "index has no documents");
  CollabOut co;
  co.kfb = kfb;
  co.chunks = chunks;
  co.k = k;
  co.nthreads = nthreads;
  co.ids = ids;
  co.scores = scores;
  co.n_full = n_full;
  co.rabitq = rabitq;
  Outs o;
  o.collab = &co;
  o.rabitq = rabitq;
  hipStream_t s = (hipStream_t)hip_stream;
  rc = guarded([&] { return run(idx, Q, q_dtype, nq, Tq, nprobe, nc, 1, STOP_COLLAB, o, s); });
  if (rc) return rc;
  CHIMERA_HIP(hipStreamSynchronize(s));
  return CHIMERA_OK;
}

int chimera_search_collab(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                          int32_t nprobe, int32_t ncand, int32_t kfb, int32_t chunks, int32_t k, int32_t *ids,
                          float *scores, int32_t *n_full, int32_t nthreads, void *hip_stream) {
  return collab_common(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, kfb, chunks, k, ids, scores, n_full, nthreads,
                       hip_stream, false);
}

int chimera_search_collab_rabitq(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                                 int32_t nprobe, int32_t ncand, int32_t kfb, int32_t chunks, int32_t k, int32_t *ids,
                                 float *scores, int32_t *n_full, int32_t nthreads, void *hip_stream) {
  return collab_common(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, kfb, chunks, k, ids, scores, n_full, nthreads,
                       hip_stream, true);
}

int chimera_probe(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d, int32_t nprobe,
                  int32_t *cent_ids, int32_t *cent_keys, void *hip_stream) {
  int rc = check_query_args(idx, Q, q_dtype, nq, Tq, d, nprobe);
  if (rc) return rc;
  if (nq > 0 && (!cent_ids || !cent_keys)) return fail(CHIMERA_E_INVAL, "null output pointer");
  if (nq == 0) return CHIMERA_OK;
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  Outs o;
  o.cent_ids = cent_ids;
  o.cent_keys = cent_keys;
  return guarded([&] {
    return run(idx, Q, q_dtype, nq, Tq, nprobe, 1, 1, STOP_PROBE, o, (hipStream_t)hip_stream);
  });
}

int chimera_candidates(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                       int32_t nprobe, int64_t *offsets, int32_t *doc_ids, int64_t capacity, void *hip_stream) {
  int rc = check_query_args(idx, Q, q_dtype, nq, Tq, d, nprobe);
  if (rc) return rc;
  if (!offsets || (capacity > 0 && !doc_ids) || capacity < 0) return fail(CHIMERA_E_INVAL, "bad output arguments");
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  if (nq == 0) {
    int64_t z = 0;
    CHIMERA_HIP(hipMemcpy(offsets, &z, 8, hipMemcpyHostToDevice));
    return CHIMERA_OK;
  }
  Outs o;
  o.offsets = offsets;
  o.doc_ids = doc_ids;
  o.capacity = capacity;
  return guarded([&] {
    return run(idx, Q, q_dtype, nq, Tq, nprobe, 1, 1, STOP_CANDIDATES, o, (hipStream_t)hip_stream);
  });
}

int chimera_prune(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d, int32_t nprobe,
                  int32_t ncand, int32_t *cand_ids, int32_t *cand_keys, int32_t *n_valid, void *hip_stream) {
  return chimera_prune_refine(idx, Q, q_dtype, nq, Tq, d, nprobe, ncand, CHIMERA_REFINE_CENTROID, cand_ids, cand_keys,
                              n_valid, hip_stream);
}

int chimera_prune_refine(chimera_index *idx, const void *Q, int q_dtype, int64_t nq, int32_t Tq, int32_t d,
                         int32_t nprobe, int32_t ncand, int32_t refine, int32_t *cand_ids, int32_t *cand_keys,
                         int32_t *n_valid, void *hip_stream) {
  int rc = check_query_args(idx, Q, q_dtype, nq, Tq, d, nprobe, refine);
  if (rc) return rc;
  if (ncand < 1) return fail(CHIMERA_E_INVAL, "ncand must be >= 1");
  if (ncand > CHIMERA_MAX_NCAND) return fail(CHIMERA_E_UNSUPPORTED, "ncand %d > %d", ncand, CHIMERA_MAX_NCAND);
  if (nq > 0 && (!cand_ids || !cand_keys || !n_valid)) return fail(CHIMERA_E_INVAL, "null output pointer");
  if (nq == 0) return CHIMERA_OK;
  BusyGuard bg(idx);
  if (!bg.ok) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  DeviceGuard dg(idx->device);
  if (!dg.ok) return fail(CHIMERA_E_DEVICE, "cannot select device %d", idx->device);
  int nc = (int)std::min<int64_t>(ncand, idx->ndocs);
  if (nc == 0) return fail(CHIMERA_E_INVAL, "index has no documents");
  Outs o;
  o.cand_ids = cand_ids;
  o.cand_keys = cand_keys;
  o.n_valid = n_valid;
  return guarded([&] {
    return run(idx, Q, q_dtype, nq, Tq, nprobe, nc, 1, STOP_PRUNE, o, (hipStream_t)hip_stream, refine);
  });
}

int chimera_stage_times(chimera_index *idx, float *ms6) {
  if (!idx || !ms6) return fail(CHIMERA_E_INVAL, "null argument");
  if (!idx->timing) return fail(CHIMERA_E_INVAL, "stage timing is off (set CHIMERA_STAGE_TIMING=1 before load)");
  for (int i = 0; i < 7; ++i) ms6[i] = 0.f;
  // events per sub-batch of a search: round, probe, walk, select, score, top-k, end
  const int per = 7;
  if (idx->ev_used == 0 || idx->ev_used % per != 0) return fail(CHIMERA_E_INVAL, "no search recorded");
  CHIMERA_HIP(hipEventSynchronize(idx->ev[idx->ev_used - 1]));
  for (int b = 0; b + per <= idx->ev_used; b += per)
    for (int i = 0; i < 6; ++i) {
      float ms = 0.f;
      CHIMERA_HIP(hipEventElapsedTime(&ms, idx->ev[b + i], idx->ev[b + i + 1]));
      ms6[i] += ms;
    }
  ms6[6] = (float)(idx->ev_used / per);
  idx->ev_used = 0;
  return CHIMERA_OK;
}

}  // extern "C"
