// collab.cpp - the host half of the CPU-GPU collaborative document scoring
// (Sec. 4, document scoring; Alg. 3).
//
// The GPU scores each query's kept candidates chunk by chunk from their
// compressed codes (k_residual_score over a candidate range) and copies each
// chunk's keys into pinned host memory behind an event.  Host threads wait
// for chunk i, rank every candidate seen so far by its GPU key, and compute
// full-precision scores for the ones that entered the current top
// ceil((i+1) kfb / c) and have none yet, while the GPU works on chunk i+1.
// The final answer is the top-k of the full-precision scores.
//
// Full-precision scores are exact: query and document values are grid
// integers (multiples of 2^-11, as the builder and the query rounding make
// them), so a product is an integer in units of 2^-22, a 128-term dot
// product fits int32, and the sum over query tokens is int64.  The document
// tokens are read onto the grid once, when the store is attached, into an
// int16 copy the index owns; the queries are read per search.
#include <hip/hip_runtime.h>
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "internal.h"

namespace chimera {

// ------------------------------------------------------------ thread pool
// Fixed workers; run(n, fn) calls fn(i) for every i in [0, n) on the
// workers and the calling thread, and returns when all calls are done.
class Pool {
 public:
  explicit Pool(int nthreads) : nworkers_(std::max(0, nthreads - 1)) {
    for (int w = 0; w < nworkers_; ++w) th_.emplace_back([this] { work(); });
  }
  ~Pool() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto &t : th_) t.join();
  }
  int threads() const { return nworkers_ + 1; }
  // false if some fn(i) threw (the others still ran)
  bool run(int64_t n, const std::function<void(int64_t)> &fn) {
    if (n <= 0) return true;
    {
      std::lock_guard<std::mutex> lk(mu_);
      fn_ = &fn;
      n_ = n;
      next_.store(0);
      pending_ = nworkers_;
      ++gen_;
    }
    cv_.notify_all();
    drain(fn, n);
    std::unique_lock<std::mutex> lk(mu_);
    done_.wait(lk, [this] { return pending_ == 0; });
    fn_ = nullptr;
    return !failed_.exchange(false);
  }

 private:
  void drain(const std::function<void(int64_t)> &fn, int64_t n) {
    for (int64_t i = next_.fetch_add(1); i < n; i = next_.fetch_add(1)) {
      try {
        fn(i);
      } catch (...) {
        failed_.store(true);
      }
    }
  }
  void work() {
    uint64_t seen = 0;
    for (;;) {
      const std::function<void(int64_t)> *fn;
      int64_t n;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        fn = fn_;
        n = n_;
      }
      drain(*fn, n);
      {
        std::lock_guard<std::mutex> lk(mu_);
        if (--pending_ == 0) done_.notify_one();
      }
    }
  }
  const int nworkers_;
  std::vector<std::thread> th_;
  std::mutex mu_;
  std::condition_variable cv_, done_;
  const std::function<void(int64_t)> *fn_ = nullptr;
  int64_t n_ = 0;
  std::atomic<int64_t> next_{0};
  std::atomic<bool> failed_{false};
  int pending_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

// ------------------------------------------------- per-index host state
struct Collab {
  Pool *pool = nullptr;
  // pinned staging, sized for the largest sub-batch seen
  int32_t *h_cand = nullptr, *h_fhat = nullptr, *h_nval = nullptr;
  uint16_t *h_qs = nullptr;
  size_t cap_cand = 0, cap_fhat = 0, cap_q = 0, cap_qs = 0;
  hipEvent_t ev_sel = nullptr;
  std::vector<hipEvent_t> ev;  // one per chunk
  // per-query working state of one sub-batch
  std::vector<std::vector<uint64_t>> ranked;              // GPU order keys of the candidates seen so far
  std::vector<std::vector<uint8_t>> done;                 // candidate has a full-precision score
  std::vector<std::vector<std::pair<int64_t, int32_t>>> full;  // (F, doc id)
  std::vector<int16_t> qk;                                // [nb][dim/2][TqP][2] query grid integers
  std::vector<int32_t> xq;                                // [nb][Tq][dim] rotated queries (RaBitQ re-rank)
};

static void free_pinned(void *&p) {
  if (p) (void)hipHostFree(p);
  p = nullptr;
}

void collab_free(chimera_index *idx) {
  Collab *c = idx->collab;
  if (!c) return;
  delete c->pool;
  free_pinned((void *&)c->h_cand);
  free_pinned((void *&)c->h_fhat);
  free_pinned((void *&)c->h_nval);
  free_pinned((void *&)c->h_qs);
  if (c->ev_sel) (void)hipEventDestroy(c->ev_sel);
  for (hipEvent_t e : c->ev) (void)hipEventDestroy(e);
  delete c;
  idx->collab = nullptr;
}

template <class T>
static int grow_pinned(T *&p, size_t &cap, size_t n) {
  if (n <= cap) return CHIMERA_OK;
  free_pinned((void *&)p);
  cap = 0;
  void *q = nullptr;
  if (hipHostMalloc(&q, n * sizeof(T), hipHostMallocDefault) != hipSuccess)
    return fail(CHIMERA_E_NOMEM, "pinned host buffer of %zu bytes", n * sizeof(T));
  p = (T *)q;
  cap = n;
  return CHIMERA_OK;
}

// ------------------------------------------------ full-precision scores
// F(V) = sum_j max_t <Q_j, v_t> in units of 2^-22 (Def. 1 on the
// full-precision tokens).  A bf16 value v reads as the grid integer
// nearbyint(2048 v), which is what the builder makes of it (an integer
// already when |v| >= 2^-4).  Query values are at most 2 in magnitude (L2
// norm <= 2) and attached document values at most 1 (grid_in_range), so
// every partial dot product fits int32; the sum over query tokens is int64.
//
// The query is kept pair-interleaved and token-minor, qp[p][j][2] = (Q_j[2p],
// Q_j[2p+1]) with j padded to a multiple of 16, so that one multiply-add
// instruction takes 8 (AVX2) or 16 (AVX-512) query tokens times two
// dimensions of one document token, broadcast, and no horizontal sums are
// needed: each lane accumulates one query token's dot product.
constexpr int kQBlock = 16;
static_assert(CHIMERA_DIM == 128, "the full-precision kernels take 64 dimension pairs per token");

static inline __attribute__((always_inline)) void to_grid(const uint16_t *src, int64_t n, int16_t *dst) {
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t u = (uint32_t)src[i] << 16;
    float v;
    std::memcpy(&v, &u, 4);
    const float k = std::nearbyint(v * 2048.0f);
    dst[i] = (int16_t)(int32_t)std::fmin(std::fmax(k, -32768.0f), 32767.0f);
  }
}

// Attached document values lie in [-1, 1], as the builder requires of the
// tokens it indexes (grid integers within +-2^11).  With a query token of L2
// norm <= 2, every partial sum of a dot product is then at most
// 2 * sqrt(128) < 23 in magnitude, far below 2^31 in units of 2^-22.  NaN and
// infinities convert to -2^15 or 2^15 - 1 and fail the test too.
static bool grid_within(const int16_t *g, int64_t n, int lim) {
  int bad = 0;
  for (int64_t i = 0; i < n; ++i) bad |= (g[i] > lim) | (g[i] < -lim);
  return !bad;
}
static bool grid_in_range(const int16_t *g, int64_t n) { return grid_within(g, n, 2048); }
// Queries are held to components in [-2, 2] (implied by L2 norm <= 2): with
// document values in [-1, 1] a dot product is then below 128 * 2^12 * 2^11 =
// 2^30 in magnitude whatever the norm, so no input overflows the host's
// 32-bit sums.
static bool query_in_range(const int16_t *g, int64_t n) { return grid_within(g, n, 4096); }

// a = min(a, v), from several threads
static void atomic_min(std::atomic<int64_t> &a, int64_t v) {
  int64_t cur = a.load();
  while (v < cur && !a.compare_exchange_weak(cur, v)) {
  }
}

// best[j] = max over the L tokens of v of <qp_j, v_t>, for j < TqP
typedef void (*MaxDotFn)(const int16_t *qp, int TqP, const int16_t *v, int64_t L, int32_t *best);

__attribute__((target("avx512f,avx512bw,avx512vnni"))) static void maxdot_vnni(const int16_t *qp, int TqP,
                                                                               const int16_t *v, int64_t L,
                                                                               int32_t *best) {
  const int32_t *v2 = (const int32_t *)v;  // dimension pairs
  for (int jb = 0; jb < TqP; jb += 16) {
    __m512i bm = _mm512_set1_epi32(INT32_MIN);
    int64_t t = 0;
    for (; t + 4 <= L; t += 4) {
      __m512i a0 = _mm512_setzero_si512(), a1 = a0, a2 = a0, a3 = a0;
      const int32_t *w = v2 + t * 64;
      for (int p = 0; p < 64; ++p) {
        const __m512i q = _mm512_loadu_si512((const void *)(qp + ((size_t)p * TqP + jb) * 2));
        a0 = _mm512_dpwssd_epi32(a0, q, _mm512_set1_epi32(w[p]));
        a1 = _mm512_dpwssd_epi32(a1, q, _mm512_set1_epi32(w[64 + p]));
        a2 = _mm512_dpwssd_epi32(a2, q, _mm512_set1_epi32(w[128 + p]));
        a3 = _mm512_dpwssd_epi32(a3, q, _mm512_set1_epi32(w[192 + p]));
      }
      bm = _mm512_max_epi32(bm, _mm512_max_epi32(_mm512_max_epi32(a0, a1), _mm512_max_epi32(a2, a3)));
    }
    for (; t < L; ++t) {
      __m512i a0 = _mm512_setzero_si512();
      for (int p = 0; p < 64; ++p)
        a0 = _mm512_dpwssd_epi32(a0, _mm512_loadu_si512((const void *)(qp + ((size_t)p * TqP + jb) * 2)),
                                 _mm512_set1_epi32(v2[t * 64 + p]));
      bm = _mm512_max_epi32(bm, a0);
    }
    _mm512_storeu_si512((void *)(best + jb), bm);
  }
}

__attribute__((target("avx2"))) static void maxdot_avx2(const int16_t *qp, int TqP, const int16_t *v, int64_t L,
                                                        int32_t *best) {
  const int32_t *v2 = (const int32_t *)v;
  for (int jb = 0; jb < TqP; jb += 8) {
    __m256i bm = _mm256_set1_epi32(INT32_MIN);
    int64_t t = 0;
    for (; t + 4 <= L; t += 4) {
      __m256i a0 = _mm256_setzero_si256(), a1 = a0, a2 = a0, a3 = a0;
      const int32_t *w = v2 + t * 64;
      for (int p = 0; p < 64; ++p) {
        const __m256i q = _mm256_loadu_si256((const __m256i *)(qp + ((size_t)p * TqP + jb) * 2));
        a0 = _mm256_add_epi32(a0, _mm256_madd_epi16(q, _mm256_set1_epi32(w[p])));
        a1 = _mm256_add_epi32(a1, _mm256_madd_epi16(q, _mm256_set1_epi32(w[64 + p])));
        a2 = _mm256_add_epi32(a2, _mm256_madd_epi16(q, _mm256_set1_epi32(w[128 + p])));
        a3 = _mm256_add_epi32(a3, _mm256_madd_epi16(q, _mm256_set1_epi32(w[192 + p])));
      }
      bm = _mm256_max_epi32(bm, _mm256_max_epi32(_mm256_max_epi32(a0, a1), _mm256_max_epi32(a2, a3)));
    }
    for (; t < L; ++t) {
      __m256i a0 = _mm256_setzero_si256();
      for (int p = 0; p < 64; ++p) {
        const __m256i q = _mm256_loadu_si256((const __m256i *)(qp + ((size_t)p * TqP + jb) * 2));
        a0 = _mm256_add_epi32(a0, _mm256_madd_epi16(q, _mm256_set1_epi32(v2[t * 64 + p])));
      }
      bm = _mm256_max_epi32(bm, a0);
    }
    _mm256_storeu_si256((__m256i *)(best + jb), bm);
  }
}

static void maxdot_plain(const int16_t *qp, int TqP, const int16_t *v, int64_t L, int32_t *best) {
  for (int j = 0; j < TqP; ++j) best[j] = INT32_MIN;
  for (int64_t t = 0; t < L; ++t)
    for (int j = 0; j < TqP; ++j) {
      int32_t s = 0;
      for (int p = 0; p < 64; ++p)
        s += (int32_t)qp[((size_t)p * TqP + j) * 2] * v[t * 128 + 2 * p] +
             (int32_t)qp[((size_t)p * TqP + j) * 2 + 1] * v[t * 128 + 2 * p + 1];
      best[j] = s > best[j] ? s : best[j];
    }
}

// to_grid compiled for AVX2 (a vector round-to-nearest-even) where the host
// has it; the baseline build rounds value by value through the C library
typedef void (*ToGridFn)(const uint16_t *src, int64_t n, int16_t *dst);
__attribute__((target("avx2"))) static void to_grid_avx2(const uint16_t *src, int64_t n, int16_t *dst) {
  const __m256 scale = _mm256_set1_ps(2048.0f);
  int64_t i = 0;
  for (; i + 16 <= n; i += 16) {
    const __m256i b = _mm256_loadu_si256((const __m256i *)(src + i));
    // bf16 -> f32: the 16 bits become the high half of each 32-bit lane
    const __m256i lo = _mm256_unpacklo_epi16(_mm256_setzero_si256(), b);
    const __m256i hi = _mm256_unpackhi_epi16(_mm256_setzero_si256(), b);
    const __m256 flo = _mm256_round_ps(_mm256_mul_ps(_mm256_castsi256_ps(lo), scale),
                                       _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
    const __m256 fhi = _mm256_round_ps(_mm256_mul_ps(_mm256_castsi256_ps(hi), scale),
                                       _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC);
    // the saturating pack clamps to int16 and undoes the unpack's lane order
    _mm256_storeu_si256((__m256i *)(dst + i), _mm256_packs_epi32(_mm256_cvtps_epi32(flo), _mm256_cvtps_epi32(fhi)));
  }
  to_grid(src + i, n - i, dst + i);
}
static void to_grid_plain(const uint16_t *src, int64_t n, int16_t *dst) { to_grid(src, n, dst); }
// The widest instruction set the host has, capped by CHIMERA_COLLAB_ISA
// (plain, avx2 or vnni; read at every search, so tests can run each path).
// ip[j] = <x_j, z> over the 128 dimensions, for the Tq rows x_j of xq (int32;
// every product and sum stays below 2^31 for RaBitQ inputs: the query's
// grid integers are at most 4096 in magnitude, so |x| <= 128 * 4096 = 2^19,
// and |z| <= 15, so |ip| < 128 * 2^19 * 15 < 2^31)
typedef void (*RqDotFn)(const int32_t *xq, int Tq, const int32_t *z, int32_t *ip);

static void rqdot_plain(const int32_t *xq, int Tq, const int32_t *z, int32_t *ip) {
  for (int j = 0; j < Tq; ++j) {
    const int32_t *x = xq + (size_t)j * CHIMERA_DIM;
    int32_t acc = 0;
    for (int d = 0; d < CHIMERA_DIM; ++d) acc += x[d] * z[d];
    ip[j] = acc;
  }
}

__attribute__((target("avx2"))) static void rqdot_avx2(const int32_t *xq, int Tq, const int32_t *z, int32_t *ip) {
  __m256i zz[CHIMERA_DIM / 8];
  for (int i = 0; i < CHIMERA_DIM / 8; ++i) zz[i] = _mm256_loadu_si256((const __m256i *)(z + 8 * i));
  for (int j = 0; j < Tq; ++j) {
    const int32_t *x = xq + (size_t)j * CHIMERA_DIM;
    __m256i acc = _mm256_setzero_si256();
    for (int i = 0; i < CHIMERA_DIM / 8; ++i)
      acc = _mm256_add_epi32(acc, _mm256_mullo_epi32(_mm256_loadu_si256((const __m256i *)(x + 8 * i)), zz[i]));
    __m128i h = _mm_add_epi32(_mm256_castsi256_si128(acc), _mm256_extracti128_si256(acc, 1));
    h = _mm_add_epi32(h, _mm_shuffle_epi32(h, 0x4E));
    h = _mm_add_epi32(h, _mm_shuffle_epi32(h, 0xB1));
    ip[j] = _mm_cvtsi128_si32(h);
  }
}

__attribute__((target("avx512f"))) static void rqdot_avx512(const int32_t *xq, int Tq, const int32_t *z, int32_t *ip) {
  __m512i zz[CHIMERA_DIM / 16];
  for (int i = 0; i < CHIMERA_DIM / 16; ++i) zz[i] = _mm512_loadu_si512((const void *)(z + 16 * i));
  for (int j = 0; j < Tq; ++j) {
    const int32_t *x = xq + (size_t)j * CHIMERA_DIM;
    __m512i acc = _mm512_setzero_si512();
    for (int i = 0; i < CHIMERA_DIM / 16; ++i)
      acc = _mm512_add_epi32(acc, _mm512_mullo_epi32(_mm512_loadu_si512((const void *)(x + 16 * i)), zz[i]));
    ip[j] = _mm512_reduce_add_epi32(acc);
  }
}

struct HostKernels {
  ToGridFn to_grid;
  MaxDotFn maxdot;
  RqDotFn rqdot;
};
static HostKernels pick_kernels() {
  __builtin_cpu_init();
  const bool avx2 = __builtin_cpu_supports("avx2");
  const bool vnni = avx2 && __builtin_cpu_supports("avx512vnni") && __builtin_cpu_supports("avx512bw");
  const char *cap = std::getenv("CHIMERA_COLLAB_ISA");
  const int level = !cap ? 2 : !std::strcmp(cap, "plain") ? 0 : !std::strcmp(cap, "avx2") ? 1 : 2;
  if (vnni && level >= 2) return {to_grid_avx2, maxdot_vnni, rqdot_avx512};
  if (avx2 && level >= 1) return {to_grid_avx2, maxdot_avx2, rqdot_avx2};
  return {to_grid_plain, maxdot_plain, rqdot_plain};
}

// F(V) for the document of tokens [t0, t1) of the grid-integer store; an
// empty document scores INT64_MIN.
static int64_t full_score(const HostKernels &K, const int16_t *qp, int Tq, int TqP, const int16_t *tok, int64_t t0,
                          int64_t t1) {
  if (t1 <= t0) return INT64_MIN;
  int32_t best[CHIMERA_MAX_TQ + kQBlock];
  K.maxdot(qp, TqP, tok + t0 * 128, t1 - t0, best);
  int64_t F = 0;
  for (int j = 0; j < Tq; ++j) F += best[j];
  return F;
}

// The host score of a document from its RaBitQ 4-bit codes (codes [L][64],
// factors g4 [L]) for the rotated query tokens xq [Tq][128] (grid units):
// sum_j key(max_t g4_t * float(<xq_j, 2y_t> * 2^-12)), 2y = 2 code - 15, key
// = rint(x * 2^22); <xq_j, 2y_t> is exact in 32 bits for |Q_j| < 2^9.
static int64_t rq_full_score(const HostKernels &K, const int32_t *xq, int Tq, const uint8_t *codes, const float *g4,
                             int64_t L) {
  if (L <= 0) return INT64_MIN;
  float best[CHIMERA_MAX_TQ];
  for (int j = 0; j < Tq; ++j) best[j] = -INFINITY;
  alignas(64) int32_t z[CHIMERA_DIM];
  int32_t ips[CHIMERA_MAX_TQ];
  for (int64_t t = 0; t < L; ++t) {
    for (int i = 0; i < CHIMERA_DIM / 2; ++i) {
      const int c = codes[t * (CHIMERA_DIM / 2) + i];
      z[2 * i] = 2 * (c & 15) - 15;
      z[2 * i + 1] = 2 * (c >> 4) - 15;
    }
    K.rqdot(xq, Tq, z, ips);
    for (int j = 0; j < Tq; ++j) {
      const int32_t ip = ips[j];
      const float e = g4[t] * (float)std::ldexp((double)ip, -12);
      if (e > best[j]) best[j] = e;
    }
  }
  int64_t F = 0;
  for (int j = 0; j < Tq; ++j) F += (int64_t)std::nearbyint((double)best[j] * 4194304.0);
  return F;
}

// x <- H diag(signs) x for one query token (grid units; H the Sylvester
// Hadamard matrix, by the fast transform)
static void rq_rotate(const int16_t *row, const int8_t *signs, int32_t *x) {
  for (int d = 0; d < CHIMERA_DIM; ++d) x[d] = signs[d] * row[d];
  for (int h = 1; h < CHIMERA_DIM; h <<= 1)
    for (int i = 0; i < CHIMERA_DIM; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        const int32_t a = x[j], b = x[j + h];
        x[j] = a + b;
        x[j + h] = a - b;
      }
}

// A host task failed (an allocation): drain the stream, whose copies still
// target the pinned buffers, then report.
static int host_failed(hipStream_t s) {
  (void)hipStreamSynchronize(s);
  return fail(CHIMERA_E_NOMEM, "collaborative scoring: host allocation failed");
}

int collab_subbatch(chimera_index *idx, hipStream_t s, const uint16_t *Qs, int64_t nb, int64_t q0, int Tq, int TQP,
                    const float *ST, const RqQuery *rq, const int32_t *cand, const int32_t *nval, int ncand,
                    int32_t *fhat, const CollabOut &o) {
  if (!idx->collab) idx->collab = new Collab();
  Collab &C = *idx->collab;
  const int nthreads = o.nthreads > 0 ? o.nthreads : (int)std::max(1u, std::thread::hardware_concurrency());
  if (!C.pool || C.pool->threads() != nthreads) {
    delete C.pool;
    C.pool = new Pool(nthreads);
  }
  const int dim = idx->dim, c = o.chunks;
  const HostKernels K = pick_kernels();
  if (int rc = grow_pinned(C.h_cand, C.cap_cand, (size_t)nb * ncand)) return rc;
  if (int rc = grow_pinned(C.h_fhat, C.cap_fhat, (size_t)nb * ncand)) return rc;
  if (int rc = grow_pinned(C.h_nval, C.cap_q, (size_t)nb)) return rc;
  if (int rc = grow_pinned(C.h_qs, C.cap_qs, (size_t)nb * TQP * dim)) return rc;
  if (!C.ev_sel) CHIMERA_HIP(hipEventCreateWithFlags(&C.ev_sel, hipEventDisableTiming));
  while ((int)C.ev.size() < c) {
    hipEvent_t e;
    CHIMERA_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    C.ev.push_back(e);
  }

  // device side: the kept candidates and the rounded queries, then the
  // scores chunk by chunk, each chunk's copy behind its own event
  CHIMERA_HIP(hipMemcpyAsync(C.h_cand, cand, (size_t)nb * ncand * 4, hipMemcpyDeviceToHost, s));
  CHIMERA_HIP(hipMemcpyAsync(C.h_nval, nval, (size_t)nb * 4, hipMemcpyDeviceToHost, s));
  CHIMERA_HIP(hipMemcpyAsync(C.h_qs, Qs, (size_t)nb * TQP * dim * 2, hipMemcpyDeviceToHost, s));
  CHIMERA_HIP(hipEventRecord(C.ev_sel, s));
  for (int i = 0; i < c; ++i) {
    const int lo = (int)((int64_t)i * ncand / c), hi = (int)((int64_t)(i + 1) * ncand / c);
    if (hi > lo) {
      if (o.rabitq)
        launch_rq_score(rq->Qi8, rq->qsum, nb, TQP, idx->d_doc_off, idx->d_rq_bits, idx->d_rq_g1, cand, nval,
                        ncand, lo, hi, fhat, s);
      else
        launch_residual_score(Qs, nb, Tq, TQP, ST, idx->ncent, idx->d_doc_off, idx->d_cid, idx->d_codes,
                              idx->nbits, idx->h_weights, cand, nval, ncand, lo, hi, fhat, s);
      CHIMERA_HIP(hipGetLastError());
      CHIMERA_HIP(hipMemcpy2DAsync(C.h_fhat + lo, (size_t)ncand * 4, fhat + lo, (size_t)ncand * 4,
                                   (size_t)(hi - lo) * 4, nb, hipMemcpyDeviceToHost, s));
    }
    CHIMERA_HIP(hipEventRecord(C.ev[i], s));
  }

  // host side; CHIMERA_COLLAB_TRACE=1 prints where the host time goes
  static const bool trace = std::getenv("CHIMERA_COLLAB_TRACE") != nullptr;
  using clk = std::chrono::steady_clock;
  auto tp = clk::now();
  double t_wait = 0, t_work = 0;
  auto lap = [&](double &acc) {
    const auto now = clk::now();
    acc += std::chrono::duration<double, std::milli>(now - tp).count();
    tp = now;
  };
  CHIMERA_HIP(hipEventSynchronize(C.ev_sel));
  lap(t_wait);
  C.ranked.resize(nb);
  C.done.resize(nb);
  C.full.resize(nb);
  const int TqP = (Tq + kQBlock - 1) / kQBlock * kQBlock;
  C.qk.assign((size_t)nb * TqP * dim, 0);
  if (o.rabitq) C.xq.assign((size_t)nb * Tq * dim, 0);
  std::atomic<int64_t> bad_query{INT64_MAX};
  if (!C.pool->run(nb, [&](int64_t q) {
    C.ranked[q].clear();
    C.done[q].assign(ncand, 0);
    C.full[q].clear();
    int16_t *qp = C.qk.data() + (size_t)q * TqP * dim;  // [dim/2][TqP][2]
    int16_t row[CHIMERA_DIM];
    for (int j = 0; j < Tq; ++j) {
      K.to_grid(C.h_qs + ((size_t)q * TQP + j) * dim, dim, row);
      for (int d = 0; d < dim; ++d) qp[((size_t)(d >> 1) * TqP + j) * 2 + (d & 1)] = row[d];
      if (!query_in_range(row, dim)) atomic_min(bad_query, q0 + q);
      if (o.rabitq) rq_rotate(row, idx->rq_signs.data(), C.xq.data() + ((size_t)q * Tq + j) * dim);
    }
  }))
    return host_failed(s);
  if (bad_query.load() != INT64_MAX) {
    (void)hipStreamSynchronize(s);  // the chunk copies still target the pinned buffers
    return fail(CHIMERA_E_INVAL, "query %lld has a component that is not finite or outside [-2, 2]",
                (long long)bad_query.load());
  }
  const int16_t *tok = idx->fullbit.data();
  const int64_t *doc_off = idx->h_doc_off.data();
  lap(t_work);
  for (int i = 0; i < c; ++i) {
    CHIMERA_HIP(hipEventSynchronize(C.ev[i]));
    lap(t_wait);
    const int lo = (int)((int64_t)i * ncand / c), hi = (int)((int64_t)(i + 1) * ncand / c);
    const int64_t budget = ((int64_t)(i + 1) * o.kfb + c - 1) / c;  // ceil((i+1) kfb / c)
    if (!C.pool->run(nb, [&](int64_t q) {
      const int nv = std::min(C.h_nval[q], hi);
      std::vector<uint64_t> &R = C.ranked[q];
      const int32_t *cq = C.h_cand + q * ncand;
      const int32_t *fq = C.h_fhat + q * ncand;
      // order key: F^ desc, then candidate position asc (= document id asc)
      for (int u = lo; u < nv; ++u)
        R.push_back(((uint64_t)((uint32_t)fq[u] ^ 0x80000000u) << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)u));
      const int64_t m = std::min<int64_t>(budget, (int64_t)R.size());
      if (m <= 0) return;
      std::nth_element(R.begin(), R.begin() + (m - 1), R.end(), std::greater<uint64_t>());
      for (int64_t r = 0; r < m; ++r) {
        const uint32_t u = 0xFFFFFFFFu - (uint32_t)R[r];
        if (C.done[q][u]) continue;
        C.done[q][u] = 1;
        const int32_t V = cq[u];
        const int64_t F =
            o.rabitq ? rq_full_score(K, C.xq.data() + (size_t)q * Tq * dim, Tq, idx->rq_codes.data() + doc_off[V] * 64,
                                     idx->rq_g4.data() + doc_off[V], doc_off[V + 1] - doc_off[V])
                     : full_score(K, C.qk.data() + (size_t)q * TqP * dim, Tq, TqP, tok, doc_off[V], doc_off[V + 1]);
        C.full[q].emplace_back(F, V);
      }
    }))
      return host_failed(s);
    lap(t_work);
  }
  if (!C.pool->run(nb, [&](int64_t q) {
    auto &Fq = C.full[q];
    const int kk = std::min<int>(o.k, (int)Fq.size());
    auto better = [](const std::pair<int64_t, int32_t> &a, const std::pair<int64_t, int32_t> &b) {
      return a.first != b.first ? a.first > b.first : a.second < b.second;
    };
    std::partial_sort(Fq.begin(), Fq.begin() + kk, Fq.end(), better);
    int32_t *ids = o.ids + (q0 + q) * o.k;
    float *sc = o.scores + (q0 + q) * o.k;
    for (int r = 0; r < o.k; ++r) {
      ids[r] = r < kk ? Fq[r].second : -1;
      sc[r] = r < kk ? (float)Fq[r].first * (1.0f / 4194304.0f) : -INFINITY;
    }
    o.n_full[q0 + q] = (int32_t)Fq.size();
  }))
    return host_failed(s);
  lap(t_work);
  if (trace)
    std::fprintf(stderr, "[collab] %lld queries, %d chunks, %d threads: waiting on the GPU %.3f ms, "
                 "host work %.3f ms\n", (long long)nb, c, C.pool->threads(), t_wait, t_work);
  return CHIMERA_OK;
}

}  // namespace chimera

using namespace chimera;

// Reads tokens [0, n) of src onto the grid into dst, in parallel slices of
// whole tokens; returns the first token with a value that is not finite or
// lies outside [-1, 1], or n when there is none.
static int64_t fullbit_convert(const uint16_t *src, int64_t n, int16_t *dst) {
  const HostKernels K = pick_kernels();
  const unsigned nt = (unsigned)std::max<int64_t>(
      1, std::min<int64_t>({32, (int64_t)std::thread::hardware_concurrency(), (n + 63) / 64}));
  std::atomic<int64_t> first_bad{n};
  auto slice = [&](unsigned w) {
    const int64_t b = n * w / nt, e = n * (w + 1) / nt;
    constexpr int64_t kBlock = 64;  // tokens converted, then checked while cached
    for (int64_t t = b; t < e; t += kBlock) {
      const int64_t m = std::min(kBlock, e - t);
      int16_t *g = dst + t * CHIMERA_DIM;
      K.to_grid(src + t * CHIMERA_DIM, m * CHIMERA_DIM, g);
      if (grid_in_range(g, m * CHIMERA_DIM)) continue;
      for (int64_t u = 0; u < m; ++u)
        if (!grid_in_range(g + u * CHIMERA_DIM, CHIMERA_DIM)) {
          atomic_min(first_bad, t + u);
          break;
        }
      return;
    }
  };
  std::vector<std::thread> th;
  th.reserve(nt);
  {
    // every started thread is joined, whatever happens after it starts
    struct JoinAll {
      std::vector<std::thread> &v;
      ~JoinAll() {
        for (auto &t : v)
          if (t.joinable()) t.join();
      }
    } join_all{th};
    for (unsigned w = 0; w < nt; ++w) {
      try {
        th.emplace_back(slice, w);
      } catch (...) {
        slice(w);  // no thread available: this slice runs on the calling thread
      }
    }
  }
  return first_bad.load();
}

extern "C" int chimera_fullbit_attach(chimera_index *idx, const uint16_t *tokens, int64_t ntok) {
  if (!idx) return fail(CHIMERA_E_INVAL, "null index");
  if (tokens && ntok != idx->ntok)
    return fail(CHIMERA_E_INVAL, "full-precision store has %lld tokens, the index %lld", (long long)ntok,
                (long long)idx->ntok);
  // the same exclusion as every other call on the index
  if (idx->busy.exchange(1) != 0) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  if (!tokens) {
    std::vector<int16_t>().swap(idx->fullbit);
    idx->fullbit_filled = 0;
    idx->busy.store(0);
    return CHIMERA_OK;
  }
  int rc = CHIMERA_OK;
  try {
    std::vector<int16_t> store((size_t)ntok * CHIMERA_DIM);
    const int64_t bad = fullbit_convert(tokens, ntok, store.data());
    if (bad < ntok) {
      rc = fail(CHIMERA_E_INVAL, "full-precision token %lld has a value that is not finite or outside [-1, 1]",
                (long long)bad);
    } else {
      idx->fullbit.swap(store);
      idx->fullbit_filled = ntok;
    }
  } catch (const std::bad_alloc &) {
    rc = fail(CHIMERA_E_NOMEM, "full-precision store of %lld tokens", (long long)ntok);
  } catch (...) {
    rc = fail(CHIMERA_E_NOMEM, "full-precision store: host allocation failed");
  }
  idx->busy.store(0);
  return rc;
}

extern "C" int chimera_fullbit_attach_range(chimera_index *idx, const uint16_t *tokens, int64_t t0, int64_t n) {
  if (!idx) return fail(CHIMERA_E_INVAL, "null index");
  if (t0 < 0 || n < 0 || t0 > idx->ntok || n > idx->ntok - t0)
    return fail(CHIMERA_E_INVAL, "token range [%lld, %lld + %lld) outside the index's %lld tokens", (long long)t0,
                (long long)t0, (long long)n, (long long)idx->ntok);
  if (n > 0 && !tokens) return fail(CHIMERA_E_INVAL, "null tokens");
  if (idx->busy.exchange(1) != 0) return fail(CHIMERA_E_BUSY, "index in use by another thread");
  int rc = CHIMERA_OK;
  try {
    if (t0 == 0) {
      // a new store: the previous one, complete or not, is dropped first, so
      // that the two never coexist in host memory
      std::vector<int16_t>().swap(idx->fullbit);
      idx->fullbit_filled = 0;
      idx->fullbit.resize((size_t)idx->ntok * CHIMERA_DIM);
    }
    if (t0 != idx->fullbit_filled || idx->fullbit.size() != (size_t)idx->ntok * CHIMERA_DIM) {
      rc = fail(CHIMERA_E_INVAL, "token range starts at %lld; the store being attached holds %lld tokens",
                (long long)t0, (long long)idx->fullbit_filled);
    } else {
      const int64_t bad = fullbit_convert(tokens, n, idx->fullbit.data() + t0 * CHIMERA_DIM);
      if (bad < n)
        rc = fail(CHIMERA_E_INVAL, "full-precision token %lld has a value that is not finite or outside [-1, 1]",
                  (long long)(t0 + bad));
      else
        idx->fullbit_filled = t0 + n;
    }
  } catch (const std::bad_alloc &) {
    std::vector<int16_t>().swap(idx->fullbit);
    idx->fullbit_filled = 0;
    rc = fail(CHIMERA_E_NOMEM, "full-precision store of %lld tokens", (long long)idx->ntok);
  } catch (...) {
    std::vector<int16_t>().swap(idx->fullbit);
    idx->fullbit_filled = 0;
    rc = fail(CHIMERA_E_NOMEM, "full-precision store: host allocation failed");
  }
  idx->busy.store(0);
  return rc;
}
