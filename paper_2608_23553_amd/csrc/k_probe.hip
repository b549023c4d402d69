// k_probe.hip - query rounding, query-token x centroid scores on MFMA and
// top-nprobe centroid selection (Sec. 2.3: a query vector is compared with
// all centroids and the top-n_probe clusters are kept; Sec. 3.2 candidate
// generation, the lists C_q).
//
// S = Q C^T is the one dense contraction of the path: [rows,128] x [128,ncent]
// in bf16 with fp32 accumulation.  On the value grid every product and partial
// sum is an exact multiple of 2^-22 well inside fp32's 24-bit significand, so
// the MFMA result is exact whatever its internal summation order, and the
// selected ids are bit-exact.  S is never materialised for selection: each
// lane keeps a running sorted list of its best (score, id) keys.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

// ------------------------------------------------------------ rounding
__global__ __launch_bounds__(256) void k_round_queries(const void *__restrict__ Q, int q_dtype, int64_t nq, int Tq,
                                                       int TQP, uint16_t *__restrict__ Qs) {
  const int64_t total = nq * TQP * 128;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = e >> 7;
    const int d = (int)(e & 127);
    const int64_t q = row / TQP;
    const int j = (int)(row - q * TQP);
    uint16_t out = 0;
    if (j < Tq) {
      const int64_t src = (q * Tq + j) * 128 + d;
      float x = q_dtype == CHIMERA_F32 ? ((const float *)Q)[src]
                                       : __uint_as_float((uint32_t)((const uint16_t *)Q)[src] << 16);
      out = grid_bf16_bits(x);
    }
    Qs[e] = out;
  }
}

void launch_round_queries(const void *Q, int q_dtype, int64_t nq, int Tq, int TQP, uint16_t *Qs, hipStream_t s) {
  const int64_t total = nq * TQP * 128;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65535 * 8) blocks = 65535 * 8;
  if (blocks < 1) return;
  hipLaunchKernelGGL(k_round_queries, dim3((unsigned)blocks), dim3(256), 0, s, Q, q_dtype, nq, Tq, TQP, Qs);
}

// Query check (on request): the squared L2 norm, in grid units, of every
// query token as the search rounds it; *first_bad receives the lowest token
// index (q * Tq + j) whose norm is not below the index's limit for exact
// scores, or any non-finite value.  One wave per token.
__global__ __launch_bounds__(256) void k_check_queries(const void *__restrict__ Q, int q_dtype, int64_t ntokens,
                                                       double lim2, unsigned long long *__restrict__ first_bad) {
  const int lane = lane_id();
  for (int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); tok < ntokens; tok += (int64_t)gridDim.x * 4) {
    double ss = 0.0;
    for (int d = lane; d < 128; d += 64) {
      const int64_t src = tok * 128 + d;
      const float x = q_dtype == CHIMERA_F32 ? ((const float *)Q)[src]
                                             : __uint_as_float((uint32_t)((const uint16_t *)Q)[src] << 16);
      const double k = (double)__uint_as_float((uint32_t)grid_bf16_bits(x) << 16) * 2048.0;  // exact
      ss += k * k;
    }
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) ss += __shfl_xor(ss, m, 64);
    if (lane == 0 && !(ss < lim2)) atomicMin(first_bad, (unsigned long long)tok);
  }
}

void launch_check_queries(const void *Q, int q_dtype, int64_t ntokens, double lim2, unsigned long long *first_bad,
                          hipStream_t s) {
  int64_t blocks = (ntokens + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) return;
  hipLaunchKernelGGL(k_check_queries, dim3((unsigned)blocks), dim3(256), 0, s, Q, q_dtype, ntokens, lim2, first_bad);
}

// --------------------------------------------------------------- probe
// Insert K into L (sorted descending), dropping the smallest.
template <int P>
__device__ __forceinline__ void insert_desc(uint64_t (&L)[P], uint64_t K) {
#pragma unroll
  for (int i = 0; i < P; ++i) {
    const uint64_t a = L[i];
    const bool gt = K > a;
    L[i] = gt ? K : a;
    K = gt ? a : K;
  }
}

// Compare-exchange: a keeps the larger key.
__device__ __forceinline__ void cx(uint64_t &a, uint64_t &b) {
  const bool gt = b > a;
  const uint64_t t = a;
  a = gt ? b : a;
  b = gt ? t : b;
}

// Bitonic sorting network, descending, on K[0 .. N).
template <int N>
__device__ __forceinline__ void bitonic_sort_desc(uint64_t *K) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int l = i ^ j;
        if (l > i) {
          if ((i & k) == 0) cx(K[i], K[l]);
          else cx(K[l], K[i]);
        }
      }
}

// A (sorted descending) becomes the top N of A and B (both sorted
// descending): the elementwise maximum of A and reversed B is bitonic and
// holds those N keys; a bitonic merge sorts it.
template <int N>
__device__ __forceinline__ void merge_top_desc(uint64_t *A, const uint64_t *B) {
#pragma unroll
  for (int i = 0; i < N; ++i) A[i] = B[N - 1 - i] > A[i] ? B[N - 1 - i] : A[i];
#pragma unroll
  for (int j = N >> 1; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int l = i ^ j;
      if (l > i) cx(A[i], A[l]);
    }
}

// L (sorted descending, P keys) becomes the top P of L and the 16 keys K,
// without branches: K is sorted in groups of P, the groups are merged
// pairwise keeping the top P, and the winner is merged into L.
template <int P>
__device__ __forceinline__ void fold_tile(uint64_t (&L)[P], uint64_t (&K)[16]) {
  static_assert(P == 4 || P == 8 || P == 16, "lists of 4, 8 or 16 keys");
  constexpr int G = 16 / P;
#pragma unroll
  for (int g = 0; g < G; ++g) bitonic_sort_desc<P>(K + g * P);
#pragma unroll
  for (int step = 1; step < G; step <<= 1)
#pragma unroll
    for (int g = 0; g + step < G; g += 2 * step) merge_top_desc<P>(K + g * P, K + (g + step) * P);
  merge_top_desc<P>(L, K);
}

// One workgroup: 32 query rows (one column block) x a range of centroid tiles.
// Four waves stride over 32-centroid tiles; each wave computes a 32x32 tile
// of S^T (rows = centroids, cols = query rows) with 8 MFMA 32x32x16 steps.
// The contraction index k of MFMA step s, lane half h, element i is
// dimension 64h + 8s + i for both operands (any common permutation of the
// 128 dimensions gives the same exact sum), so every lane loads 128
// contiguous bytes of its centroid row and of its query row.
// Each lane keeps the sorted top PMAX keys of the centroids it sees.  Early in
// its stream nearly every key enters some lane's list, and a tile's 16 keys go
// in at once through sorting networks (lists of 4 to 16); lists of 4 or 8
// switch, once a lane has seen 128 * PMAX keys and entries have become rare,
// to inserting keys one by one where they beat the list's last, as lists of
// 32 and 64 do throughout.  With TAU, tau[row] is a lower bound on the row's
// nprobe-th best key (from a sample of the centroids): keys below it can
// never be selected and are dropped before they reach a list, so keys are
// inserted one by one, and rarely.
template <int PMAX, int TQP, bool WRITE_ST, bool TAU>
__global__ __launch_bounds__(256) void k_probe(const uint16_t *__restrict__ Qs, const uint16_t *__restrict__ cent,
                                               int ncent, int tiles_per_split, int64_t rows,
                                               uint64_t *__restrict__ part, float *__restrict__ ST,
                                               const uint64_t *__restrict__ tau) {
  __shared__ uint64_t lds[3][32][PMAX];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 31, h = lane >> 5;
  const int64_t qrow = (int64_t)blockIdx.x * 32 + col;
  const int split = blockIdx.y;

  bf16x8 bq[8];
  {
    const uint4 *qp = (const uint4 *)(Qs + qrow * 128 + 64 * h);
#pragma unroll
    for (int s = 0; s < 8; ++s) bq[s] = as_bf16x8(qp[s]);
  }
  uint64_t L[PMAX];
#pragma unroll
  for (int i = 0; i < PMAX; ++i) L[i] = 0;  // every real key is > 0
  const uint64_t tr = TAU ? tau[qrow] : 0;

  const int ntiles = (ncent + 31) >> 5;
  const int t0 = split * tiles_per_split;
  const int t1 = min(ntiles, t0 + tiles_per_split);
  // S^T of query qrow / TQP has ncent + 1 rows; the last, all -inf, is the
  // sentinel that the document scorer reads for token slots past a document
  const int64_t st_base = (qrow / TQP) * (int64_t)(ncent + 1) * TQP + (qrow % TQP);
  if (WRITE_ST && split == 0 && wave == 0 && h == 0) ST[st_base + (int64_t)ncent * TQP] = -INFINITY;

  for (int t = t0 + wave; t < t1; t += 4) {
    // rows past the last centroid repeat it; their scores are dropped below
    const int crow = min(t * 32 + col, ncent - 1);
    bf16x8 a[8];
    {
      const uint4 *cp = (const uint4 *)(cent + (int64_t)crow * 128 + 64 * h);
#pragma unroll
      for (int s = 0; s < 8; ++s) a[s] = as_bf16x8(cp[s]);
    }
    __builtin_amdgcn_sched_barrier(0);  // the tile's 8 loads in flight together
    f32x16 acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], bq[s], acc, 0, 0, 0);
    // D layout: lane (col, h), register v holds centroid t*32 + 8(v/4) + 4h + v%4
    const int cbase = t * 32 + 4 * h;
    const bool full = t * 32 + 32 <= ncent;  // wave-uniform: only the last tile is partial
    if (WRITE_ST) {
      float *stp = ST + st_base + (int64_t)cbase * TQP;
      // S^T is read only by the document scorer, after the walk and the
      // select: streaming (non-temporal) stores keep it out of the way
      if (full) {
#pragma unroll
        for (int v = 0; v < 16; ++v) __builtin_nontemporal_store(acc[v], &stp[(8 * (v >> 2) + (v & 3)) * TQP]);
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (cbase + 8 * (v >> 2) + (v & 3) < ncent)
            __builtin_nontemporal_store(acc[v], &stp[(8 * (v >> 2) + (v & 3)) * TQP]);
      }
    }
    // wave-uniform; lists of 16 stay on the networks throughout (measured faster)
    const bool network = !TAU && (PMAX == 16 || (PMAX <= 8 && 16 * ((t - t0 - wave) / 4 + 1) <= 128 * PMAX));
    if constexpr (PMAX <= 16) {
      if (network) {
        uint64_t K[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) K[v] = pack_key(to_key(acc[v]), (uint32_t)(cbase + 8 * (v >> 2) + (v & 3)));
        if (!full) {
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (cbase + 8 * (v >> 2) + (v & 3) >= ncent) K[v] = 0;
        }
        fold_tile<PMAX>(L, K);
      }
    }
    if (!network) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int c = cbase + 8 * (v >> 2) + (v & 3);
        if (c < ncent) {
          const uint64_t K = pack_key(to_key(acc[v]), (uint32_t)c);
          if (K >= tr && K > L[PMAX - 1]) insert_desc<PMAX>(L, K);
        }
      }
    }
  }
  // lanes h=1 hand their lists to lanes h=0 (same query row)
#pragma unroll
  for (int i = 0; i < PMAX; ++i) {
    const uint64_t K = shfl_xor_u64(L[i], 32);
    if (h == 0 && K > L[PMAX - 1]) insert_desc<PMAX>(L, K);
  }
  if (wave > 0 && h == 0) {
#pragma unroll
    for (int i = 0; i < PMAX; ++i) lds[wave - 1][col][i] = L[i];
  }
  __syncthreads();
  if (wave == 0 && h == 0) {
    for (int w = 0; w < 3; ++w)
      for (int i = 0; i < PMAX; ++i) {
        const uint64_t K = lds[w][col][i];
        if (K <= L[PMAX - 1]) break;  // the source list is sorted
        insert_desc<PMAX>(L, K);
      }
    uint64_t *out = part + ((int64_t)split * rows + qrow) * PMAX;
#pragma unroll
    for (int i = 0; i < PMAX; ++i) out[i] = L[i];
  }
}

// Splits of the centroid tiles: ~8192 workgroups (measured at 8.8M: shorter
// workgroups end a launch with fewer CUs idle, 55.5 -> 49.9 ms per step
// against ~2048), at least 4 tiles (one per wave) per split, at most 512
// splits (the merge folds every split's list).
static void plan_splits(int64_t rows, int ncent, int &nsplit, int &tiles_per_split) {
  const int ntiles = (ncent + 31) / 32;
  const int64_t ncb = rows / 32;
  int64_t want = std::min<int64_t>(512, (8192 + ncb - 1) / ncb);
  int64_t maxsplit = (ntiles + 3) / 4;
  int64_t ns = want < 1 ? 1 : want;
  if (ns > maxsplit) ns = maxsplit;
  if (ns > 65535) ns = 65535;
  tiles_per_split = (int)((ntiles + ns - 1) / ns);
  nsplit = (ntiles + tiles_per_split - 1) / tiles_per_split;
}

ProbePlan plan_probe(int64_t rows, int ncent, int nprobe) {
  ProbePlan p;
  p.pmax = nprobe <= 4 ? 4 : nprobe <= 8 ? 8 : nprobe <= 16 ? 16 : nprobe <= 32 ? 32 : 64;
  plan_splits(rows, ncent, p.nsplit, p.tiles_per_split);
  // with many centroids, the first 1/16 of them first give every row a lower
  // bound on its nprobe-th best key
  p.sample = ncent >= 65536 ? (ncent / 16 + 31) / 32 * 32 : 0;
  if (p.sample) plan_splits(rows, p.sample, p.s_nsplit, p.s_tiles_per_split);
  return p;
}

size_t probe_part_bytes(const ProbePlan &p, int64_t rows) {
  const int64_t ns = std::max(p.nsplit, p.sample ? p.s_nsplit : 0);
  return (size_t)ns * rows * p.pmax * 8 + (p.sample ? (size_t)rows * 8 : 0);
}

// Per row (one wave each): the nprobe-th best key over the partial lists of
// nsplit splits, folded as k_probe_merge folds them.
template <int PMAX>
__global__ __launch_bounds__(256) void k_probe_tau(const uint64_t *__restrict__ part, int64_t rows, int nsplit,
                                                   int nprobe, uint64_t *__restrict__ tau) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  uint64_t L[PMAX];
#pragma unroll
  for (int i = 0; i < PMAX; ++i) L[i] = 0;
  for (int sp = lane; sp < nsplit; sp += 64) {
    const uint64_t *src = part + ((int64_t)sp * rows + row) * PMAX;
    for (int i = 0; i < PMAX; ++i) {
      const uint64_t K = src[i];
      if (K <= L[PMAX - 1]) break;
      insert_desc<PMAX>(L, K);
    }
  }
  uint64_t best = 0;
  for (int r = 0; r < nprobe; ++r) {
    best = L[0];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const uint64_t o = shfl_xor_u64(best, m);
      best = o > best ? o : best;
    }
    if (L[0] == best) {  // keys are unique: one lane owns the winner
#pragma unroll
      for (int i = 0; i < PMAX - 1; ++i) L[i] = L[i + 1];
      L[PMAX - 1] = 0;
    }
  }
  if (lane == 0) tau[row] = best;
}

template <int P, int TQP>
static void launch_probe_t(const uint16_t *Qs, int64_t rows, const uint16_t *cent, int ncent, const ProbePlan &p,
                           int nprobe, uint64_t *part, float *ST, hipStream_t s) {
  uint64_t *tau = nullptr;
  if (p.sample) {
    // the sample's lists, then each row's bound
    const int64_t ns = std::max(p.nsplit, p.s_nsplit);
    tau = part + (size_t)ns * rows * P;
    hipLaunchKernelGGL((k_probe<P, TQP, false, false>), dim3((unsigned)(rows / 32), (unsigned)p.s_nsplit), dim3(256),
                       0, s, Qs, cent, p.sample, p.s_tiles_per_split, rows, part, (float *)nullptr,
                       (const uint64_t *)nullptr);
    hipLaunchKernelGGL((k_probe_tau<P>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, part, rows, p.s_nsplit,
                       nprobe, tau);
  }
  dim3 grid((unsigned)(rows / 32), (unsigned)p.nsplit);
  if (ST && tau)
    hipLaunchKernelGGL((k_probe<P, TQP, true, true>), grid, dim3(256), 0, s, Qs, cent, ncent, p.tiles_per_split, rows,
                       part, ST, (const uint64_t *)tau);
  else if (ST)
    hipLaunchKernelGGL((k_probe<P, TQP, true, false>), grid, dim3(256), 0, s, Qs, cent, ncent, p.tiles_per_split, rows,
                       part, ST, (const uint64_t *)nullptr);
  else if (tau)
    hipLaunchKernelGGL((k_probe<P, TQP, false, true>), grid, dim3(256), 0, s, Qs, cent, ncent, p.tiles_per_split, rows,
                       part, ST, (const uint64_t *)tau);
  else
    hipLaunchKernelGGL((k_probe<P, TQP, false, false>), grid, dim3(256), 0, s, Qs, cent, ncent, p.tiles_per_split,
                       rows, part, ST, (const uint64_t *)nullptr);
}

template <int P>
static void launch_probe_p(const uint16_t *Qs, int64_t rows, int TQP, const uint16_t *cent, int ncent,
                           const ProbePlan &p, int nprobe, uint64_t *part, float *ST, hipStream_t s) {
  if (TQP == 32) launch_probe_t<P, 32>(Qs, rows, cent, ncent, p, nprobe, part, ST, s);
  else launch_probe_t<P, 64>(Qs, rows, cent, ncent, p, nprobe, part, ST, s);
}

void launch_probe(const uint16_t *Qs, int64_t rows, int TQP, const uint16_t *cent, int ncent, const ProbePlan &p,
                  int nprobe, uint64_t *part, float *ST, hipStream_t s) {
  switch (p.pmax) {
    case 4: launch_probe_p<4>(Qs, rows, TQP, cent, ncent, p, nprobe, part, ST, s); break;
    case 8: launch_probe_p<8>(Qs, rows, TQP, cent, ncent, p, nprobe, part, ST, s); break;
    case 16: launch_probe_p<16>(Qs, rows, TQP, cent, ncent, p, nprobe, part, ST, s); break;
    case 32: launch_probe_p<32>(Qs, rows, TQP, cent, ncent, p, nprobe, part, ST, s); break;
    default: launch_probe_p<64>(Qs, rows, TQP, cent, ncent, p, nprobe, part, ST, s); break;
  }
}

// --------------------------------------------------------------- merge
// One wave per query row: each lane folds the sorted partial lists of splits
// lane, lane+64, ... into its own list; then nprobe rounds of a wave-wide
// maximum pop the winners in order.
template <int PMAX>
__global__ __launch_bounds__(256) void k_probe_merge(const uint64_t *__restrict__ part, int64_t nq, int Tq, int TQP,
                                                     int nsplit, int nprobe, int32_t *__restrict__ cent_ids,
                                                     int32_t *__restrict__ cent_keys) {
  const int lane = threadIdx.x & 63;
  const int64_t wrow = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // over nq*Tq valid rows
  if (wrow >= nq * Tq) return;
  const int64_t q = wrow / Tq;
  const int j = (int)(wrow - q * Tq);
  const int64_t row = q * TQP + j;
  const int64_t rows = nq * TQP;
  uint64_t L[PMAX];
#pragma unroll
  for (int i = 0; i < PMAX; ++i) L[i] = 0;
  for (int sp = lane; sp < nsplit; sp += 64) {
    const uint64_t *src = part + ((int64_t)sp * rows + row) * PMAX;
    for (int i = 0; i < PMAX; ++i) {
      const uint64_t K = src[i];
      if (K <= L[PMAX - 1]) break;
      insert_desc<PMAX>(L, K);
    }
  }
  int32_t *oi = cent_ids + row * nprobe;
  int32_t *ok = cent_keys + row * nprobe;
  for (int r = 0; r < nprobe; ++r) {
    uint64_t best = L[0];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const uint64_t o = shfl_xor_u64(best, m);
      best = o > best ? o : best;
    }
    // keys are unique (distinct ids), so exactly one lane owns the winner
    if (L[0] == best) {
#pragma unroll
      for (int i = 0; i < PMAX - 1; ++i) L[i] = L[i + 1];
      L[PMAX - 1] = 0;
    }
    if (lane == 0) {
      oi[r] = (int32_t)key_id(best);
      ok[r] = key_score(best);
    }
  }
}

void launch_probe_merge(const uint64_t *part, int64_t nq, int Tq, int TQP, const ProbePlan &p, int nprobe,
                        int32_t *cent_ids, int32_t *cent_keys, hipStream_t s) {
  const int64_t nrows = nq * Tq;
  dim3 grid((unsigned)((nrows + 3) / 4));
  switch (p.pmax) {
    case 4: hipLaunchKernelGGL(k_probe_merge<4>, grid, dim3(256), 0, s, part, nq, Tq, TQP, p.nsplit, nprobe, cent_ids, cent_keys); break;
    case 8: hipLaunchKernelGGL(k_probe_merge<8>, grid, dim3(256), 0, s, part, nq, Tq, TQP, p.nsplit, nprobe, cent_ids, cent_keys); break;
    case 16: hipLaunchKernelGGL(k_probe_merge<16>, grid, dim3(256), 0, s, part, nq, Tq, TQP, p.nsplit, nprobe, cent_ids, cent_keys); break;
    case 32: hipLaunchKernelGGL(k_probe_merge<32>, grid, dim3(256), 0, s, part, nq, Tq, TQP, p.nsplit, nprobe, cent_ids, cent_keys); break;
    default: hipLaunchKernelGGL(k_probe_merge<64>, grid, dim3(256), 0, s, part, nq, Tq, TQP, p.nsplit, nprobe, cent_ids, cent_keys); break;
  }
}

}  // namespace chimera
