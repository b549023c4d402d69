// k_prune.hip - candidate generation and candidate refinement.
//
// Candidate set (Sec. 3.2, the set S): documents with a token in a probed
// posting list.  Partial score (Sec. 3.2, the F' definition; Alg. 2):
//   F'(V) = sum_j max{ S[j][c] : c in C_j, V in list(c) }   (0 if none).
// The max is taken by visiting each query token's probed lists in rank
// order (C_j is sorted by S descending): the first list of rank r that holds
// V carries the maximum, so one atomic OR on a per-(query, doc) bit mask
// detects the first hit and one integer atomic add accumulates F'.  Integer
// atomics make the result independent of scheduling.  This plays the role of
// the paper's fused atomic aggregation (Sec. 4.2, Alg. 4) with one update
// per (doc, query token) instead of an atomic max per retrieved token, and
// with the score table held in LDS one document range at a time.
#include "device_common.h"
#include "internal.h"

namespace chimera {

__global__ __launch_bounds__(256) void k_fill_zero(uint4 *__restrict__ p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

void launch_fill_zero(void *p, size_t bytes, hipStream_t s) {
  // scratch carve-outs are 256-byte aligned and sized in 256-byte steps
  size_t n16 = (bytes + 15) / 16;
  if (!n16) return;
  size_t blocks = (n16 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, s, (uint4 *)p, n16);
}

// Workgroup (query q, doc range [d0, d0 + WALK_RANGE)): the state of the
// range lives in LDS, so the atomics are LDS atomics and each document's
// state is written to HBM once.  For each rank r (in order, one barrier per
// rank) every query token j clips its rank-r posting list to the range by
// binary search (lists are ascending) and walks the clipped part.  Workgroup
// b runs on XCD b % 8; all ranges of query q run on XCD q % 8.
constexpr int WALK_THREADS = 512;
constexpr int WALK_RANGE = 8192;

__device__ __forceinline__ int64_t lower_bound_i32(const int32_t *__restrict__ a, int64_t lo, int64_t hi, int64_t x) {
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if ((int64_t)a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

template <typename MaskT>
__global__ __launch_bounds__(WALK_THREADS) void k_cand_walk(
    const int32_t *__restrict__ cent_ids, const int32_t *__restrict__ cent_keys, int64_t nq, int Tq, int TQP,
    int nprobe, const int64_t *__restrict__ ivf_off, const int32_t *__restrict__ ivf_doc, int64_t ndocs, int ncent,
    int nranges, MaskT *__restrict__ mask, int32_t *__restrict__ fp) {
  __shared__ MaskT smask[WALK_RANGE];
  __shared__ int32_t sfp[WALK_RANGE];
  __shared__ int64_t lo_s[64], hi_s[64];
  __shared__ int32_t key_s[64];
  const int b = blockIdx.x;
  const int64_t q = (b & 7) + 8 * (int64_t)((b >> 3) / nranges);
  const int range = (b >> 3) % nranges;
  if (q >= nq) return;
  const int64_t d0 = (int64_t)range * WALK_RANGE;
  const int64_t d1 = min(ndocs, d0 + WALK_RANGE);
  const int nd = (int)(d1 - d0);
  for (int v = threadIdx.x; v < WALK_RANGE; v += WALK_THREADS) {
    smask[v] = 0;
    sfp[v] = 0;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = WALK_THREADS / 64;
  for (int r = 0; r < nprobe; ++r) {
    if (threadIdx.x < Tq) {
      const int j = threadIdx.x;
      const int32_t c = cent_ids[(q * TQP + j) * nprobe + r];
      int64_t lo = 0, hi = 0;
      if ((uint32_t)c < (uint32_t)ncent) {
        const int64_t beg = ivf_off[c], end = ivf_off[c + 1];
        lo = lower_bound_i32(ivf_doc, beg, end, d0);
        hi = lower_bound_i32(ivf_doc, lo, end, d1);
      }
      lo_s[j] = lo;
      hi_s[j] = hi;
      key_s[j] = cent_keys[(q * TQP + j) * nprobe + r];
    }
    __syncthreads();  // also orders rank r-1's LDS atomics before rank r's
    for (int j = wave; j < Tq; j += nwaves) {
      const MaskT bit = (MaskT)1 << j;
      const int32_t key = key_s[j];
      const int64_t hi = hi_s[j];
      for (int64_t p = lo_s[j] + lane; p < hi; p += 64) {
        const int v = (int)(ivf_doc[p] - d0);
        const MaskT old = atomicOr(&smask[v], bit);
        if (!(old & bit)) atomicAdd(&sfp[v], key);
      }
    }
    __syncthreads();
  }
  MaskT *m = mask + q * ndocs + d0;
  int32_t *f = fp + q * ndocs + d0;
  for (int v = threadIdx.x; v < nd; v += WALK_THREADS) {
    m[v] = smask[v];
    f[v] = sfp[v];
  }
}

void launch_cand_walk(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                      const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent, void *mask,
                      int32_t *fp, hipStream_t s) {
  const int nranges = (int)((ndocs + WALK_RANGE - 1) / WALK_RANGE);
  const int64_t blocks = (nq + 7) / 8 * 8 * nranges;
  if (blocks == 0) return;
  if (TQP == 32)
    hipLaunchKernelGGL(k_cand_walk<uint32_t>, dim3((unsigned)blocks), dim3(WALK_THREADS), 0, s, cent_ids, cent_keys,
                       nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, nranges, (uint32_t *)mask, fp);
  else
    hipLaunchKernelGGL(k_cand_walk<unsigned long long>, dim3((unsigned)blocks), dim3(WALK_THREADS), 0, s, cent_ids,
                       cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, nranges,
                       (unsigned long long *)mask, fp);
}

// ------------------------------------------------------- block helpers
// Exclusive prefix sum over the block; thread 0 leaves the block total in
// *total (shared), readable by every thread once the call returns.
__device__ __forceinline__ int block_exclusive_scan(int x, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      const int t = wsum[w];
      wsum[w] = acc;
      acc += t;
    }
    *total = acc;
  }
  __syncthreads();
  const int res = wsum[wave] + incl - x;
  __syncthreads();  // wsum is reused by the next call
  return res;
}

template <typename MaskT>
__device__ __forceinline__ bool is_hit(const MaskT *m, int64_t v) {
  return m[v] != 0;
}

// Per-query ordered compaction of hits.  mode 0: top-ncand refinement
// (F' desc, doc asc) written in ascending doc order; mode 1: every hit.
constexpr int SEL_THREADS = 1024;
constexpr int SEL_ITEMS = 4;

template <typename MaskT, int MODE>
__global__ __launch_bounds__(SEL_THREADS) void k_select(const MaskT *__restrict__ mask, const int32_t *__restrict__ fp,
                                                        int64_t ndocs, int ncand, const int64_t *__restrict__ offsets,
                                                        int32_t *__restrict__ out_ids, int32_t *__restrict__ out_keys,
                                                        int32_t *__restrict__ n_valid) {
  __shared__ int hist[256];
  __shared__ int wsum[16];
  __shared__ int s_total;
  __shared__ long long s_nhit;
  __shared__ unsigned s_prefix, s_pmask;
  __shared__ long long s_remaining;
  const int64_t q = blockIdx.x;
  const MaskT *m = mask + q * ndocs;
  const int32_t *f = fp + q * ndocs;

  // --- threshold by radix selection on u = F' ^ 0x80000000 (order-preserving)
  unsigned T = 0;
  long long need = 0;  // hits with u == T still to take
  bool take_all = true;
  if (MODE == 0) {
    if (threadIdx.x == 0) s_nhit = 0;
    __syncthreads();
    long long local = 0;
    for (int64_t v = threadIdx.x; v < ndocs; v += SEL_THREADS) local += is_hit(m, v);
    atomicAdd((unsigned long long *)&s_nhit, (unsigned long long)local);
    __syncthreads();
    take_all = s_nhit <= ncand;
    if (!take_all) {
      if (threadIdx.x == 0) { s_prefix = 0; s_pmask = 0; s_remaining = ncand; }
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int b = threadIdx.x; b < 256; b += SEL_THREADS) hist[b] = 0;
        __syncthreads();
        const unsigned prefix = s_prefix, pmask = s_pmask;
        for (int64_t v = threadIdx.x; v < ndocs; v += SEL_THREADS) {
          if (!is_hit(m, v)) continue;
          const unsigned u = (unsigned)f[v] ^ 0x80000000u;
          if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
          long long rem = s_remaining, cum = 0;
          int sel = 0;
          for (int b = 255; b >= 0; --b) {
            if (cum + hist[b] >= rem) { sel = b; break; }
            cum += hist[b];
          }
          s_remaining = rem - cum;
          s_prefix = prefix | ((unsigned)sel << shift);
          s_pmask = pmask | (255u << shift);
        }
        __syncthreads();
      }
      T = s_prefix;
      need = s_remaining;
    }
  }

  // --- ordered compaction
  int64_t base_out = MODE == 1 ? offsets[q] : q * (int64_t)ncand;
  long long written = 0, ties_seen = 0;
  const int64_t chunk = (int64_t)SEL_THREADS * SEL_ITEMS;
  for (int64_t c0 = 0; c0 < ndocs; c0 += chunk) {
    const int64_t v0 = c0 + (int64_t)threadIdx.x * SEL_ITEMS;
    int take_flags = 0, tie_flags = 0, ntie = 0;
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i) {
      const int64_t v = v0 + i;
      if (v < ndocs && is_hit(m, v)) {
        if (MODE == 1 || take_all) {
          take_flags |= 1 << i;
        } else {
          const unsigned u = (unsigned)f[v] ^ 0x80000000u;
          if (u > T) take_flags |= 1 << i;
          else if (u == T) { tie_flags |= 1 << i; ++ntie; }
        }
      }
    }
    int tie_total = 0;
    int tie_rank = 0;
    if (MODE == 0 && !take_all) {
      tie_rank = block_exclusive_scan(ntie, wsum, &s_total);
      tie_total = s_total;
    }
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i)
      if (tie_flags & (1 << i)) {
        if (ties_seen + tie_rank < need) take_flags |= 1 << i;
        ++tie_rank;
      }
    const int ntake = __popc(take_flags);
    int pos = block_exclusive_scan(ntake, wsum, &s_total);
    const int take_total = s_total;
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i)
      if (take_flags & (1 << i)) {
        const int64_t v = v0 + i;
        if (MODE == 1 || written + pos < ncand) {
          out_ids[base_out + written + pos] = (int32_t)v;
          if (MODE == 0) out_keys[base_out + written + pos] = f[v];
        }
        ++pos;
      }
    written += take_total;
    ties_seen += tie_total;
    __syncthreads();
  }
  if (MODE == 0) {
    for (int64_t i = written + threadIdx.x; i < ncand; i += SEL_THREADS) {
      out_ids[base_out + i] = -1;
      out_keys[base_out + i] = 0;
    }
    if (threadIdx.x == 0) n_valid[q] = (int32_t)(written < ncand ? written : ncand);
  }
}

void launch_select(const void *mask, const int32_t *fp, int64_t nq, int TQP, int64_t ndocs, int ncand,
                   int32_t *cand_ids, int32_t *cand_keys, int32_t *n_valid, hipStream_t s) {
  dim3 grid((unsigned)nq);
  if (TQP == 32)
    hipLaunchKernelGGL((k_select<uint32_t, 0>), grid, dim3(SEL_THREADS), 0, s, (const uint32_t *)mask, fp, ndocs, ncand,
                       (const int64_t *)nullptr, cand_ids, cand_keys, n_valid);
  else
    hipLaunchKernelGGL((k_select<unsigned long long, 0>), grid, dim3(SEL_THREADS), 0, s,
                       (const unsigned long long *)mask, fp, ndocs, ncand, (const int64_t *)nullptr, cand_ids,
                       cand_keys, n_valid);
}

template <typename MaskT>
__global__ __launch_bounds__(256) void k_count_hits(const MaskT *__restrict__ mask, int64_t ndocs,
                                                    int64_t *__restrict__ counts) {
  __shared__ unsigned long long acc;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  const MaskT *m = mask + (int64_t)blockIdx.x * ndocs;
  unsigned long long local = 0;
  for (int64_t v = threadIdx.x; v < ndocs; v += 256) local += m[v] != 0;
  atomicAdd(&acc, local);
  __syncthreads();
  if (threadIdx.x == 0) counts[blockIdx.x] = (int64_t)acc;
}

void launch_count_hits(const void *mask, int64_t nq, int TQP, int64_t ndocs, int64_t *counts, hipStream_t s) {
  if (TQP == 32)
    hipLaunchKernelGGL(k_count_hits<uint32_t>, dim3((unsigned)nq), dim3(256), 0, s, (const uint32_t *)mask, ndocs, counts);
  else
    hipLaunchKernelGGL(k_count_hits<unsigned long long>, dim3((unsigned)nq), dim3(256), 0, s,
                       (const unsigned long long *)mask, ndocs, counts);
}

void launch_list_hits(const void *mask, int64_t nq, int TQP, int64_t ndocs, const int64_t *offsets, int32_t *doc_ids,
                      hipStream_t s) {
  dim3 grid((unsigned)nq);
  if (TQP == 32)
    hipLaunchKernelGGL((k_select<uint32_t, 1>), grid, dim3(SEL_THREADS), 0, s, (const uint32_t *)mask,
                       (const int32_t *)nullptr, ndocs, 0, offsets, doc_ids, (int32_t *)nullptr, (int32_t *)nullptr);
  else
    hipLaunchKernelGGL((k_select<unsigned long long, 1>), grid, dim3(SEL_THREADS), 0, s,
                       (const unsigned long long *)mask, (const int32_t *)nullptr, ndocs, 0, offsets, doc_ids,
                       (int32_t *)nullptr, (int32_t *)nullptr);
}

}  // namespace chimera
