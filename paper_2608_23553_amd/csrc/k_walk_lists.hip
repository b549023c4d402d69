// k_walk_lists.hip - candidate generation and partial scores for an index
// without dense posting lists (Sec. 3.2: the candidate set S and F', Alg. 2,
// with the centroid score standing in for the token score).
//
// The same outputs as the bucketed walk of k_prune.hip, organised the other
// way round: there, every list's next entries wait in registers and are
// gathered per rank into LDS buckets, which pays off when a few hot lists
// carry most entries (Zipf-popular corpora, where those lists become dense
// masks).  When the centroids are used about evenly, every probed list
// holds a few to a few dozen entries per range, more than a thread's window,
// and here each list is walked straight from memory by one wave at its rank.
//
// Workgroup (query q, group g): the doc ranges [d0, d0 + R) of a contiguous
// group of ranges, one after the other.  The state of a range (per document,
// the mask of query tokens already credited and F') lives in LDS, so the
// atomics are LDS atomics and each document's F' is written to HBM once.
// Every probed list (query token j, rank r) keeps a cursor in LDS across the
// group's ranges: it is positioned once (by binary search, not at all for
// the first group) and then only moves forward, and a list whose next
// document lies past the current range costs nothing there.  For each rank
// r (in order, one barrier per rank) every list of that rank is walked up to
// the range's end by one wave.  Query tokens that probe the same centroid at
// the same rank share one walk of its list: one atomic OR of the group's
// token mask tells which of them see the document for the first time.  The
// workgroup then writes F' (or NO_HIT for documents outside S_Q and deleted
// ones) and adds the range's histogram of the top 12 bits of the order key to
// the query's histogram, the first pass of the refinement select.
// Workgroup b runs on XCD b % 8; with 8 or more queries all groups of query q
// run on XCD q % 8, with fewer they spread over every XCD.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

constexpr int LW_THREADS = 512;

// Walk state of one probed list (rank r, query token j): entries
// ivf_doc[beg .. beg + len), cursor pos and the document at the cursor
// (INT32_MAX past the end, or when another token's list stands for this
// one), and the group's token mask and score sum.
template <typename MaskT>
struct ListCursor {
  int64_t beg;
  MaskT mask;
  int32_t pos, len, next, gsum;
};

// One wave walks a list from pos up to the range's end d1, U blocks of 64
// entries per step (entries past d1 are read but not applied; the next range
// reads them again); leaves pos at the first entry >= d1 and next = its doc.
template <int U, typename MaskT>
__device__ __forceinline__ void walk_to_end(const int32_t *__restrict__ list, int32_t len, int64_t d0, int64_t d1,
                                            MaskT gmask, int32_t gsum, const int32_t *keys, int lane, MaskT *smask,
                                            int32_t *sfp, int32_t &pos, int32_t &next) {
  bool done = false;
  while (!done) {
    int32_t doc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int32_t p = pos + 64 * u + lane;
      doc[u] = p < len ? list[p] : INT32_MAX;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool in = doc[u] < d1;
      if (in) {
        const int v = (int)(doc[u] - d0);
        const MaskT fresh = gmask & ~atomicOr(&smask[v], gmask);  // tokens for which this is the first hit
        if (fresh == gmask) {
          atomicAdd(&sfp[v], gsum);
        } else if (fresh) {
          int32_t add = 0;
          for (MaskT m = fresh; m; m &= m - 1) add += keys[__builtin_ctzll((unsigned long long)m)];
          atomicAdd(&sfp[v], add);
        }
      }
      const unsigned long long out = __ballot(!in);  // lanes at or past the range's end
      if (out && !done) {
        const int first = __ffsll((long long)out) - 1;
        next = __shfl(doc[u], first, 64);
        pos += 64 * u + first;
        done = true;
      }
    }
    if (!done) pos += 64 * U;
  }
}

// Documents per range: 8192 with 32-bit token masks and fewer than 512
// lists, else 4096.
static inline int lw_range_docs(int TQP, int nprobe, int Tq) { return TQP == 32 && nprobe * Tq < 512 ? 8192 : 4096; }

template <typename MaskT, int R>
__global__ __launch_bounds__(LW_THREADS) void k_list_walk(
    const int32_t *__restrict__ cent_ids, const int32_t *__restrict__ cent_keys, int64_t nq, int Tq, int TQP,
    int nprobe, const int64_t *__restrict__ ivf_off, const int32_t *__restrict__ ivf_doc, int64_t ndocs, int ncent,
    const uint64_t *__restrict__ deleted, int nranges, int G, int M, int32_t *__restrict__ fp,
    uint32_t *__restrict__ hist) {
  static_assert(R * sizeof(MaskT) >= SEL_BINS * 4, "the histogram reuses the mask array");
  extern __shared__ __align__(16) unsigned char lw_lds[];
  MaskT *smask = (MaskT *)lw_lds;                              // [R]
  int32_t *sfp = (int32_t *)(smask + R);                       // [R]
  ListCursor<MaskT> *L = (ListCursor<MaskT> *)(sfp + R);       // [nprobe][Tq]
  int32_t *skey = (int32_t *)(L + nprobe * Tq);                // [nprobe][Tq] S[j][c] keys
  int32_t *scid = skey + nprobe * Tq;                          // [nprobe][Tq] centroid ids
  const int b = blockIdx.x;
  const int64_t q = nq >= 8 ? (b & 7) + 8 * (int64_t)((b >> 3) / G) : b / G;
  const int g = nq >= 8 ? (b >> 3) % G : b % G;
  if (q >= nq) return;
  const int rg0 = g * M, rg1 = min(nranges, rg0 + M);
  if (rg0 >= rg1) return;  // uniform, before any barrier
  const int64_t dstart = (int64_t)rg0 * R;
  const int nl = nprobe * Tq;
  for (int t = threadIdx.x; t < nl; t += LW_THREADS) {
    const int r = t / Tq, j = t - r * Tq;
    const int64_t e = (q * TQP + j) * nprobe + r;
    scid[t] = cent_ids[e];
    skey[t] = cent_keys[e];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < nl; t += LW_THREADS) {
    const int r = t / Tq, j = t - r * Tq;
    const int32_t c = scid[t];
    ListCursor<MaskT> w;
    w.beg = 0;
    w.pos = 0;
    w.len = 0;
    w.mask = 0;
    w.gsum = 0;
    // one pass over the rank's centroids: is j the group's first token, and
    // the group's mask and score sum
    bool head = (uint32_t)c < (uint32_t)ncent;
    MaskT gm = 0;
    int32_t gs = 0;
    for (int i = 0; i < Tq; ++i) {
      const bool same = scid[r * Tq + i] == c;
      head = head && !(same && i < j);
      gm |= same ? (MaskT)1 << i : (MaskT)0;
      gs += same ? skey[r * Tq + i] : 0;
    }
    if (head) {
      w.mask = gm;
      w.gsum = gs;
      const int64_t beg = ivf_off[c], end = ivf_off[c + 1];
      const int64_t p = dstart > 0 ? lower_bound_i32(ivf_doc, beg, end, dstart) : beg;
      w.beg = beg;
      w.len = (int32_t)(end - beg);
      w.pos = (int32_t)(p - beg);
    }
    w.next = w.pos < w.len ? ivf_doc[w.beg + w.pos] : INT32_MAX;
    L[t] = w;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = LW_THREADS / 64;
  for (int rg = rg0; rg < rg1; ++rg) {
    const int64_t d0 = (int64_t)rg * R;
    const int64_t d1 = min(ndocs, d0 + R);
    const int nd = (int)(d1 - d0);
    for (int v = threadIdx.x; v < R; v += LW_THREADS) {
      smask[v] = 0;
      sfp[v] = 0;
    }
    __syncthreads();  // the lists are set up; the previous range's reads are done
    for (int r = 0; r < nprobe; ++r) {
      // list j of rank r is always walked by wave j % nwaves
      for (int j = wave; j < Tq; j += nwaves) {
        ListCursor<MaskT> *w = &L[r * Tq + j];
        if (w->next >= d1) continue;  // wave-uniform: nothing of this list in the range
        const MaskT gmask = w->mask;
        const int32_t gsum = w->gsum, len = w->len;
        const int32_t *list = ivf_doc + w->beg;
        int32_t pos = w->pos, next = INT32_MAX;
        // lists expected to hold more than 64 entries per range keep 8 blocks
        // of 64 entries in flight per step, others one
        if ((int64_t)len * R > 64 * ndocs)
          walk_to_end<8>(list, len, d0, d1, gmask, gsum, skey + r * Tq, lane, smask, sfp, pos, next);
        else
          walk_to_end<1>(list, len, d0, d1, gmask, gsum, skey + r * Tq, lane, smask, sfp, pos, next);
        if (lane == 0) {
          w->pos = pos;
          w->next = next;
        }
      }
      __syncthreads();  // rank r's LDS updates complete before rank r+1's
    }
    // documents outside S_Q, and deleted ones, get NO_HIT
    for (int v = threadIdx.x; v < nd; v += LW_THREADS)
      if (smask[v] == 0 || (deleted && ((deleted[(d0 + v) >> 6] >> ((d0 + v) & 63)) & 1))) sfp[v] = NO_HIT;
    __syncthreads();
    uint32_t *sh = (uint32_t *)smask;  // the masks are no longer needed
    for (int i = threadIdx.x; i < SEL_BINS; i += LW_THREADS) sh[i] = 0;
    __syncthreads();
    int32_t *f = fp + q * ndocs + d0;
    for (int v = threadIdx.x; v < nd; v += LW_THREADS) {
      const int32_t x = sfp[v];
      f[v] = x;
      if (x != NO_HIT) atomicAdd(&sh[fp_key(x) >> 20], 1u);
    }
    __syncthreads();
    uint32_t *hq = hist + q * SEL_BINS;
    for (int i = threadIdx.x; i < SEL_BINS; i += LW_THREADS)
      if (sh[i]) atomicAdd(&hq[i], sh[i]);
    __syncthreads();  // sh (the mask array) is cleared by the next range
  }
}

template <typename MaskT, int R>
static void launch_lw_t(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                 const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent, const uint64_t *deleted,
                 int32_t *fp, uint32_t *hist, hipStream_t s) {
  const int nranges = (int)((ndocs + R - 1) / R);
  // ranges per workgroup: enough groups per query for about 4096 workgroups
  int G = (int)std::min<int64_t>(nranges, std::max<int64_t>(1, (4096 + nq - 1) / nq));
  const int M = (nranges + G - 1) / G;
  G = (nranges + M - 1) / M;
  const int64_t blocks = (nq >= 8 ? (nq + 7) / 8 * 8 : nq) * G;
  if (blocks == 0 || nranges == 0) return;
  const size_t lds = list_walk_lds_bytes(TQP, nprobe, Tq);
  static bool attr = [] {
    return hipFuncSetAttribute((const void *)k_list_walk<MaskT, R>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               160 * 1024) == hipSuccess;
  }();
  (void)attr;
  hipLaunchKernelGGL((k_list_walk<MaskT, R>), dim3((unsigned)blocks), dim3(LW_THREADS), lds, s, cent_ids, cent_keys,
                     nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, deleted, nranges, G, M, fp, hist);
}

size_t list_walk_lds_bytes(int TQP, int nprobe, int Tq) {
  const size_t mask = TQP == 32 ? 4 : 8, R = (size_t)lw_range_docs(TQP, nprobe, Tq);
  const size_t cur = TQP == 32 ? sizeof(ListCursor<uint32_t>) : sizeof(ListCursor<unsigned long long>);
  return R * (mask + 4) + (size_t)nprobe * Tq * (cur + 8);
}

void launch_list_walk(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                      const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent,
                      const uint64_t *deleted, int32_t *fp, uint32_t *hist, hipStream_t s) {
  if (TQP == 32 && lw_range_docs(TQP, nprobe, Tq) == 8192)
    launch_lw_t<uint32_t, 8192>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, deleted, fp,
                                hist, s);
  else if (TQP == 32)
    launch_lw_t<uint32_t, 4096>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, deleted, fp,
                                hist, s);
  else
    launch_lw_t<unsigned long long, 4096>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent,
                                          deleted, fp, hist, s);
}

}  // namespace chimera
