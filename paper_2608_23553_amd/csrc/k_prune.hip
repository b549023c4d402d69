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
#include <algorithm>
#include <climits>

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

// Workgroup (query q, group g): the document ranges [d0, d0 + R) of a
// contiguous group of ranges, one after the other.  The state of a range
// (per document: the mask of query tokens already credited, and F') lives in
// LDS, so the updates are LDS atomics and each document's F' is written to
// HBM once.  Query tokens that probe the same centroid at the same rank form
// a group whose list is walked once, with the group's token mask and score
// sum (on the Zipf-popular corpora this halves the entries walked).  Ranks
// are applied in order, one barrier apart, so the first rank whose list
// holds a document gives each token its maximum: one atomic OR of the
// group's mask tells which tokens see the document for the first time.
//
// Every list's next entries wait in registers, loaded a range ahead:
//  * a short list (a few entries per range, the usual case) belongs to one
//    thread for the workgroup's lifetime, with a window of its next WIN
//    entries;
//  * a long list (more than WALK_LONG entries expected per range) belongs to
//    one wave, with a window of its next 64 entries (one per lane);
//  * a dense list (see dense_lists) is not walked: each thread applies it to
//    the documents it owns from their 64-bit masks, loaded a range ahead.
// At the start of a range the windows' entries inside it are copied into
// per-rank buckets in LDS and the windows are refilled; the ranks then run
// over the buckets, so they wait on no memory.  Only a list with more
// entries in one range than its window holds goes on through memory, at its
// rank.  The workgroup then writes F' (or NO_HIT for documents outside S_Q)
// and adds the range's histogram of the top 12 bits of the order key to the
// query's histogram, the first pass of the refinement select.  Workgroup b
// runs on XCD b % 8: with 8 or more queries all groups of query q run on XCD
// q % 8, with fewer they spread over every XCD.
constexpr int WALK_THREADS = 512;
constexpr int WALK_WAVES = WALK_THREADS / 64;
constexpr int WALK_LONG = 4;        // expected entries per range above which a list belongs to a wave
constexpr int WALK_LONG_SLOTS = 4;  // lists per wave
constexpr int WALK_MAX_LONG = WALK_LONG_SLOTS * WALK_WAVES;  // beyond that, lists stay with threads
constexpr int WALK_MAX_LISTS = 4 * WALK_THREADS;              // Tq * nprobe
constexpr int WALK_SHORT_ENTRIES = 4096;                      // short-list windows in all
constexpr int WALK_BUCKET = WALK_SHORT_ENTRIES + WALK_MAX_LONG * 64;
constexpr int WALK_DOC_BITS = 13;   // a bucket entry: list index << 13 | document in the range

// Window of a thread's short list: WIN = 8, 4 or 2 entries as a thread owns
// 1, 2 or 4 lists (WALK_SHORT_ENTRIES in all).
template <int LPT>
constexpr int walk_win() {
  return WALK_SHORT_ENTRIES / (LPT * WALK_THREADS);
}

// Documents per range: 4096 with 32-bit token masks, 2048 with 64-bit masks
// (two workgroups per compute unit; 8192 needs one, measured 4x slower).
static inline int walk_range_docs(int TQP, int, int) { return TQP == 32 ? 4096 : 2048; }

// LDS cursor of a wave's list: entries ivf_doc[beg .. beg + len), pos the
// first entry not yet credited; t its list index r * Tq + j.
struct LongList {
  int64_t beg;
  int32_t pos, len, t, rank, n, off;  // n, off: entries in the current range and their bucket offset
};

// Register state of a thread's short list: entries lp[0 .. len); e[i] holds
// lp[pos0 + i] for i < avail; e[0 .. c) are credited.  rank < 0: no list.
template <int WIN>
struct ShortList {
  const int32_t *lp;
  int32_t len, pos0, avail, c, rank, t;
  int32_t e[WIN];
};

// Credits the group (gmask, gsum) to document v of the range: the tokens of
// the group not yet seen there add their scores.
template <typename MaskT>
__device__ __forceinline__ void credit(MaskT *smask, int32_t *sfp, int v, MaskT gmask, int32_t gsum,
                                       const int32_t *keys) {
  const MaskT fresh = gmask & ~atomicOr(&smask[v], gmask);
  if (fresh == gmask) {
    atomicAdd(&sfp[v], gsum);
  } else if (fresh) {
    int32_t add = 0;
    for (MaskT m = fresh; m; m &= m - 1) add += keys[__builtin_ctzll((unsigned long long)m)];
    atomicAdd(&sfp[v], add);
  }
}

// One wave walks a list from pos up to the range's end d1, U blocks of 64
// entries per step; leaves pos at the first entry >= d1.
template <int U, typename MaskT>
__device__ __forceinline__ void walk_list(const int32_t *__restrict__ list, int32_t len, int64_t d0, int64_t d1,
                                          MaskT gmask, int32_t gsum, const int32_t *keys, int lane, MaskT *smask,
                                          int32_t *sfp, int32_t &pos) {
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
      if (in && !done) credit(smask, sfp, (int)(doc[u] - d0), gmask, gsum, keys);
      const unsigned long long out = __ballot(!in);  // lanes at or past the range's end
      if (out && !done) {
        pos += 64 * u + (__ffsll((long long)out) - 1);
        done = true;
      }
    }
    if (!done) pos += 64 * U;
  }
}

// Entries lp[pos .. pos + n) of a window, every load issued (indices past
// the list read its last entry and are not used), so each range issues the
// same loads.
template <int N>
__device__ __forceinline__ void load_window(const int32_t *lp, int32_t pos, int32_t len, int32_t (&e)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) e[i] = lp[min(pos + i, len - 1)];
}

// Byte offsets of the walk's LDS arrays (each 16-byte aligned).
struct WalkLds {
  size_t smask, sfp, bucket, ll, lmask, lsum, skey, scid, dcount, bcnt, bbase, dgm, dgs, dls, nlong, total;
};
__host__ __device__ inline WalkLds walk_lds_layout(int R, int mask_bytes, int nprobe, int Tq) {
  const size_t nl = (size_t)nprobe * Tq;
  WalkLds L;
  size_t o = 0;
  auto take = [&o](size_t bytes) {
    const size_t at = o;
    o += (bytes + 15) / 16 * 16;
    return at;
  };
  L.smask = take((size_t)R * mask_bytes);
  L.sfp = take((size_t)R * 4);
  L.bucket = take((size_t)WALK_BUCKET * 4);
  L.ll = take(WALK_MAX_LONG * sizeof(LongList));
  L.lmask = take(nl * mask_bytes);
  L.lsum = take(nl * 4);
  L.skey = take(nl * 4);
  L.scid = take(nl * 4);
  L.dcount = take((size_t)nprobe * 4);
  L.bcnt = take((size_t)nprobe * 4);
  L.bbase = take((size_t)nprobe * 4);
  L.dgm = take(nl * mask_bytes);
  L.dgs = take(nl * 4);
  L.dls = take(nl);
  L.nlong = take(4);
  L.total = o;
  return L;
}

template <typename MaskT, int R, int LPT>
__global__ __launch_bounds__(WALK_THREADS) void k_cand_walk(
    const int32_t *__restrict__ cent_ids, const int32_t *__restrict__ cent_keys, int64_t nq, int Tq, int TQP,
    int nprobe, const int64_t *__restrict__ ivf_off, const int32_t *__restrict__ ivf_doc, int64_t ndocs, int ncent,
    int ndense, const int8_t *__restrict__ dense_slot, const uint64_t *__restrict__ doc_dense,
    const uint64_t *__restrict__ deleted, int nranges, int G, int M, int32_t *__restrict__ fp,
    uint32_t *__restrict__ hist) {
  constexpr int DPT = R / WALK_THREADS;  // documents of a range each thread owns in the dense phase
  constexpr int WIN = walk_win<LPT>();
  static_assert(R * sizeof(MaskT) >= SEL_BINS * 4, "the histogram reuses the mask array");
  static_assert(R <= (1 << WALK_DOC_BITS), "a bucket entry holds the document in 13 bits");
  extern __shared__ __align__(16) unsigned char walk_lds[];
  const int nl = nprobe * Tq;
  const WalkLds lay = walk_lds_layout(R, (int)sizeof(MaskT), nprobe, Tq);
  MaskT *smask = (MaskT *)(walk_lds + lay.smask);        // [R] tokens already credited, per document
  int32_t *sfp = (int32_t *)(walk_lds + lay.sfp);        // [R] F' accumulators
  uint32_t *bucket = (uint32_t *)(walk_lds + lay.bucket);  // [WALK_BUCKET] the range's entries, by rank
  LongList *LL = (LongList *)(walk_lds + lay.ll);        // [WALK_MAX_LONG]
  MaskT *lmask = (MaskT *)(walk_lds + lay.lmask);        // [nl] group token masks
  int32_t *lsum = (int32_t *)(walk_lds + lay.lsum);      // [nl] group score sums
  int32_t *skey = (int32_t *)(walk_lds + lay.skey);      // [nl] S[j][c] keys, index r * Tq + j
  int32_t *scid = (int32_t *)(walk_lds + lay.scid);      // [nl] centroid ids
  int32_t *dcount = (int32_t *)(walk_lds + lay.dcount);  // [nprobe] dense groups per rank
  int32_t *bcnt = (int32_t *)(walk_lds + lay.bcnt);      // [nprobe] bucket entries per rank
  int32_t *bbase = (int32_t *)(walk_lds + lay.bbase);    // [nprobe] first bucket entry of each rank
  // the dense groups of rank r: k < dcount[r] at r * Tq + k
  MaskT *dgm = (MaskT *)(walk_lds + lay.dgm);            // [nl] token masks
  int32_t *dgs = (int32_t *)(walk_lds + lay.dgs);        // [nl] score sums
  int8_t *dls = (int8_t *)(walk_lds + lay.dls);          // [nl] dense slots
  int32_t *nlong = (int32_t *)(walk_lds + lay.nlong);    // wave-owned lists
  // workgroup b runs on XCD b % 8: with 8 or more queries, the groups of
  // query q run on XCD q % 8; fewer queries spread over every XCD
  const int b = blockIdx.x;
  const int64_t q = nq >= 8 ? (b & 7) + 8 * (int64_t)((b >> 3) / G) : b / G;
  const int g = nq >= 8 ? (b >> 3) % G : b % G;
  if (q >= nq) return;
  const int rg0 = g * M, rg1 = min(nranges, rg0 + M);
  if (rg0 >= rg1) return;  // uniform, before any barrier
  const int64_t dstart = (int64_t)rg0 * R;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t = threadIdx.x; t < nl; t += WALK_THREADS) {
    const int r = t / Tq, j = t - r * Tq;
    const int64_t e = (q * TQP + j) * nprobe + r;
    scid[t] = cent_ids[e];
    skey[t] = cent_keys[e];
  }
  for (int r = threadIdx.x; r < nprobe; r += WALK_THREADS) dcount[r] = 0;
  if (threadIdx.x == 0) *nlong = 0;
  __syncthreads();
  // classify list t = threadIdx.x + WALK_THREADS * i: group head or not,
  // dense, long or short; a short list stays with this thread (slot i)
  ShortList<WIN> S[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int t = threadIdx.x + WALK_THREADS * i;
    S[i].rank = -1;
    S[i].avail = 0;
    S[i].lp = ivf_doc;  // a readable entry for slots without a list
    S[i].len = 1;
    S[i].pos0 = 0;
    S[i].c = 0;
    if (t >= nl) continue;
    const int r = t / Tq, j = t - r * Tq;
    const int32_t c = scid[t];
    // one pass over the rank's centroids: is j the group's first token, and
    // the group's mask and score sum
    bool head = (uint32_t)c < (uint32_t)ncent;
    MaskT gm = 0;
    int32_t gs = 0;
    for (int u = 0; u < Tq; ++u) {
      const bool same = scid[r * Tq + u] == c;
      head = head && !(same && u < j);
      gm |= same ? (MaskT)1 << u : (MaskT)0;
      gs += same ? skey[r * Tq + u] : 0;
    }
    lmask[t] = gm;
    lsum[t] = gs;
    if (!head) continue;
    if (ndense > 0 && dense_slot[c] >= 0) {
      // a dense list: applied from the documents' masks, never walked
      const int k = atomicAdd(&dcount[r], 1);
      dls[r * Tq + k] = dense_slot[c];
      dgm[r * Tq + k] = gm;
      dgs[r * Tq + k] = gs;
      continue;
    }
    const int64_t beg = ivf_off[c], end = ivf_off[c + 1];
    const int64_t p = dstart > 0 ? lower_bound_i32(ivf_doc, beg, end, dstart) : beg;
    const int32_t len = (int32_t)(end - beg), pos = (int32_t)(p - beg);
    if (pos >= len) continue;  // nothing left in the group's documents
    if ((int64_t)(len - pos) * R > (int64_t)WALK_LONG * (ndocs - dstart)) {
      const int k = atomicAdd(nlong, 1);
      if (k < WALK_MAX_LONG) {
        LongList w;
        w.beg = beg;
        w.pos = pos;
        w.len = len;
        w.t = t;
        w.rank = r;
        LL[k] = w;
        continue;
      }
    }
    S[i].lp = ivf_doc + beg;
    S[i].len = len;
    S[i].pos0 = pos;
    S[i].c = 0;
    S[i].rank = r;
    S[i].t = t;
    S[i].avail = min(WIN, len - pos);
    load_window(S[i].lp, pos, len, S[i].e);
  }
  __syncthreads();
  // the wave's lists and their windows: slot i is list wave + WALK_WAVES * i
  const int nlw = min(*nlong, WALK_MAX_LONG);
  // (lane l holds entry pos + l, loaded as is: lanes past the list's end hold
  // its last entry and are masked where the window is read)
  int32_t lw[WALK_LONG_SLOTS];
#pragma unroll
  for (int i = 0; i < WALK_LONG_SLOTS; ++i) {
    const int k = wave + WALK_WAVES * i;
    if (k < nlw) {
      const LongList w = LL[k];
      lw[i] = ivf_doc[w.beg + min(w.pos + lane, w.len - 1)];
    }
  }
  // dense-list masks of the documents this thread owns (tid + WALK_THREADS * i),
  // loaded at the end of the previous range
  uint64_t dm[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) {
    const int64_t v = dstart + threadIdx.x + WALK_THREADS * i;
    dm[i] = ndense > 0 && v < ndocs ? doc_dense[v] : 0;
  }
  for (int rg = rg0; rg < rg1; ++rg) {
    const int64_t d0 = (int64_t)rg * R;
    const int64_t d1 = min(ndocs, d0 + R);
    const int nd = (int)(d1 - d0);
    for (int v = threadIdx.x; v < R; v += WALK_THREADS) {
      smask[v] = 0;
      sfp[v] = 0;
    }
    for (int r = threadIdx.x; r < nprobe; r += WALK_THREADS) bcnt[r] = 0;
    __syncthreads();  // the range is cleared; the previous range's reads are done

    // the windows' entries inside the range: count them per rank and reserve
    // their places in the rank's bucket
    int snew[LPT], soff[LPT];
    bool sovf[LPT];
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      snew[i] = 0;
      soff[i] = 0;
      sovf[i] = false;
      if (S[i].avail == 0) continue;
      int mt = 0;
#pragma unroll
      for (int u = 0; u < WIN; ++u) mt += (u < S[i].avail && S[i].e[u] < d1) ? 1 : 0;
      snew[i] = mt - S[i].c;
      sovf[i] = mt == S[i].avail && S[i].pos0 + S[i].avail < S[i].len;
      if (snew[i] > 0) soff[i] = atomicAdd(&bcnt[S[i].rank], snew[i]);
    }
#pragma unroll
    for (int i = 0; i < WALK_LONG_SLOTS; ++i) {
      const int k = wave + WALK_WAVES * i;
      if (k >= nlw) continue;  // wave-uniform
      const LongList w = LL[k];
      const int n = __popcll(__ballot(w.pos + lane < w.len && lw[i] < d1));
      if (lane == 0) {
        LL[k].n = n;
        if (n > 0) LL[k].off = atomicAdd(&bcnt[LL[k].rank], n);
      }
    }
    __syncthreads();
    if (wave == 0) {  // bucket base of each rank: exclusive prefix sum (nprobe <= 64)
      const int x = lane < nprobe ? bcnt[lane] : 0;
      int incl = x;
#pragma unroll
      for (int dd = 1; dd < 64; dd <<= 1) {
        const int y = __shfl_up(incl, dd, 64);
        if (lane >= dd) incl += y;
      }
      if (lane < nprobe) bbase[lane] = incl - x;
    }
    __syncthreads();
    // copy the entries into the buckets, then move every window forward;
    // the refills are needed a range later
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      if (S[i].avail == 0) continue;
      if (snew[i] > 0) {
        uint32_t *bk = bucket + bbase[S[i].rank] + soff[i] - S[i].c;
#pragma unroll
        for (int u = 0; u < WIN; ++u)
          if (u >= S[i].c && u < S[i].c + snew[i])
            bk[u] = (uint32_t)S[i].t << WALK_DOC_BITS | (uint32_t)(S[i].e[u] - d0);
      }
      S[i].c += snew[i];
    }
#pragma unroll
    for (int i = 0; i < WALK_LONG_SLOTS; ++i) {
      const int k = wave + WALK_WAVES * i;
      if (k >= nlw) continue;  // wave-uniform
      const LongList w = LL[k];
      const int n = w.n;
      if (n == 0) continue;
      if (lane < n) bucket[bbase[w.rank] + w.off + lane] = (uint32_t)w.t << WALK_DOC_BITS | (uint32_t)(lw[i] - d0);
      if (n < 64 && lane == 0) LL[k].pos = w.pos + n;  // a full window goes on through memory at its rank
    }
    __syncthreads();  // the buckets are complete

    for (int r = 0; r < nprobe; ++r) {
      const int ndg = dcount[r];
      const int32_t *keys = skey + r * Tq;
      // the rank's bucket, spread over every thread
      const int e1 = bbase[r] + bcnt[r];
      for (int e = bbase[r] + threadIdx.x; e < e1; e += WALK_THREADS) {
        const uint32_t x = bucket[e];
        const int t = (int)(x >> WALK_DOC_BITS);
        credit(smask, sfp, (int)(x & ((1u << WALK_DOC_BITS) - 1)), lmask[t], lsum[t], keys);
      }
      // lists with more entries in the range than their window held
#pragma unroll
      for (int i = 0; i < LPT; ++i) {
        if (!sovf[i] || S[i].rank != r) continue;
        int32_t p = S[i].pos0 + S[i].avail;
        const MaskT gm = lmask[S[i].t];
        const int32_t gs = lsum[S[i].t];
        while (p < S[i].len) {
          const int32_t d = S[i].lp[p];
          if (d >= d1) break;
          credit(smask, sfp, (int)(d - d0), gm, gs, keys);
          ++p;
        }
        S[i].pos0 = p;
        S[i].c = 0;
      }
#pragma unroll
      for (int i = 0; i < WALK_LONG_SLOTS; ++i) {
        const int k = wave + WALK_WAVES * i;
        if (k >= nlw) continue;  // wave-uniform
        const LongList w = LL[k];
        if (w.rank != r || w.n != 64) continue;
        int32_t pos = w.pos + 64;
        walk_list<8>(ivf_doc + w.beg, w.len, d0, d1, lmask[w.t], lsum[w.t], keys, lane, smask, sfp, pos);
        if (lane == 0) LL[k].pos = pos;
      }
      if (ndg > 0) {  // uniform
        // dense lists of rank r: each thread applies them to the documents it
        // owns from their masks.  The groups of one rank hold disjoint
        // tokens, so a document's hits add up to one token mask and one
        // score sum; the groups are visited in the same order by every lane.
        // They are credited with the same atomics as the rank's other lists,
        // whose tokens they do not share, so the two need no barrier between
        // them: only the earlier ranks must be complete.
        MaskT nb[DPT];
        int32_t sall[DPT];
#pragma unroll
        for (int i = 0; i < DPT; ++i) {
          nb[i] = 0;
          sall[i] = 0;
        }
        for (int k = 0; k < ndg; ++k) {
          const int sl = dls[r * Tq + k];
          const MaskT gm = dgm[r * Tq + k];
          const int32_t gs = dgs[r * Tq + k];
#pragma unroll
          for (int i = 0; i < DPT; ++i) {
            const bool hit = (dm[i] >> sl) & 1;
            nb[i] |= hit ? gm : (MaskT)0;
            sall[i] += hit ? gs : 0;
          }
        }
#pragma unroll
        for (int i = 0; i < DPT; ++i)
          if (nb[i]) credit(smask, sfp, threadIdx.x + WALK_THREADS * i, nb[i], sall[i], keys);
      }
      __syncthreads();  // rank r's LDS updates complete before rank r+1's
    }
    // the next range's inputs, loaded now and first read a range from now:
    // every window at its list's new position (its lines are cached), and
    // the dense masks
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      S[i].pos0 += S[i].c;
      S[i].c = 0;
      S[i].avail = S[i].rank < 0 ? 0 : min(WIN, S[i].len - S[i].pos0);
      load_window(S[i].lp, S[i].pos0, S[i].len, S[i].e);
    }
#pragma unroll
    for (int i = 0; i < WALK_LONG_SLOTS; ++i) {
      const int k = wave + WALK_WAVES * i;
      if (k < nlw) {  // wave-uniform
        const LongList w = LL[k];
        lw[i] = ivf_doc[w.beg + min(w.pos + lane, w.len - 1)];
      }
    }
    if (rg + 1 < rg1) {
#pragma unroll
      for (int i = 0; i < DPT; ++i) {
        const int64_t v = d1 + threadIdx.x + WALK_THREADS * i;
        dm[i] = ndense > 0 && v < ndocs ? doc_dense[v] : 0;
      }
    }
    // documents outside S_Q, and deleted ones, get NO_HIT
    for (int v = threadIdx.x; v < nd; v += WALK_THREADS)
      if (smask[v] == 0 || (deleted && ((deleted[(d0 + v) >> 6] >> ((d0 + v) & 63)) & 1))) sfp[v] = NO_HIT;
    __syncthreads();
    uint32_t *sh = (uint32_t *)smask;  // the masks are no longer needed
    for (int i = threadIdx.x; i < SEL_BINS; i += WALK_THREADS) sh[i] = 0;
    __syncthreads();
    int32_t *f = fp + q * ndocs + d0;
    for (int v = threadIdx.x; v < nd; v += WALK_THREADS) {
      const int32_t x = sfp[v];
      f[v] = x;
      if (x != NO_HIT) atomicAdd(&sh[fp_key(x) >> 20], 1u);
    }
    __syncthreads();
    uint32_t *hq = hist + q * SEL_BINS;
    for (int i = threadIdx.x; i < SEL_BINS; i += WALK_THREADS)
      if (sh[i]) atomicAdd(&hq[i], sh[i]);
    __syncthreads();  // sh (the mask array) is cleared by the next range
  }
}

size_t walk_lds_bytes(int TQP, int nprobe, int Tq) {
  if ((size_t)nprobe * Tq > (size_t)WALK_MAX_LISTS) return SIZE_MAX;
  // either walk may run (k_walk_lists.hip takes indexes without dense lists)
  return std::max(walk_lds_layout(walk_range_docs(TQP, nprobe, Tq), TQP == 32 ? 4 : 8, nprobe, Tq).total,
                  list_walk_lds_bytes(TQP, nprobe, Tq));
}

template <typename MaskT, int R, int LPT>
static void launch_walk_t(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                          const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent, int ndense,
                          const int8_t *dense_slot, const uint64_t *doc_dense, const uint64_t *deleted, int32_t *fp, uint32_t *hist,
                          hipStream_t s) {
  const int nranges = (int)((ndocs + R - 1) / R);
  // ranges per workgroup: enough groups per query for about 32768 workgroups
  // (measured at 8.8M and 1M: shorter workgroups leave fewer CUs idle at a
  // launch's end than fewer, longer ones; 8.8M walk 403 -> 383 ms, 1M 12.1
  // -> 10.0 ms, against about 4096)
  int G = (int)std::min<int64_t>(nranges, std::max<int64_t>(1, (32768 + nq - 1) / nq));
  const int M = (nranges + G - 1) / G;
  G = (nranges + M - 1) / M;
  const int64_t blocks = (nq >= 8 ? (nq + 7) / 8 * 8 : nq) * G;
  if (blocks == 0 || nranges == 0) return;
  const size_t lds = walk_lds_bytes(TQP, nprobe, Tq);
  static bool attr = [] {
    return hipFuncSetAttribute((const void *)k_cand_walk<MaskT, R, LPT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               160 * 1024) == hipSuccess;
  }();
  (void)attr;
  hipLaunchKernelGGL((k_cand_walk<MaskT, R, LPT>), dim3((unsigned)blocks), dim3(WALK_THREADS), lds, s, cent_ids,
                     cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, ndense, dense_slot, doc_dense,
                     deleted, nranges, G, M, fp, hist);
}

template <typename MaskT, int R>
static void launch_walk_r(int lpt, const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP,
                          int nprobe, const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent,
                          int ndense, const int8_t *dense_slot, const uint64_t *doc_dense, const uint64_t *deleted, int32_t *fp,
                          uint32_t *hist, hipStream_t s) {
  if (lpt <= 1)
    launch_walk_t<MaskT, R, 1>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, ndense,
                               dense_slot, doc_dense, deleted, fp, hist, s);
  else if (lpt <= 2)
    launch_walk_t<MaskT, R, 2>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, ndense,
                               dense_slot, doc_dense, deleted, fp, hist, s);
  else
    launch_walk_t<MaskT, R, 4>(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, ndense,
                               dense_slot, doc_dense, deleted, fp, hist, s);
}

void launch_cand_walk(const int32_t *cent_ids, const int32_t *cent_keys, int64_t nq, int Tq, int TQP, int nprobe,
                      const int64_t *ivf_off, const int32_t *ivf_doc, int64_t ndocs, int ncent, int ndense,
                      const int8_t *dense_slot, const uint64_t *doc_dense, const uint64_t *deleted, int32_t *fp, uint32_t *hist,
                      hipStream_t s) {
  // without dense lists the centroids are used about evenly: each probed list
  // is walked from memory at its rank (k_walk_lists.hip); measured 2x faster
  // there than the bucketed walk, which wins on skewed (Zipf) lists
  if (ndense == 0) {
    launch_list_walk(cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent, deleted, fp, hist, s);
    return;
  }
  const int lpt = (nprobe * Tq + WALK_THREADS - 1) / WALK_THREADS;  // at most 4 (walk_lds_bytes)
  if (TQP == 32)
    launch_walk_r<uint32_t, 4096>(lpt, cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs, ncent,
                                  ndense, dense_slot, doc_dense, deleted, fp, hist, s);
  else
    launch_walk_r<unsigned long long, 2048>(lpt, cent_ids, cent_keys, nq, Tq, TQP, nprobe, ivf_off, ivf_doc, ndocs,
                                            ncent, ndense, dense_slot, doc_dense, deleted, fp, hist, s);
}

// ------------------------------------------------------- block helpers
constexpr int SEL_THREADS = 1024;
constexpr int SEL_ITEMS = 4;
constexpr int SEL_UNROLL = 8;       // independent F' loads per thread in a histogram pass
constexpr int SEL_COMPACT_ITEMS = 16;  // consecutive documents per thread in k_select's compaction

// Exclusive prefix sum over the block; thread 0 leaves the block total in
// *total (shared), readable by every thread once the call returns.
__device__ __forceinline__ long long block_exclusive_scan(long long x, long long *wsum, long long *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  long long incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const long long y = __shfl_up(incl, d, 64);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long acc = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      const long long t = wsum[w];
      wsum[w] = acc;
      acc += t;
    }
    *total = acc;
  }
  __syncthreads();
  const long long res = wsum[wave] + incl - x;
  __syncthreads();  // wsum is reused by the next call
  return res;
}

// Radix-select step: over bins[0..nbins) taken from the highest bin down,
// find the bin b where the running count reaches rem.  Leaves b in *s_bin
// and the count of the bins above b in *s_above.
__device__ __forceinline__ void select_bin(const uint32_t *bins, int nbins, long long rem, long long *wsum,
                                           long long *s_tot, int *s_bin, long long *s_above) {
  const int per = (nbins + (int)blockDim.x - 1) / (int)blockDim.x;
  const int top = nbins - 1 - (int)threadIdx.x * per;  // this thread's bins: top, top-1, ... (descending)
  long long local = 0;
  for (int i = 0; i < per; ++i)
    if (top - i >= 0) local += bins[top - i];
  const long long excl = block_exclusive_scan(local, wsum, s_tot);
  if (excl < rem && excl + local >= rem) {
    long long cum = excl;
    for (int i = 0; i < per; ++i) {
      const int bb = top - i;
      if (bb < 0) break;
      if (cum + bins[bb] >= rem) {
        *s_bin = bb;
        *s_above = cum;
        break;
      }
      cum += bins[bb];
    }
  }
  __syncthreads();
}

// Per-query selection of the ncand best hits by (F' desc, doc asc), written
// in ascending doc order.  The first radix pass (top 12 key bits) comes from
// the walk's histogram; two more passes over F' (12 and 8 bits) give the
// exact threshold key T and how many documents with key T to keep (the
// lowest ids first).  MODE 1 lists every hit at offsets[q] (the candidate-set
// tap).
template <int MODE>
__global__ __launch_bounds__(SEL_THREADS) void k_select(const int32_t *__restrict__ fp,
                                                        const uint32_t *__restrict__ hist1, int64_t ndocs, int ncand,
                                                        const int64_t *__restrict__ offsets,
                                                        int32_t *__restrict__ out_ids, int32_t *__restrict__ out_keys,
                                                        int32_t *__restrict__ n_valid) {
  __shared__ uint32_t hist[SEL_BINS];
  __shared__ long long wsum[SEL_THREADS / 64];
  __shared__ long long s_tot, s_above;
  __shared__ int s_bin;
  const int64_t q = blockIdx.x;
  const int32_t *f = fp + q * ndocs;

  uint32_t T = 0;
  long long need = 0;  // hits with key == T still to take
  bool take_all = true;
  if (MODE == 0) {
    long long local = 0;
    for (int i = threadIdx.x; i < SEL_BINS; i += SEL_THREADS) {
      hist[i] = hist1[q * SEL_BINS + i];
      local += hist[i];
    }
    block_exclusive_scan(local, wsum, &s_tot);
    const long long nhit = s_tot;
    take_all = nhit <= ncand;
    if (!take_all) {
      long long rem = ncand;
      // pass 1 (histogram from the walk): key bits 31..20
      select_bin(hist, SEL_BINS, rem, wsum, &s_tot, &s_bin, &s_above);
      const uint32_t b1 = (uint32_t)s_bin;
      rem -= s_above;
      // pass 2: key bits 19..8 among keys with top bits b1
      for (int i = threadIdx.x; i < SEL_BINS; i += SEL_THREADS) hist[i] = 0;
      __syncthreads();
      for (int64_t v0 = threadIdx.x; v0 < ndocs; v0 += SEL_THREADS * SEL_UNROLL) {
        int32_t x[SEL_UNROLL];
#pragma unroll
        for (int i = 0; i < SEL_UNROLL; ++i) {
          const int64_t v = v0 + (int64_t)i * SEL_THREADS;
          x[i] = v < ndocs ? f[v] : NO_HIT;
        }
#pragma unroll
        for (int i = 0; i < SEL_UNROLL; ++i) {
          const uint32_t u = fp_key(x[i]);
          if (x[i] != NO_HIT && (u >> 20) == b1) atomicAdd(&hist[(u >> 8) & 4095u], 1u);
        }
      }
      __syncthreads();
      select_bin(hist, SEL_BINS, rem, wsum, &s_tot, &s_bin, &s_above);
      const uint32_t p2 = (b1 << 12) | (uint32_t)s_bin;
      rem -= s_above;
      // pass 3: key bits 7..0 among keys with top bits p2
      for (int i = threadIdx.x; i < 256; i += SEL_THREADS) hist[i] = 0;
      __syncthreads();
      for (int64_t v0 = threadIdx.x; v0 < ndocs; v0 += SEL_THREADS * SEL_UNROLL) {
        int32_t x[SEL_UNROLL];
#pragma unroll
        for (int i = 0; i < SEL_UNROLL; ++i) {
          const int64_t v = v0 + (int64_t)i * SEL_THREADS;
          x[i] = v < ndocs ? f[v] : NO_HIT;
        }
#pragma unroll
        for (int i = 0; i < SEL_UNROLL; ++i) {
          const uint32_t u = fp_key(x[i]);
          if (x[i] != NO_HIT && (u >> 8) == p2) atomicAdd(&hist[u & 255u], 1u);
        }
      }
      __syncthreads();
      select_bin(hist, 256, rem, wsum, &s_tot, &s_bin, &s_above);
      T = (p2 << 8) | (uint32_t)s_bin;
      need = rem - s_above;
    }
  }

  // --- ordered compaction
  const int64_t base_out = MODE == 1 ? offsets[q] : q * (int64_t)ncand;
  long long written = 0, ties_seen = 0;
  const int64_t chunk = (int64_t)SEL_THREADS * SEL_COMPACT_ITEMS;
  for (int64_t c0 = 0; c0 < ndocs; c0 += chunk) {
    const int64_t v0 = c0 + (int64_t)threadIdx.x * SEL_COMPACT_ITEMS;
    int take_flags = 0, tie_flags = 0, ntie = 0;
    int32_t xs[SEL_COMPACT_ITEMS];
#pragma unroll
    for (int i = 0; i < SEL_COMPACT_ITEMS; ++i) {
      const int64_t v = v0 + i;
      xs[i] = v < ndocs ? f[v] : NO_HIT;
      if (xs[i] != NO_HIT) {
        if (MODE == 1 || take_all) {
          take_flags |= 1 << i;
        } else {
          const uint32_t u = fp_key(xs[i]);
          if (u > T) take_flags |= 1 << i;
          else if (u == T) { tie_flags |= 1 << i; ++ntie; }
        }
      }
    }
    long long tie_total = 0, tie_rank = 0;
    if (MODE == 0 && !take_all) {
      tie_rank = block_exclusive_scan(ntie, wsum, &s_tot);
      tie_total = s_tot;
    }
#pragma unroll
    for (int i = 0; i < SEL_COMPACT_ITEMS; ++i)
      if (tie_flags & (1 << i)) {
        if (ties_seen + tie_rank < need) take_flags |= 1 << i;
        ++tie_rank;
      }
    long long pos = block_exclusive_scan(__popc(take_flags), wsum, &s_tot);
    const long long take_total = s_tot;
#pragma unroll
    for (int i = 0; i < SEL_COMPACT_ITEMS; ++i)
      if (take_flags & (1 << i)) {
        if (MODE == 1 || written + pos < ncand) {
          out_ids[base_out + written + pos] = (int32_t)(v0 + i);
          if (MODE == 0) out_keys[base_out + written + pos] = xs[i];
        }
        ++pos;
      }
    written += take_total;
    ties_seen += tie_total;
  }
  if (MODE == 0) {
    for (int64_t i = written + threadIdx.x; i < ncand; i += SEL_THREADS) {
      out_ids[base_out + i] = -1;
      out_keys[base_out + i] = 0;
    }
    if (threadIdx.x == 0) n_valid[q] = (int32_t)(written < ncand ? written : ncand);
  }
}

// ---------------------------------------------------------------------
// Refinement select split over P chunks of documents per query, so that a
// launch with few queries still fills the chip, and long F' rows are read by
// many workgroups (with 128 queries or more over fewer than 2^19 documents,
// k_select runs one workgroup per query instead).  A radix select on the order
// key u = fp_key(F') finds the ncand-th largest key T and how many documents
// with key T to keep (the lowest ids): bits 31..20 come from the walk's
// histogram, bits 19..8 and 7..0 from two histogram passes over the chunks
// (global atomics, only documents whose higher bits match count).  The middle
// pass reads F' and lists each chunk's documents at or above the 12-bit
// prefix, which the last pass reads instead of F'.  The last
// pass also records, per chunk, how many keys lie above the 24-bit prefix and
// the chunk's own histogram of the low 8 bits, so that once T is known every
// chunk's kept and tied counts follow without another pass; the counts are
// scanned per query, and each chunk that keeps documents writes its part of
// the candidate list in ascending doc order.
// SelState per query: the bins found so far, the count still to place, T and
// the ties to keep.
struct SelState {
  long long rem;     // candidates still to place below the bins fixed so far
  uint32_t prefix;   // key bits fixed so far
  uint32_t T;        // threshold key (0: keep every hit)
  long long need;    // documents with key T to keep
  long long total;   // candidates written
};
constexpr int SPLIT_THREADS = 256;

// Documents per chunk of the split select: a multiple of 16, so that chunks
// start 16-byte aligned within an F' row.
__host__ __device__ inline int64_t sel_chunk_docs(int64_t ndocs, int P) { return ((ndocs + P - 1) / P + 15) / 16 * 16; }


// Per query: bin of bits 31..20 from the walk's histogram; clears the
// histograms of the next passes.
__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_first(const uint32_t *__restrict__ hist1, int ncand,
                                                             uint32_t *__restrict__ hist2, uint32_t *__restrict__ hist3,
                                                             SelState *__restrict__ st) {
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot, s_above;
  __shared__ int s_bin;
  const int64_t q = blockIdx.x;
  const uint32_t *h = hist1 + q * SEL_BINS;
  long long local = 0;
  for (int i = threadIdx.x; i < SEL_BINS; i += SPLIT_THREADS) {
    local += h[i];
    hist2[q * SEL_BINS + i] = 0;
  }
  for (int i = threadIdx.x; i < 256; i += SPLIT_THREADS) hist3[q * 256 + i] = 0;
  block_exclusive_scan(local, wsum, &s_tot);
  const long long nhit = s_tot;
  if (nhit <= ncand) {
    if (threadIdx.x == 0) st[q] = SelState{0, 0, 0, 0, 0};
    return;
  }
  select_bin(h, SEL_BINS, ncand, wsum, &s_tot, &s_bin, &s_above);
  if (threadIdx.x == 0) st[q] = SelState{ncand - s_above, (uint32_t)s_bin, 1, 0, 0};
}

// Per query: the next bin from a pass's histogram; after the last pass, the
// threshold key T and the ties to keep.
template <int BITS, bool LAST>
__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_next(const uint32_t *__restrict__ hin, SelState *__restrict__ st) {
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot, s_above;
  __shared__ int s_bin;
  const int64_t q = blockIdx.x;
  const SelState s0 = st[q];
  if (s0.T == 0) return;
  select_bin(hin + q * (1 << BITS), 1 << BITS, s0.rem, wsum, &s_tot, &s_bin, &s_above);
  if (threadIdx.x == 0) {
    SelState s1 = s0;
    s1.prefix = (s0.prefix << BITS) | (uint32_t)s_bin;
    s1.rem = s0.rem - s_above;
    if (LAST) {
      s1.T = s1.prefix;
      s1.need = s1.rem;
    }
    st[q] = s1;
  }
}

// Last histogram pass over one chunk (bits 7..0 under the 24-bit prefix),
// over the middle pass's list of the chunk (or its F' when that list was not
// kept), plus the chunk's own record: chunk_hist [256] of those keys and
// chunk_above, the number of keys above the prefix (every hit when all are
// kept).
// The last histogram pass also lists, per chunk and in document order, the
// documents whose 24-bit key prefix reaches the bin being resolved (those
// above it and those in it), so that the write pass reads these lists
// instead of F' again.  A list longer than cap is not kept (the write pass
// then reads the chunk's F').
constexpr int SEL_LAST_ITEMS = 16;  // contiguous F' entries per thread and step
constexpr uint32_t SEL_NO_LIST = 0xFFFFFFFFu;

__host__ __device__ inline int sel_list_cap(int64_t ndocs, int P, int ncand) {
  const int64_t per = sel_chunk_docs(ndocs, P);
  return (int)std::min<int64_t>(per, 4 * ((int64_t)ncand / P) + 1024);
}

// The middle histogram pass over one chunk (bits 19..8 under the 12-bit
// prefix), which also lists, in document order, the chunk's documents whose
// top 12 key bits reach the prefix (those above the prefix's bin and those in
// it: every document the select can keep), so that the last pass reads these
// lists instead of F'.  A list longer than cap is not kept (clen = SEL_NO_LIST;
// the last pass then reads the chunk's F').
__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_mid(const int32_t *__restrict__ fp, int64_t ndocs, int P,
                                                           const SelState *__restrict__ st,
                                                           uint32_t *__restrict__ hout, int cap,
                                                           int2 *__restrict__ clist, uint32_t *__restrict__ clen) {
  __shared__ uint32_t h[SEL_BINS];
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot;
  const int64_t q = blockIdx.x / P;
  const int c = blockIdx.x % P;
  if (st[q].T == 0) return;  // uniform: every hit is kept
  const uint32_t prefix = st[q].prefix;
  for (int i = threadIdx.x; i < SEL_BINS; i += SPLIT_THREADS) h[i] = 0;
  __syncthreads();
  const int64_t per = sel_chunk_docs(ndocs, P), v0 = min(ndocs, c * per), v1 = min(ndocs, v0 + per);
  const int32_t *f = fp + q * ndocs;
  int2 *L = clist + ((int64_t)q * P + c) * cap;
  long long nlist = 0;  // uniform
  const int64_t step = (int64_t)SPLIT_THREADS * SEL_LAST_ITEMS;
  const bool vec = ((uintptr_t)f & 15) == 0 && (v0 & 3) == 0;
  for (int64_t vb = v0; vb < v1; vb += step) {
    const int64_t vt = vb + (int64_t)threadIdx.x * SEL_LAST_ITEMS;
    int32_t x[SEL_LAST_ITEMS];
    if (vec && vt + SEL_LAST_ITEMS <= v1) {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; i += 4) {
        const int4 y = *(const int4 *)(f + vt + i);
        x[i] = y.x;
        x[i + 1] = y.y;
        x[i + 2] = y.z;
        x[i + 3] = y.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; ++i) x[i] = vt + i < v1 ? f[vt + i] : NO_HIT;
    }
    int flags = 0;
#pragma unroll
    for (int i = 0; i < SEL_LAST_ITEMS; ++i) {
      if (x[i] == NO_HIT) continue;
      const uint32_t u = fp_key(x[i]);
      if ((u >> 20) > prefix) {
        flags |= 1 << i;
      } else if ((u >> 20) == prefix) {
        atomicAdd(&h[(u >> 8) & (SEL_BINS - 1)], 1u);
        flags |= 1 << i;
      }
    }
    long long pos = block_exclusive_scan(__popc(flags), wsum, &s_tot);
    const long long tot = s_tot;
#pragma unroll
    for (int i = 0; i < SEL_LAST_ITEMS; ++i)
      if (flags & (1 << i)) {
        if (nlist + pos < cap) L[nlist + pos] = make_int2((int)(vt + i), x[i]);
        ++pos;
      }
    nlist += tot;
  }
  __syncthreads();
  uint32_t *o = hout + q * SEL_BINS;
  for (int i = threadIdx.x; i < SEL_BINS; i += SPLIT_THREADS)
    if (h[i]) atomicAdd(&o[i], h[i]);
  if (threadIdx.x == 0) clen[(int64_t)q * P + c] = nlist <= cap ? (uint32_t)nlist : SEL_NO_LIST;
}

__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_last(const int32_t *__restrict__ fp, int64_t ndocs, int P,
                                                            const SelState *__restrict__ st,
                                                            uint32_t *__restrict__ hout,
                                                            uint32_t *__restrict__ chunk_hist,
                                                            uint32_t *__restrict__ chunk_above, int cap,
                                                            const int2 *__restrict__ mlist,
                                                            const uint32_t *__restrict__ mlen,
                                                            int2 *__restrict__ clist, uint32_t *__restrict__ clen) {
  __shared__ uint32_t h[256];
  __shared__ uint32_t s_above;
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot;
  const int64_t q = blockIdx.x / P;
  const int c = blockIdx.x % P;
  const bool all = st[q].T == 0;  // uniform: every hit is kept (no list: the write pass reads F')
  const uint32_t prefix = st[q].prefix;
  for (int i = threadIdx.x; i < 256; i += SPLIT_THREADS) h[i] = 0;
  if (threadIdx.x == 0) s_above = 0;
  __syncthreads();
  const int64_t per = sel_chunk_docs(ndocs, P), v0 = min(ndocs, c * per), v1 = min(ndocs, v0 + per);
  const int32_t *f = fp + q * ndocs;
  int2 *L = clist + ((int64_t)q * P + c) * cap;
  uint32_t above = 0;
  long long nlist = 0;  // uniform
  const int64_t step = (int64_t)SPLIT_THREADS * SEL_LAST_ITEMS;
  // the middle pass's list of the chunk (documents with the 12-bit prefix or
  // above, with their F'), when it kept one; else F' itself
  const uint32_t ml = all ? SEL_NO_LIST : mlen[(int64_t)q * P + c];
  const bool from_list = ml != SEL_NO_LIST;  // uniform
  const int2 *M = mlist + ((int64_t)q * P + c) * cap;
  const int64_t b0 = from_list ? 0 : v0, b1 = from_list ? (int64_t)ml : v1;
  // 16-byte loads where the row allows it (every F' row starts 16-byte
  // aligned when ndocs is a multiple of 4, and chunks start at multiples of 16)
  const bool vec = !from_list && ((uintptr_t)f & 15) == 0 && (v0 & 3) == 0;
  for (int64_t vb = b0; vb < b1; vb += step) {
    const int64_t vt = vb + (int64_t)threadIdx.x * SEL_LAST_ITEMS;
    int32_t x[SEL_LAST_ITEMS], d[SEL_LAST_ITEMS];
    if (from_list) {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; ++i) {
        const int2 e = vt + i < b1 ? M[vt + i] : make_int2(0, NO_HIT);
        d[i] = e.x;
        x[i] = e.y;
      }
    } else if (vec && vt + SEL_LAST_ITEMS <= v1) {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; i += 4) {
        const int4 y = *(const int4 *)(f + vt + i);
        x[i] = y.x;
        x[i + 1] = y.y;
        x[i + 2] = y.z;
        x[i + 3] = y.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; ++i) x[i] = vt + i < v1 ? f[vt + i] : NO_HIT;
    }
    if (!from_list) {
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; ++i) d[i] = (int)(vt + i);
    }
    int flags = 0;
#pragma unroll
    for (int i = 0; i < SEL_LAST_ITEMS; ++i) {
      if (x[i] == NO_HIT) continue;
      const uint32_t u = fp_key(x[i]);
      if (all || (u >> 8) > prefix) {
        ++above;
        flags |= 1 << i;
      } else if ((u >> 8) == prefix) {
        atomicAdd(&h[u & 255u], 1u);
        flags |= 1 << i;
      }
    }
    if (!all) {
      long long pos = block_exclusive_scan(__popc(flags), wsum, &s_tot);
      const long long tot = s_tot;
#pragma unroll
      for (int i = 0; i < SEL_LAST_ITEMS; ++i)
        if (flags & (1 << i)) {
          if (nlist + pos < cap) L[nlist + pos] = make_int2(d[i], x[i]);
          ++pos;
        }
      nlist += tot;
    }
  }
  atomicAdd(&s_above, above);
  __syncthreads();
  uint32_t *o = hout + q * 256, *ch = chunk_hist + ((int64_t)q * P + c) * 256;
  for (int i = threadIdx.x; i < 256; i += SPLIT_THREADS) {
    ch[i] = h[i];
    if (h[i]) atomicAdd(&o[i], h[i]);
  }
  if (threadIdx.x == 0) {
    chunk_above[(int64_t)q * P + c] = s_above;
    clen[(int64_t)q * P + c] = !all && nlist <= cap ? (uint32_t)nlist : SEL_NO_LIST;
  }
}

// Per query: every chunk's kept (key > T) and tied (key == T) counts from its
// record, then (in order) its output offset, ties before it and the number it
// keeps [3 per chunk], the number of candidates, and the padding of the
// unused slots.
__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_scan(int P, int ncand, SelState *__restrict__ st,
                                                            const uint32_t *__restrict__ chunk_hist,
                                                            const uint32_t *__restrict__ chunk_above,
                                                            long long *__restrict__ counts, int32_t *__restrict__ out_ids,
                                                            int32_t *__restrict__ out_keys,
                                                            int32_t *__restrict__ n_valid) {
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot;
  const int64_t q = blockIdx.x;
  const uint32_t T = st[q].T;
  const long long need = st[q].need;
  const int b3 = (int)(T & 255u);
  // thread t owns chunks [c0, c1): two block scans (ties before each chunk,
  // then output offsets) instead of one thread walking every chunk
  const int per = (P + SPLIT_THREADS - 1) / SPLIT_THREADS;
  const int c0 = min(P, (int)threadIdx.x * per), c1 = min(P, c0 + per);
  long long my_ties = 0;
  for (int c = c0; c < c1; ++c) {
    const uint32_t *ch = chunk_hist + ((int64_t)q * P + c) * 256;
    long long above = chunk_above[(int64_t)q * P + c], ties = 0;
    if (T != 0) {
      for (int b = b3 + 1; b < 256; ++b) above += ch[b];
      ties = ch[b3];
    }
    counts[3 * (q * P + c)] = above;
    counts[3 * (q * P + c) + 1] = ties;
    my_ties += ties;
  }
  long long tb = block_exclusive_scan(my_ties, wsum, &s_tot);
  long long my_take = 0;
  for (int c = c0; c < c1; ++c) {
    long long *cc = counts + 3 * (q * P + c);
    const long long a = cc[0], t = cc[1];
    const long long take = a + max(0ll, min(t, need - tb));
    cc[1] = tb;
    cc[2] = take;
    tb += t;
    my_take += take;
  }
  long long off = block_exclusive_scan(my_take, wsum, &s_tot);
  const long long n = min(s_tot, (long long)ncand);
  for (int c = c0; c < c1; ++c) {
    long long *cc = counts + 3 * (q * P + c);
    cc[0] = off;
    off += cc[2];
  }
  if (threadIdx.x == 0) {
    st[q].total = n;
    n_valid[q] = (int32_t)n;
  }
  for (long long i = n + threadIdx.x; i < ncand; i += SPLIT_THREADS) {
    out_ids[q * ncand + i] = -1;
    out_keys[q * ncand + i] = 0;
  }
}

// Per chunk: the ordered compaction of its kept documents, from the chunk's
// list when the last pass kept one, else from F'.
__global__ __launch_bounds__(SPLIT_THREADS) void k_sel_write(const int32_t *__restrict__ fp, int64_t ndocs, int P,
                                                             int ncand, const SelState *__restrict__ st,
                                                             const long long *__restrict__ counts, int cap,
                                                             const int2 *__restrict__ clist,
                                                             const uint32_t *__restrict__ clen,
                                                             int32_t *__restrict__ out_ids,
                                                             int32_t *__restrict__ out_keys) {
  __shared__ long long wsum[SPLIT_THREADS / 64];
  __shared__ long long s_tot;
  const int64_t q = blockIdx.x / P;
  const int c = blockIdx.x % P;
  const uint32_t T = st[q].T;
  const long long need = st[q].need;
  const long long *cc = counts + 3 * (q * P + c);
  if (cc[2] == 0 || cc[0] >= ncand) return;  // uniform: the chunk keeps nothing that fits
  long long written = cc[0], ties_seen = cc[1];
  const uint32_t nl = clen[q * P + c];
  const bool from_list = nl != SEL_NO_LIST;  // uniform
  const int2 *L = clist + (q * P + c) * (int64_t)cap;
  const int64_t per = sel_chunk_docs(ndocs, P), vb = min(ndocs, c * per), ve = min(ndocs, vb + per);
  const int64_t b0 = from_list ? 0 : vb, b1 = from_list ? (int64_t)nl : ve;
  const int32_t *f = fp + q * ndocs;
  const int64_t step = (int64_t)SPLIT_THREADS * SEL_ITEMS;
  for (int64_t c0 = b0; c0 < b1; c0 += step) {
    const int64_t j0 = c0 + (int64_t)threadIdx.x * SEL_ITEMS;
    int take_flags = 0, tie_flags = 0, ntie = 0;
    int32_t xs[SEL_ITEMS], vs[SEL_ITEMS];
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i) {
      const int64_t j = j0 + i;
      if (from_list) {
        const int2 e = j < b1 ? L[j] : make_int2(-1, NO_HIT);
        vs[i] = e.x;
        xs[i] = e.y;
      } else {
        vs[i] = (int32_t)j;
        xs[i] = j < b1 ? f[j] : NO_HIT;
      }
      if (xs[i] != NO_HIT) {
        const uint32_t u = fp_key(xs[i]);
        if (u > T) take_flags |= 1 << i;
        else if (u == T) { tie_flags |= 1 << i; ++ntie; }
      }
    }
    long long tie_rank = block_exclusive_scan(ntie, wsum, &s_tot);
    const long long tie_total = s_tot;
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i)
      if (tie_flags & (1 << i)) {
        if (ties_seen + tie_rank < need) take_flags |= 1 << i;
        ++tie_rank;
      }
    long long pos = block_exclusive_scan(__popc(take_flags), wsum, &s_tot);
    const long long take_total = s_tot;
#pragma unroll
    for (int i = 0; i < SEL_ITEMS; ++i)
      if (take_flags & (1 << i)) {
        if (written + pos < ncand) {
          out_ids[q * ncand + written + pos] = vs[i];
          out_keys[q * ncand + written + pos] = xs[i];
        }
        ++pos;
      }
    written += take_total;
    ties_seen += tie_total;
  }
}

// Chunks per query of the split select: about 16384 workgroups over the
// batch (measured at 8.8M: 34 ms per step against 55 ms for 2048), each
// chunk at least 4096 documents.
int select_chunks(int64_t nq, int64_t ndocs) {
  const int64_t by_q = (16384 + nq - 1) / std::max<int64_t>(1, nq);
  const int64_t by_docs = (ndocs + 4095) / 4096;
  return (int)std::max<int64_t>(1, std::min(by_q, by_docs));
}

size_t select_scratch_bytes(int64_t nq, int64_t ndocs, int ncand) {
  const int P = select_chunks(nq, ndocs);
  const size_t cap = (size_t)sel_list_cap(ndocs, P, ncand);
  return (size_t)nq * (sizeof(SelState) + (SEL_BINS + 256) * 4 + (size_t)P * (24 + 256 * 4 + 4 + 4 + cap * 8)) +
         (size_t)nq * P * (4 + cap * 8) + 1024;
}

void launch_select(const int32_t *fp, const uint32_t *hist, int64_t nq, int64_t ndocs, int ncand, void *scratch,
                   int32_t *cand_ids, int32_t *cand_keys, int32_t *n_valid, hipStream_t s) {
  if (nq <= 0) return;
  if (nq >= 128 && ndocs < (1 << 19)) {
    // enough queries to fill the chip with one workgroup each, over short
    // enough F' rows (one launch; measured faster than the split passes at
    // 100k documents, slower at 1M)
    hipLaunchKernelGGL((k_select<0>), dim3((unsigned)nq), dim3(SEL_THREADS), 0, s, fp, hist, ndocs, ncand,
                       (const int64_t *)nullptr, cand_ids, cand_keys, n_valid);
    return;
  }
  const int P = select_chunks(nq, ndocs);
  SelState *st = (SelState *)scratch;
  uint32_t *hist2 = (uint32_t *)(st + nq);
  uint32_t *hist3 = hist2 + nq * SEL_BINS;
  long long *counts = (long long *)(((uintptr_t)(hist3 + nq * 256) + 15) & ~(uintptr_t)15);
  uint32_t *chunk_hist = (uint32_t *)(counts + 3 * nq * P);
  uint32_t *chunk_above = chunk_hist + (size_t)nq * P * 256;
  uint32_t *clen = chunk_above + (size_t)nq * P;
  const int cap = sel_list_cap(ndocs, P, ncand);
  int2 *clist = (int2 *)(((uintptr_t)(clen + (size_t)nq * P) + 15) & ~(uintptr_t)15);
  uint32_t *mlen = (uint32_t *)(clist + (size_t)nq * P * cap);
  int2 *mlist = (int2 *)(((uintptr_t)(mlen + (size_t)nq * P) + 15) & ~(uintptr_t)15);
  const dim3 gq((unsigned)nq), gc((unsigned)(nq * P)), tb(SPLIT_THREADS);
  hipLaunchKernelGGL(k_sel_first, gq, tb, 0, s, hist, ncand, hist2, hist3, st);
  hipLaunchKernelGGL(k_sel_mid, gc, tb, 0, s, fp, ndocs, P, st, hist2, cap, mlist, mlen);
  hipLaunchKernelGGL((k_sel_next<12, false>), gq, tb, 0, s, hist2, st);
  hipLaunchKernelGGL(k_sel_last, gc, tb, 0, s, fp, ndocs, P, st, hist3, chunk_hist, chunk_above, cap, mlist, mlen,
                     clist, clen);
  hipLaunchKernelGGL((k_sel_next<8, true>), gq, tb, 0, s, hist3, st);
  hipLaunchKernelGGL(k_sel_scan, gq, tb, 0, s, P, ncand, st, chunk_hist, chunk_above, counts, cand_ids, cand_keys,
                     n_valid);
  hipLaunchKernelGGL(k_sel_write, gc, tb, 0, s, fp, ndocs, P, ncand, st, counts, cap, clist, clen, cand_ids,
                     cand_keys);
}

__global__ __launch_bounds__(256) void k_count_hits(const int32_t *__restrict__ fp, int64_t ndocs,
                                                    int64_t *__restrict__ counts) {
  __shared__ unsigned long long acc;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  const int32_t *f = fp + (int64_t)blockIdx.x * ndocs;
  unsigned long long local = 0;
  for (int64_t v = threadIdx.x; v < ndocs; v += 256) local += f[v] != NO_HIT;
  atomicAdd(&acc, local);
  __syncthreads();
  if (threadIdx.x == 0) counts[blockIdx.x] = (int64_t)acc;
}

void launch_count_hits(const int32_t *fp, int64_t nq, int64_t ndocs, int64_t *counts, hipStream_t s) {
  hipLaunchKernelGGL(k_count_hits, dim3((unsigned)nq), dim3(256), 0, s, fp, ndocs, counts);
}

void launch_list_hits(const int32_t *fp, int64_t nq, int64_t ndocs, const int64_t *offsets, int32_t *doc_ids,
                      hipStream_t s) {
  hipLaunchKernelGGL((k_select<1>), dim3((unsigned)nq), dim3(SEL_THREADS), 0, s, fp, (const uint32_t *)nullptr, ndocs,
                     0, offsets, doc_ids, (int32_t *)nullptr, (int32_t *)nullptr);
}

}  // namespace chimera
