// k_refine.hip - candidate refinement from the retrieved tokens' own scores.
//
// Sec. 3.2 (candidate refinement, Alg. 2) estimates a document's score from
// the tokens retrieved by candidate generation: per query token j, the
// maximum over the document's tokens that lie in one of j's probed lists of
// that token's approximate inner product with q_j, 0 if there is none, summed
// over query tokens.  Here a retrieved token t scores as document scoring
// scores it, S[j][cid t] + <q_j, w[codes t]> (centroid score plus decoded
// residual), so the estimate is exact on the tokens it sees; the paper uses
// 1-bit codes for the same purpose.
//
// Workgroup (query q, group of document ranges), like the centroid-only walk,
// but the state of a range is the maximum key of every (document, query
// token), LDS `m[j][v]`, since a decoded score is not decided by the rank of
// its list.  Every probed list (j, r) is token-level (ascending token ids,
// hence ascending documents) with a cursor that only moves forward; all lists
// are walked in any order (maxima commute).  A list expected to hold at most
// 32 entries per range is walked by one lane (one list per thread, so the
// lists' memory latencies overlap, and q_j stays in that lane's registers
// across ranges); longer lists are walked by a whole wave, one entry per
// lane.  Per entry the lane decodes the token's code bytes through the
// byte-indexed weight table and takes the dot product with q_j two
// dimensions at a time (v_dot2 on bf16 pairs; on the value grid every product
// and partial sum is an exact fp32 value, so the key is exact), then one LDS
// atomic max.  The range then sums
// its rows into F' (or NO_HIT), writes them, and adds its histogram of the top
// 12 key bits, the same outputs as the centroid-only walk, so the select,
// document scoring and top-k that follow are shared.
#include <algorithm>
#include <climits>

#include "device_common.h"
#include "internal.h"

namespace chimera {

constexpr int REF_THREADS = 256;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// Cursor on probed list (query token j, rank r): tokens ivf_tok[beg .. beg +
// len), position pos, the token there (INT32_MAX past the end) and S[j][c].
struct RefList {
  int64_t beg;
  int32_t len, pos, next, skey;
};

// Key of token t for query token j: S[j][c] + <q_j, w[codes t]>, q_j as 64
// bf16 pairs (dimensions 2i, 2i+1 in word i).
template <int NBITS>
__device__ __forceinline__ int32_t key_of_code(const uint4 (&cc)[NBITS], const uint32_t (&qv)[64],
                                               const uint32_t *lut, int32_t skey) {
  constexpr int CB = 16 * NBITS;
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < CB / 16; ++u) {
    const uint4 c4 = cc[u];
    const uint32_t cw[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const uint32_t byte = (cw[k >> 2] >> (8 * (k & 3))) & 255u;
      const int bi = 16 * u + k;  // code byte index
      if (NBITS == 2) {
        // byte bi holds dimensions 4bi .. 4bi+3: q pairs 2bi, 2bi+1
        const uint2 wv = *(const uint2 *)&lut[2 * byte];
        acc = dot2(wv.x, qv[2 * bi], acc);
        acc = dot2(wv.y, qv[2 * bi + 1], acc);
      } else {
        // byte bi holds dimensions 2bi, 2bi+1: q pair bi
        acc = dot2(lut[byte], qv[bi], acc);
      }
    }
  }
  return skey + to_key(acc);
}

template <int NBITS>
__device__ __forceinline__ void load_code(const uint8_t *__restrict__ codes, int32_t t, uint4 (&cc)[NBITS]) {
  const uint4 *cp = (const uint4 *)(codes + (int64_t)t * (16 * NBITS));
#pragma unroll
  for (int u = 0; u < NBITS; ++u) cc[u] = cp[u];
}

template <int NBITS>
__device__ __forceinline__ int32_t token_key(const uint8_t *__restrict__ codes, int32_t t, const uint32_t (&qv)[64],
                                             const uint32_t *lut, int32_t skey) {
  uint4 cc[NBITS];
  load_code<NBITS>(codes, t, cc);
  return key_of_code<NBITS>(cc, qv, lut, skey);
}

// A list walked by one lane: expected entries per range at most this.
constexpr int REF_LANE_ENTRIES = 32;
// Entries of a lane's list handled together.
constexpr int REF_BATCH = 2;

// Documents per range: the state m is TQP x RR int32, 32 KiB.
template <int TQP>
constexpr int ref_range_docs() { return 8192 / TQP; }

// (document, query token) entries a range records for its sweep; beyond this
// the range sweeps its whole state instead.
constexpr int REF_TOUCH_CAP = 2048;

// m[idx] = max(m[idx], key); the first update of an entry (which holds NO_HIT
// between ranges) records idx.
__device__ __forceinline__ void ref_update(int32_t *m, int32_t *tl, int32_t *ntl, int idx, int32_t key) {
  if (atomicMax(&m[idx], key) == NO_HIT) {
    const int slot = atomicAdd(ntl, 1);
    if (slot < REF_TOUCH_CAP) tl[slot] = idx;
  }
}

template <int NBITS, int TQP>
__global__ __launch_bounds__(REF_THREADS) void k_refine_walk(
    const int32_t *__restrict__ cent_ids, const int32_t *__restrict__ cent_keys, const uint16_t *__restrict__ Qs,
    int64_t nq, int Tq, int nprobe, const int64_t *__restrict__ tok_off, const int32_t *__restrict__ ivf_tok,
    const int32_t *__restrict__ tok_doc, const int64_t *__restrict__ doc_off, const uint8_t *__restrict__ codes,
    uint4 w_lo, uint4 w_hi, int64_t ndocs, const uint64_t *__restrict__ deleted, int nranges, int G, int M,
    int32_t *__restrict__ fp, uint32_t *__restrict__ hist) {
  constexpr int RR = ref_range_docs<TQP>();
  static_assert((RR & (RR - 1)) == 0 && RR % 32 == 0, "ranges of a power of two documents");
  extern __shared__ __align__(16) unsigned char ref_lds[];
  int32_t *m = (int32_t *)ref_lds;                         // [TQP][RR] query token major, NO_HIT between ranges
  uint32_t *hsh = (uint32_t *)(m + RR * TQP);              // [SEL_BINS] the group's histogram
  int32_t *tl = (int32_t *)(hsh + SEL_BINS);               // [REF_TOUCH_CAP] entries updated in the range
  int32_t *sfp = tl + REF_TOUCH_CAP;                       // [RR] F' being summed
  uint32_t *hitw = (uint32_t *)(sfp + RR);                 // [RR / 32] documents hit in the range
  uint32_t *lut = hitw + RR / 32;                          // [256][NBITS == 2 ? 2 : 1]
  RefList *L = (RefList *)(lut + 512);                     // [nprobe * Tq], list i = r * Tq + j
  int32_t *wide = (int32_t *)(L + nprobe * Tq);            // [nprobe * Tq] lists walked by a wave
  int32_t &s_nwide = wide[nprobe * Tq];                    // their number
  int32_t &s_ntl = wide[nprobe * Tq + 1];                  // entries recorded in tl
  // (all of it in the dynamic allocation: the launch asks for the whole LDS)

  // workgroup b runs on XCD b % 8: with 8 or more queries, the groups of
  // query q run on XCD q % 8; fewer queries spread over every XCD
  const int b = blockIdx.x;
  const int64_t q = nq >= 8 ? (b & 7) + 8 * (int64_t)((b >> 3) / G) : b / G;
  const int g = nq >= 8 ? (b >> 3) % G : b % G;
  if (q >= nq) return;
  const int rg0 = g * M, rg1 = min(nranges, rg0 + M);
  if (rg0 >= rg1) return;  // uniform, before any barrier
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nwaves = REF_THREADS / 64;

  // byte -> bf16 weights of its dimensions (2-bit: 4, in two bf16 pairs;
  // 4-bit: 2, one pair)
  {
    const uint16_t w[16] = {
        (uint16_t)w_lo.x, (uint16_t)(w_lo.x >> 16), (uint16_t)w_lo.y, (uint16_t)(w_lo.y >> 16),
        (uint16_t)w_lo.z, (uint16_t)(w_lo.z >> 16), (uint16_t)w_lo.w, (uint16_t)(w_lo.w >> 16),
        (uint16_t)w_hi.x, (uint16_t)(w_hi.x >> 16), (uint16_t)w_hi.y, (uint16_t)(w_hi.y >> 16),
        (uint16_t)w_hi.z, (uint16_t)(w_hi.z >> 16), (uint16_t)w_hi.w, (uint16_t)(w_hi.w >> 16)};
    const int e = threadIdx.x;  // 256 threads, one table entry each
    if (NBITS == 2) {
      lut[2 * e] = (uint32_t)w[e & 3] | ((uint32_t)w[(e >> 2) & 3] << 16);
      lut[2 * e + 1] = (uint32_t)w[(e >> 4) & 3] | ((uint32_t)w[(e >> 6) & 3] << 16);
    } else {
      lut[e] = (uint32_t)w[e & 15] | ((uint32_t)w[e >> 4] << 16);
    }
  }
  // list cursors, positioned at the group's first token
  const int nl = nprobe * Tq;
  if (threadIdx.x == 0) {
    s_nwide = 0;
    s_ntl = 0;
  }
  for (int i = threadIdx.x; i < RR * TQP; i += REF_THREADS) m[i] = NO_HIT;
  for (int i = threadIdx.x; i < SEL_BINS; i += REF_THREADS) hsh[i] = 0;
  for (int i = threadIdx.x; i < RR; i += REF_THREADS) sfp[i] = 0;
  for (int i = threadIdx.x; i < RR / 32; i += REF_THREADS) hitw[i] = 0;
  __syncthreads();
  const int64_t tstart = doc_off[(int64_t)rg0 * RR];
  for (int i = threadIdx.x; i < nl; i += REF_THREADS) {
    const int r = i / Tq, j = i - r * Tq;
    const int64_t e = (q * TQP + j) * nprobe + r;
    const int32_t c = cent_ids[e];
    const int64_t beg = tok_off[c], end = tok_off[c + 1];
    const int64_t p = tstart > 0 ? lower_bound_i32(ivf_tok, beg, end, tstart) : beg;
    RefList w;
    w.beg = beg;
    w.len = (int32_t)(end - beg);
    w.pos = (int32_t)(p - beg);
    w.next = w.pos < w.len ? ivf_tok[p] : INT32_MAX;
    w.skey = cent_keys[e];
    if ((int64_t)w.len * RR > (int64_t)REF_LANE_ENTRIES * ndocs) {
      wide[atomicAdd(&s_nwide, 1)] = i;
      w.len = -w.len;  // marks a list walked by a wave
    }
    L[i] = w;
  }
  int32_t qj = -1;  // the query token whose q this thread holds
  uint32_t qv[64];

  for (int rg = rg0; rg < rg1; ++rg) {
    const int64_t d0 = (int64_t)rg * RR;
    const int64_t d1 = min(ndocs, d0 + RR);
    const int nd = (int)(d1 - d0);
    const int64_t t1 = doc_off[d1];  // tokens of the range: [doc_off[d0], t1)
    __syncthreads();  // cursors, table and state ready; the previous range's resets done

    // lists walked by one lane each
    for (int i = threadIdx.x; i < nl; i += REF_THREADS) {
      RefList *w = &L[i];
      int32_t t = w->next;
      if (t >= t1 || w->len < 0) continue;
      const int j = i % Tq;
      if (j != qj) {
        const uint4 *qp = (const uint4 *)(Qs + (q * TQP + j) * 128);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const uint4 x = qp[k];
          qv[4 * k] = x.x; qv[4 * k + 1] = x.y; qv[4 * k + 2] = x.z; qv[4 * k + 3] = x.w;
        }
        qj = j;
      }
      const int32_t len = w->len, skey = w->skey;
      const int32_t *list = ivf_tok + w->beg;
      int32_t pos = w->pos;
      // REF_BATCH entries at a time: their ids, then their codes and
      // documents, are loaded together (the entries ascend, so those inside
      // the range are a prefix; the others load entry pos's data and are
      // dropped)
      for (;;) {
        int32_t tt[REF_BATCH + 1];
        tt[0] = t;
#pragma unroll
        for (int u = 1; u <= REF_BATCH; ++u) tt[u] = pos + u < len ? list[pos + u] : INT32_MAX;
        uint4 cc[REF_BATCH][NBITS];
        int32_t key[REF_BATCH], doc[REF_BATCH];
#pragma unroll
        for (int u = 0; u < REF_BATCH; ++u) {
          const int32_t tu = tt[u] < t1 ? tt[u] : t;
          load_code<NBITS>(codes, tu, cc[u]);
          doc[u] = tok_doc[tu];
        }
#pragma unroll
        for (int u = 0; u < REF_BATCH; ++u) {
          __builtin_amdgcn_sched_barrier(0);  // one entry's products at a time
          key[u] = key_of_code<NBITS>(cc[u], qv, lut, skey);
        }
        int n = 0;
#pragma unroll
        for (int u = 0; u < REF_BATCH; ++u)
          if (tt[u] < t1) {
            ref_update(m, tl, &s_ntl, j * RR + (doc[u] - (int)d0), key[u]);
            n = u + 1;
          }
        pos += n;
        t = tt[n];
        if (n < REF_BATCH || t >= t1) break;
      }
      w->pos = pos;
      w->next = t;
    }
    // lists walked by a whole wave, one entry per lane
    const int nwide = s_nwide;
    for (int wi = wave; wi < nwide; wi += nwaves) {
      const int i = wide[wi];
      RefList *w = &L[i];
      if (w->next >= t1) continue;  // wave-uniform: nothing of this list in the range
      const int j = i % Tq;
      const int32_t len = -w->len, skey = w->skey;
      const int32_t *list = ivf_tok + w->beg;
      {  // q_j into the lane's q registers (their cached token is dropped)
        const uint4 *qp = (const uint4 *)(Qs + (q * TQP + j) * 128);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const uint4 x = qp[k];
          qv[4 * k] = x.x; qv[4 * k + 1] = x.y; qv[4 * k + 2] = x.z; qv[4 * k + 3] = x.w;
        }
        qj = -1;
      }
      int32_t pos = w->pos, next = INT32_MAX;
      for (;;) {
        const int32_t p = pos + lane;
        const int32_t t = p < len ? list[p] : INT32_MAX;
        const bool in = t < t1;
        if (in) ref_update(m, tl, &s_ntl, j * RR + (tok_doc[t] - (int)d0), token_key<NBITS>(codes, t, qv, lut, skey));
        const unsigned long long out = __ballot(!in);
        if (out) {
          const int first = __ffsll((long long)out) - 1;
          next = __shfl(t, first, 64);
          pos += first;
          break;
        }
        pos += 64;
      }
      if (lane == 0) {
        w->pos = pos;
        w->next = next;
      }
    }
    __syncthreads();
    // sum the updated entries into F' and put them back to NO_HIT
    const int ntl = s_ntl;  // uniform
    auto take = [&](int idx) {
      const int32_t x = m[idx];
      m[idx] = NO_HIT;
      const int v = idx & (RR - 1);
      atomicAdd(&sfp[v], x);
      atomicOr(&hitw[v >> 5], 1u << (v & 31));
    };
    if (ntl <= REF_TOUCH_CAP) {
      for (int e = threadIdx.x; e < ntl; e += REF_THREADS) take(tl[e]);
    } else {
      for (int idx = threadIdx.x; idx < Tq * RR; idx += REF_THREADS)
        if (m[idx] != NO_HIT) take(idx);
    }
    __syncthreads();
    int32_t *f = fp + q * ndocs + d0;
    for (int v = threadIdx.x; v < nd; v += REF_THREADS) {
      // deleted documents get NO_HIT
      const bool hit = ((hitw[v >> 5] >> (v & 31)) & 1u) &&
                       !(deleted && ((deleted[(d0 + v) >> 6] >> ((d0 + v) & 63)) & 1));
      const int32_t x = hit ? sfp[v] : NO_HIT;
      f[v] = x;
      sfp[v] = 0;
      if (hit) atomicAdd(&hsh[fp_key(x) >> 20], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < RR / 32; i += REF_THREADS) hitw[i] = 0;
    if (threadIdx.x == 0) s_ntl = 0;
  }
  __syncthreads();
  uint32_t *hq = hist + q * SEL_BINS;
  for (int i = threadIdx.x; i < SEL_BINS; i += REF_THREADS)
    if (hsh[i]) atomicAdd(&hq[i], hsh[i]);
}

size_t refine_lds_bytes(int TQP, int nprobe, int Tq) {
  const size_t RR = 8192 / TQP;
  return RR * TQP * 4 + SEL_BINS * 4 + REF_TOUCH_CAP * 4 + RR * 4 + RR / 8 + 512 * 4 +
         (size_t)nprobe * Tq * (sizeof(RefList) + 4) + 8;
}

template <int NBITS, int TQP>
static void launch_refine_t(const int32_t *cent_ids, const int32_t *cent_keys, const uint16_t *Qs, int64_t nq, int Tq,
                            int nprobe, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                            const int64_t *doc_off, const uint8_t *codes, uint4 w_lo, uint4 w_hi, int64_t ndocs,
                            const uint64_t *deleted, int32_t *fp, uint32_t *hist, hipStream_t s) {
  constexpr int RR = ref_range_docs<TQP>();
  const int nranges = (int)((ndocs + RR - 1) / RR);
  // ranges per workgroup: enough groups per query for about 4096 workgroups
  int G = (int)std::min<int64_t>(nranges, std::max<int64_t>(1, (4096 + nq - 1) / nq));
  const int M = (nranges + G - 1) / G;
  G = (nranges + M - 1) / M;
  const int64_t blocks = (nq >= 8 ? (nq + 7) / 8 * 8 : nq) * G;
  if (blocks == 0 || nranges == 0) return;
  const size_t lds = refine_lds_bytes(TQP, nprobe, Tq);
  static bool attr = [] {
    return hipFuncSetAttribute((const void *)k_refine_walk<NBITS, TQP>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               160 * 1024) == hipSuccess;
  }();
  (void)attr;
  hipLaunchKernelGGL((k_refine_walk<NBITS, TQP>), dim3((unsigned)blocks), dim3(REF_THREADS), lds, s, cent_ids,
                     cent_keys, Qs, nq, Tq, nprobe, tok_off, ivf_tok, tok_doc, doc_off, codes, w_lo, w_hi, ndocs,
                     deleted, nranges, G, M, fp, hist);
}

void launch_refine_walk(const int32_t *cent_ids, const int32_t *cent_keys, const uint16_t *Qs, int64_t nq, int Tq,
                        int TQP, int nprobe, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                        const int64_t *doc_off, const uint8_t *codes, int nbits, const uint16_t *weights_host,
                        int64_t ndocs, const uint64_t *deleted, int32_t *fp, uint32_t *hist, hipStream_t s) {
  uint32_t w[8] = {0};
  const int B = 1 << nbits;
  for (int u = 0; u < B; ++u) w[u >> 1] |= (uint32_t)weights_host[u] << (16 * (u & 1));
  const uint4 w_lo = make_uint4(w[0], w[1], w[2], w[3]), w_hi = make_uint4(w[4], w[5], w[6], w[7]);
#define CHIMERA_RF(NB, TP)                                                                                       \
  launch_refine_t<NB, TP>(cent_ids, cent_keys, Qs, nq, Tq, nprobe, tok_off, ivf_tok, tok_doc, doc_off, codes, \
                          w_lo, w_hi, ndocs, deleted, fp, hist, s)
  if (nbits == 2 && TQP == 32) CHIMERA_RF(2, 32);
  else if (nbits == 2) CHIMERA_RF(2, 64);
  else if (TQP == 32) CHIMERA_RF(4, 32);
  else CHIMERA_RF(4, 64);
#undef CHIMERA_RF
}

}  // namespace chimera
