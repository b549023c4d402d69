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
__device__ __forceinline__ int32_t token_key(const uint8_t *__restrict__ codes, int32_t t, const uint32_t (&qv)[64],
                                             const uint32_t *lut, int32_t skey) {
  constexpr int CB = 16 * NBITS;
  const uint4 *cp = (const uint4 *)(codes + (int64_t)t * CB);
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < CB / 16; ++u) {
    const uint4 c4 = cp[u];
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

// A list walked by one lane: expected entries per range at most this.
constexpr int REF_LANE_ENTRIES = 32;

// Documents per range: the state m is TQP x RR int32, 64 KiB.
template <int TQP>
constexpr int ref_range_docs() { return 16384 / TQP; }

template <int NBITS, int TQP>
__global__ __launch_bounds__(REF_THREADS) void k_refine_walk(
    const int32_t *__restrict__ cent_ids, const int32_t *__restrict__ cent_keys, const uint16_t *__restrict__ Qs,
    int64_t nq, int Tq, int nprobe, const int64_t *__restrict__ tok_off, const int32_t *__restrict__ ivf_tok,
    const int32_t *__restrict__ tok_doc, const int64_t *__restrict__ doc_off, const uint8_t *__restrict__ codes,
    uint4 w_lo, uint4 w_hi, int64_t ndocs, int nranges, int G, int M, int32_t *__restrict__ fp,
    uint32_t *__restrict__ hist) {
  constexpr int RR = ref_range_docs<TQP>();
  static_assert(RR * TQP >= SEL_BINS, "the histogram reuses the state array");
  extern __shared__ __align__(16) unsigned char ref_lds[];
  int32_t *m = (int32_t *)ref_lds;                         // [TQP][RR]: query token major
  int32_t *sfp = m + RR * TQP;                             // [RR]
  uint32_t *lut = (uint32_t *)(sfp + RR);                  // [256][NBITS == 2 ? 2 : 1]
  RefList *L = (RefList *)(lut + 256 * (NBITS == 2 ? 2 : 1));  // [nprobe * Tq], list i = r * Tq + j
  int32_t *wide = (int32_t *)(L + nprobe * Tq);                 // [nprobe * Tq] lists walked by a wave
  int32_t &s_nwide = wide[nprobe * Tq];                         // their number
  // (all of it in the dynamic allocation: the launch asks for the whole LDS)

  const int b = blockIdx.x;
  const int64_t q = (b & 7) + 8 * (int64_t)((b >> 3) / G);
  const int g = (b >> 3) % G;
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
  if (threadIdx.x == 0) s_nwide = 0;
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
    for (int i = threadIdx.x; i < RR * TQP; i += REF_THREADS) m[i] = NO_HIT;
    __syncthreads();  // cursors, table and state ready; the previous range's reads done

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
      do {
        const int32_t tn = pos + 1 < len ? list[pos + 1] : INT32_MAX;  // next entry, loaded early
        const int32_t key = token_key<NBITS>(codes, t, qv, lut, skey);
        atomicMax(&m[j * RR + (tok_doc[t] - (int)d0)], key);
        ++pos;
        t = tn;
      } while (t < t1);
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
        if (in) atomicMax(&m[j * RR + (tok_doc[t] - (int)d0)], token_key<NBITS>(codes, t, qv, lut, skey));
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
    for (int v = threadIdx.x; v < nd; v += REF_THREADS) {
      int32_t s = 0;
      bool hit = false;
      for (int j = 0; j < Tq; ++j) {
        const int32_t x = m[j * RR + v];
        if (x != NO_HIT) {
          s += x;
          hit = true;
        }
      }
      sfp[v] = hit ? s : NO_HIT;
    }
    __syncthreads();
    uint32_t *sh = (uint32_t *)m;  // the state is no longer needed
    for (int i = threadIdx.x; i < SEL_BINS; i += REF_THREADS) sh[i] = 0;
    __syncthreads();
    int32_t *f = fp + q * ndocs + d0;
    for (int v = threadIdx.x; v < nd; v += REF_THREADS) {
      const int32_t x = sfp[v];
      f[v] = x;
      if (x != NO_HIT) atomicAdd(&sh[fp_key(x) >> 20], 1u);
    }
    __syncthreads();
    uint32_t *hq = hist + q * SEL_BINS;
    for (int i = threadIdx.x; i < SEL_BINS; i += REF_THREADS)
      if (sh[i]) atomicAdd(&hq[i], sh[i]);
    __syncthreads();  // sh (the state array) is reset by the next range
  }
}

size_t refine_lds_bytes(int TQP, int nprobe, int Tq) {
  const size_t RR = 16384 / TQP;
  return RR * TQP * 4 + RR * 4 + 256 * 8 + (size_t)nprobe * Tq * (sizeof(RefList) + 4) + 4;
}

template <int NBITS, int TQP>
static void launch_refine_t(const int32_t *cent_ids, const int32_t *cent_keys, const uint16_t *Qs, int64_t nq, int Tq,
                            int nprobe, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                            const int64_t *doc_off, const uint8_t *codes, uint4 w_lo, uint4 w_hi, int64_t ndocs,
                            int32_t *fp, uint32_t *hist, hipStream_t s) {
  constexpr int RR = ref_range_docs<TQP>();
  const int nranges = (int)((ndocs + RR - 1) / RR);
  // ranges per workgroup: enough groups per query for about 4096 workgroups
  int G = (int)std::min<int64_t>(nranges, std::max<int64_t>(1, (4096 + nq - 1) / nq));
  const int M = (nranges + G - 1) / G;
  G = (nranges + M - 1) / M;
  const int64_t blocks = (nq + 7) / 8 * 8 * G;
  if (blocks == 0 || nranges == 0) return;
  const size_t lds = refine_lds_bytes(TQP, nprobe, Tq);
  static bool attr = [] {
    return hipFuncSetAttribute((const void *)k_refine_walk<NBITS, TQP>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               160 * 1024) == hipSuccess;
  }();
  (void)attr;
  hipLaunchKernelGGL((k_refine_walk<NBITS, TQP>), dim3((unsigned)blocks), dim3(REF_THREADS), lds, s, cent_ids,
                     cent_keys, Qs, nq, Tq, nprobe, tok_off, ivf_tok, tok_doc, doc_off, codes, w_lo, w_hi, ndocs,
                     nranges, G, M, fp, hist);
}

void launch_refine_walk(const int32_t *cent_ids, const int32_t *cent_keys, const uint16_t *Qs, int64_t nq, int Tq,
                        int TQP, int nprobe, const int64_t *tok_off, const int32_t *ivf_tok, const int32_t *tok_doc,
                        const int64_t *doc_off, const uint8_t *codes, int nbits, const uint16_t *weights_host,
                        int64_t ndocs, int32_t *fp, uint32_t *hist, hipStream_t s) {
  uint32_t w[8] = {0};
  const int B = 1 << nbits;
  for (int u = 0; u < B; ++u) w[u >> 1] |= (uint32_t)weights_host[u] << (16 * (u & 1));
  const uint4 w_lo = make_uint4(w[0], w[1], w[2], w[3]), w_hi = make_uint4(w[4], w[5], w[6], w[7]);
#define CHIMERA_RF(NB, TP)                                                                                       \
  launch_refine_t<NB, TP>(cent_ids, cent_keys, Qs, nq, Tq, nprobe, tok_off, ivf_tok, tok_doc, doc_off, codes, \
                          w_lo, w_hi, ndocs, fp, hist, s)
  if (nbits == 2 && TQP == 32) CHIMERA_RF(2, 32);
  else if (nbits == 2) CHIMERA_RF(2, 64);
  else if (TQP == 32) CHIMERA_RF(4, 32);
  else CHIMERA_RF(4, 64);
#undef CHIMERA_RF
}

}  // namespace chimera
