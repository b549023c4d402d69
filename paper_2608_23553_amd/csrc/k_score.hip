// k_score.hip - document scoring of the refined candidates and the final
// top-k (Sec. 3.2 document scoring: the complete score over all tokens of
// each survivor, on the GPU; Sec. 4.2 document score aggregation; Alg. 1,
// final topK).
//
// Token score of doc token t against query token j (Chamfer, Def. 1, on the
// decoded token c_cid(t) + w[code_t]):
//     s[j][t] = S[j][cid(t)] + sum_d Q_j[d] * w[code_t[d]]
// The first term is read from the per-query S^T table written by the probe;
// the second is a [16 doc tokens x 128] x [128 x Tq] bf16 MFMA product whose
// doc-token operand is decoded in registers from the packed codes through an
// LDS lookup table indexed by code byte (the bucket-weight counterpart of the
// LUT inner product of Sec. 4.1: one lookup yields 4 (2-bit) or 2 (4-bit)
// bf16 weights).  The S term enters as the MFMA accumulator's initial value.
// Each document's codes are one contiguous span (document-major layout), so
// every lane issues one 64- or 128-bit load per 16-token tile.  The maximum
// over the document's tokens stays in registers and the sum over query
// tokens is an integer sum of exact keys.
#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

// 16x16x32 MFMA operand layout (A: 16 x 32, B: 32 x 16, D: 16 x 16):
//   A: lane l holds row l%16, contraction slots 8(l/16) .. +7
//   B: lane l holds col l%16, contraction slots 8(l/16) .. +7
//   D: lane l, register v holds row 4(l/16) + v, col l%16
// Contraction slot (step s, lane group g, element i) is dimension 32g + 8s + i
// for both operands: group g of the A side reads the bytes of dimensions
// 32g .. 32g+31 of its token, a contiguous piece of the packed code.
// Column n of column block cb is query token j = NCB*n + cb, so the NCB
// S^T values a lane needs for one doc token are adjacent in memory.
//
// Work split: a workgroup scores 4*dpw candidates of one query, each wave dpw
// (<= 64) of them as one flat stream of 16-token tiles.  The loop is software
// pipelined: while tile t is decoded and multiplied, the centroid ids of
// tile t+2, the codes of tile t+1 and the S^T rows of tile t+1 (whose
// addresses need tile t+1's ids) are in flight.  The loop is unrolled by two
// so that no register that is still being loaded is ever copied.
//
// The limit is the texture address unit: it spends 16 cycles on every 64-lane
// load of 64 or 128 bits (4 on a 32-bit one), and a tile takes six such loads
// (ids, codes, four S^T gathers).  Each gather touches only 4 cache lines
// (four full S^T rows): loads that touch more lines per instruction stall on
// L1 tag lookups instead.  Addresses are a wave-uniform 64-bit base (scalar
// registers) plus a small 32-bit lane offset; loads are never predicated: a
// tile may read up to 15 tokens past its document, which the index pads at
// the end of the token arrays, and those rows are masked only in a
// document's last, partial tile.
// Workgroup b runs on XCD b % 8; with 8 or more queries all workgroups of
// query q are given XCD q % 8 and queries are issued in order, so an XCD works
// on a few queries at a time and much of their S^T tables stays in its L2.
// With fewer than 8 queries, every XCD takes chunks of every query.
constexpr int RS_CACHE = 0;  // cache policy of every load (default)

template <int NBITS>
struct RsCodes {
  uint32_t w[NBITS == 2 ? 2 : 4];
};
struct RsIds {
  int32_t c[4];
};
// Wave-uniform tile cursor: document slot u, first token base, and that
// document's token offset and length (kept in scalar registers).
struct RsCur {
  int u, base, len;
  int64_t beg;
};

// Buffer resource (gfx9 family word 3) over [p, p + bytes): loads take a
// scalar base and a 32-bit lane offset, and read 0 past the range.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rs_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

template <int NBITS, int NCB>
struct RsWave {
  static constexpr int TQP = NCB * 16;
  static constexpr int CB = 16 * NBITS;
  const uint8_t *__restrict__ codes;
  const int32_t *__restrict__ cid;
  __amdgpu_buffer_rsrc_t st_rsrc;
  int64_t my_beg, beg0;
  int my_len, ndw, n, g;

  __device__ __forceinline__ void set_doc(RsCur &c, int u) const {
    c.u = __builtin_amdgcn_readfirstlane(u);
    c.base = 0;
    if (c.u < ndw) {
      c.len = __builtin_amdgcn_readlane(my_len, c.u);
      const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)my_beg, c.u);
      const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)my_beg >> 32), c.u);
      c.beg = (int64_t)(((uint64_t)hi << 32) | lo);
    } else {
      c.len = 0;
      c.beg = beg0;  // past the wave's last tile: read (and ignore) a valid tile
    }
  }
  // next 16-token tile of the wave's document stream
  __device__ __forceinline__ void advance(RsCur &c) const {
    if (c.u < ndw) {
      const int nb = c.base + 16;
      if (nb >= c.len) set_doc(c, c.u + 1);
      else c.base = __builtin_amdgcn_readfirstlane(nb);
    }
  }
  __device__ __forceinline__ void load_ids(RsIds &I, const RsCur &c) const {
    const __amdgpu_buffer_rsrc_t r = rs_rsrc(cid + c.beg + c.base, 64);
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (uint32_t)(16 * g), 0, RS_CACHE);
    I.c[0] = (int32_t)v[0]; I.c[1] = (int32_t)v[1]; I.c[2] = (int32_t)v[2]; I.c[3] = (int32_t)v[3];
  }
  __device__ __forceinline__ void load_codes(RsCodes<NBITS> &K, const RsCur &c) const {
    const __amdgpu_buffer_rsrc_t r = rs_rsrc(codes + (c.beg + c.base) * CB, 16 * CB);
    const uint32_t off = (uint32_t)(n * CB + (CB / 4) * g);
    if (NBITS == 2) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, RS_CACHE);
      K.w[0] = v[0]; K.w[1] = v[1];
    } else {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, RS_CACHE);
      K.w[0] = v[0]; K.w[1] = v[1]; K.w[2 % (NBITS == 2 ? 2 : 4)] = v[2]; K.w[3 % (NBITS == 2 ? 2 : 4)] = v[3];
    }
  }
  __device__ __forceinline__ void gather(float (&st)[4][NCB], const RsIds &I) const {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const uint32_t off = ((uint32_t)I.c[v] * TQP + NCB * n) * 4;
      if (NCB == 2) {
        const auto x = __builtin_amdgcn_raw_buffer_load_b64(st_rsrc, off, 0, 0);
        st[v][0] = __uint_as_float(x[0]); st[v][1 % NCB] = __uint_as_float(x[1]);
      } else {
        const auto x = __builtin_amdgcn_raw_buffer_load_b128(st_rsrc, off, 0, 0);
        st[v][0] = __uint_as_float(x[0]); st[v][1 % NCB] = __uint_as_float(x[1]);
        st[v][2 % NCB] = __uint_as_float(x[2]); st[v][3 % NCB] = __uint_as_float(x[3]);
      }
    }
  }
};

template <int NBITS, int NCB>
__global__ __launch_bounds__(256) void k_residual_score(
    const uint16_t *__restrict__ Qs, int64_t nq, int Tq, const float *__restrict__ ST, int ncent,
    const int64_t *__restrict__ doc_off, const int32_t *__restrict__ cid, const uint8_t *__restrict__ codes,
    uint4 w_lo, uint4 w_hi, const int32_t *__restrict__ cand_ids, const int32_t *__restrict__ n_valid, int ncand,
    int nchunks, int dpw, int32_t *__restrict__ fhat) {
  constexpr int TQP = NCB * 16;
  const int docs_per_block = 4 * dpw;
  const int b = blockIdx.x;
  const int64_t q = nq >= 8 ? (b & 7) + 8 * (int64_t)((b >> 3) / nchunks) : b / nchunks;
  const int chunk = nq >= 8 ? (b >> 3) % nchunks : b % nchunks;
  if (q >= nq) return;
  const int nv = n_valid[q];
  if (chunk * docs_per_block >= nv) return;  // uniform: before the only barrier

  // 2-bit: byte -> 4 weights (two bf16x2 words); 4-bit: byte -> 2 weights
  __shared__ uint2 lut2[NBITS == 2 ? 256 : 1];
  __shared__ uint32_t lut4[NBITS == 4 ? 256 : 1];
  {
    const uint16_t w[16] = {
        (uint16_t)w_lo.x, (uint16_t)(w_lo.x >> 16), (uint16_t)w_lo.y, (uint16_t)(w_lo.y >> 16),
        (uint16_t)w_lo.z, (uint16_t)(w_lo.z >> 16), (uint16_t)w_lo.w, (uint16_t)(w_lo.w >> 16),
        (uint16_t)w_hi.x, (uint16_t)(w_hi.x >> 16), (uint16_t)w_hi.y, (uint16_t)(w_hi.y >> 16),
        (uint16_t)w_hi.z, (uint16_t)(w_hi.z >> 16), (uint16_t)w_hi.w, (uint16_t)(w_hi.w >> 16)};
    const int e = threadIdx.x;  // 256 threads, one table entry each
    if (NBITS == 2)
      lut2[e] = make_uint2((uint32_t)w[e & 3] | ((uint32_t)w[(e >> 2) & 3] << 16),
                           (uint32_t)w[(e >> 4) & 3] | ((uint32_t)w[(e >> 6) & 3] << 16));
    else
      lut4[e] = (uint32_t)w[e & 15] | ((uint32_t)w[e >> 4] << 16);
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // this wave's documents: candidates chunk*4*dpw + wave + 4u, u < dpw; lane u holds doc u
  const int first = chunk * docs_per_block + wave;
  const int rem = nv - first;
  RsWave<NBITS, NCB> W;
  W.ndw = __builtin_amdgcn_readfirstlane(rem <= 0 ? 0 : min(dpw, (rem + 3) >> 2));
  if (W.ndw == 0) return;
  W.codes = codes;
  W.cid = cid;
  W.st_rsrc = rs_rsrc(ST + q * (int64_t)ncent * TQP, (uint32_t)ncent * TQP * 4);
  W.n = lane & 15;
  W.g = lane >> 4;
  W.my_beg = 0;
  W.my_len = 0;
  if (lane < W.ndw) {
    const int32_t V = cand_ids[q * ncand + first + 4 * lane];
    W.my_beg = doc_off[V];
    W.my_len = (int)(doc_off[V + 1] - W.my_beg);
  }
  {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)W.my_beg, 0);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)W.my_beg >> 32), 0);
    W.beg0 = (int64_t)(((uint64_t)hi << 32) | lo);
  }
  const int n = W.n, g = W.g;

  bf16x8 bq[NCB][4];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const uint4 *qp = (const uint4 *)(Qs + ((q * TQP) + NCB * n + cb) * 128 + 32 * g);
#pragma unroll
    for (int s = 0; s < 4; ++s) bq[cb][s] = as_bf16x8(qp[s]);
  }

  // cursors of tiles t (c), t+1 (nx) and t+2 (m)
  RsCur cc, nx, mm;
  W.set_doc(cc, 0);
  nx = cc;
  W.advance(nx);
  mm = nx;
  W.advance(mm);

  RsIds id0, id1;          // ids of tiles t+1 and t+2 (ring of 2)
  RsCodes<NBITS> k0, k1;   // codes of tiles t and t+1 (ring of 2)
  float st0[4][NCB], st1[4][NCB];  // S^T rows of tiles t and t+1 (ring of 2)
  {
    RsIds idc;
    W.load_ids(idc, cc);
    W.load_codes(k0, cc);
    W.load_ids(id0, nx);
    W.gather(st0, idc);
  }

  float mx[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) mx[cb] = -INFINITY;

  // One pipeline step.  In: kc/stc hold tile t; idn holds the ids of t+1.
  // Out: kn/stn hold tile t+1; idm holds the ids of t+2.
  auto step = [&](RsCodes<NBITS> &kc, float (&stc)[4][NCB], RsIds &idn, RsCodes<NBITS> &kn, float (&stn)[4][NCB],
                  RsIds &idm) {
    W.load_ids(idm, mm);
    W.load_codes(kn, nx);
    W.gather(stn, idn);
    const int len = cc.len, cbase = cc.base;
    bf16x8 a[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 u;
      if (NBITS == 2) {
        // step s covers code bytes 2s and 2s+1 of this lane's 8 bytes
        const uint32_t word = kc.w[s >> 1];
        const uint2 lo = lut2[(word >> (16 * (s & 1))) & 255u];
        const uint2 hi = lut2[(word >> (16 * (s & 1) + 8)) & 255u];
        u = make_uint4(lo.x, lo.y, hi.x, hi.y);
      } else {
        // step s covers code bytes 4s .. 4s+3 (word s)
        const uint32_t word = kc.w[s % (NBITS == 2 ? 2 : 4)];
        u = make_uint4(lut4[word & 255u], lut4[(word >> 8) & 255u], lut4[(word >> 16) & 255u], lut4[word >> 24]);
      }
      a[s] = as_bf16x8(u);
    }
    f32x4 acc[NCB];
    const bool partial = cbase + 16 > len;  // wave-uniform
#pragma unroll
    for (int v = 0; v < 4; ++v) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[cb][v] = stc[v][cb];
    }
    if (partial) {
      // rows past the document start at -inf and never win the maximum
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (cbase + 4 * g + v >= len)
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb][v] = -INFINITY;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], bq[cb][s], acc[cb], 0, 0, 0);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
      mx[cb] = fmaxf(mx[cb], fmaxf(fmaxf(acc[cb][0], acc[cb][1]), fmaxf(acc[cb][2], acc[cb][3])));
    if (cbase + 16 >= len) {
      // last tile of document cu: segmented max across the four lane groups,
      // then the exact integer sum over query tokens
      int key = 0;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        float m = mx[cb];
        m = fmaxf(m, shfl_xor(m, 16));
        m = fmaxf(m, shfl_xor(m, 32));
        if (NCB * n + cb < Tq) key += to_key(m);
        mx[cb] = -INFINITY;
      }
      key += shfl_xor(key, 1);
      key += shfl_xor(key, 2);
      key += shfl_xor(key, 4);
      key += shfl_xor(key, 8);
      if (lane == 0) fhat[q * ncand + first + 4 * cc.u] = key;
    }
    cc = nx;
    nx = mm;
    W.advance(mm);
  };

  while (true) {
    step(k0, st0, id0, k1, st1, id1);
    if (cc.u >= W.ndw) break;
    step(k1, st1, id1, k0, st0, id0);
    if (cc.u >= W.ndw) break;
  }
}

void launch_residual_score(const uint16_t *Qs, int64_t nq, int Tq, int TQP, const float *ST, int ncent,
                           const int64_t *doc_off, const int32_t *cid, const uint8_t *codes, int nbits,
                           const uint16_t *weights_host, const int32_t *cand_ids, const int32_t *n_valid, int ncand,
                           int32_t *fhat, hipStream_t s) {
  uint32_t w[8] = {0};
  const int B = 1 << nbits;
  for (int u = 0; u < B; ++u) w[u >> 1] |= (uint32_t)weights_host[u] << (16 * (u & 1));
  const uint4 w_lo = make_uint4(w[0], w[1], w[2], w[3]), w_hi = make_uint4(w[4], w[5], w[6], w[7]);
  // documents per wave: 16, fewer for small batches so that the chip still
  // gets about 2048 workgroups
  const int dpw = (int)std::max<int64_t>(1, std::min<int64_t>(16, (int64_t)ncand * nq / (4 * 2048)));
  const int nchunks = (ncand + 4 * dpw - 1) / (4 * dpw);
  const int64_t blocks = (nq >= 8 ? (nq + 7) / 8 * 8 : nq) * nchunks;
  if (blocks == 0) return;
#define CHIMERA_RS(NB, NC)                                                                                          \
  hipLaunchKernelGGL((k_residual_score<NB, NC>), dim3((unsigned)blocks), dim3(256), 0, s, Qs, nq, Tq, ST, ncent, \
                     doc_off, cid, codes, w_lo, w_hi, cand_ids, n_valid, ncand, nchunks, dpw, fhat)
  if (nbits == 2 && TQP == 32) CHIMERA_RS(2, 2);
  else if (nbits == 2) CHIMERA_RS(2, 4);
  else if (TQP == 32) CHIMERA_RS(4, 2);
  else CHIMERA_RS(4, 4);
#undef CHIMERA_RS
}

// ---------------------------------------------------------------- top-k
// One workgroup per query: radix selection of the k-th largest 64-bit key
// (F^ desc, doc asc) among the kept candidates, then a bitonic sort of the
// k winners in LDS.
constexpr int TOPK_THREADS = 1024;

__global__ __launch_bounds__(TOPK_THREADS) void k_topk(const int32_t *__restrict__ fhat,
                                                       const int32_t *__restrict__ cand_ids,
                                                       const int32_t *__restrict__ n_valid, int ncand, int k, int kpow2,
                                                       int32_t *__restrict__ ids, float *__restrict__ scores) {
  extern __shared__ uint64_t sk[];  // [kpow2]
  __shared__ int hist[256];
  __shared__ unsigned long long s_prefix, s_pmask;
  __shared__ int s_remaining, s_count;
  const int64_t q = blockIdx.x;
  const int n = n_valid[q];
  const int m = min(k, n);
  const int32_t *fh = fhat + q * ncand;
  const int32_t *ci = cand_ids + q * ncand;

  unsigned long long T = 0;  // every key >= T is taken
  if (n > k) {
    if (threadIdx.x == 0) { s_prefix = 0; s_pmask = 0; s_remaining = k; }
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
      for (int b = threadIdx.x; b < 256; b += TOPK_THREADS) hist[b] = 0;
      __syncthreads();
      const unsigned long long prefix = s_prefix, pmask = s_pmask;
      for (int i = threadIdx.x; i < n; i += TOPK_THREADS) {
        const unsigned long long K = pack_key(fh[i], (uint32_t)ci[i]);
        if ((K & pmask) == prefix) atomicAdd(&hist[(K >> shift) & 255], 1);
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        int rem = s_remaining, cum = 0, sel = 0;
        for (int b = 255; b >= 0; --b) {
          if (cum + hist[b] >= rem) { sel = b; break; }
          cum += hist[b];
        }
        s_remaining = rem - cum;
        s_prefix = prefix | ((unsigned long long)sel << shift);
        s_pmask = pmask | (255ull << shift);
      }
      __syncthreads();
    }
    T = s_prefix;  // keys are distinct: exactly k keys are >= T
  }
  for (int i = threadIdx.x; i < kpow2; i += TOPK_THREADS) sk[i] = 0;
  if (threadIdx.x == 0) s_count = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += TOPK_THREADS) {
    const unsigned long long K = pack_key(fh[i], (uint32_t)ci[i]);
    if (K >= T) {
      const int p = atomicAdd(&s_count, 1);
      if (p < kpow2) sk[p] = K;
    }
  }
  __syncthreads();
  // bitonic sort, descending
  for (int size = 2; size <= kpow2; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < kpow2; i += TOPK_THREADS) {
        const int p = i ^ stride;
        if (p > i) {
          const uint64_t a = sk[i], b = sk[p];
          const bool desc = (i & size) == 0;
          if (desc ? (a < b) : (a > b)) { sk[i] = b; sk[p] = a; }
        }
      }
      __syncthreads();
    }
  for (int r = threadIdx.x; r < k; r += TOPK_THREADS) {
    if (r < m) {
      const uint64_t K = sk[r];
      ids[q * k + r] = (int32_t)key_id(K);
      scores[q * k + r] = (float)key_score(K) * (1.0f / KEY_SCALE);
    } else {
      ids[q * k + r] = -1;
      scores[q * k + r] = -INFINITY;
    }
  }
}

void launch_topk(const int32_t *fhat, const int32_t *cand_ids, const int32_t *n_valid, int64_t nq, int ncand, int k,
                 int32_t *ids, float *scores, hipStream_t s) {
  int kp = 1;
  while (kp < k) kp <<= 1;
  hipLaunchKernelGGL(k_topk, dim3((unsigned)nq), dim3(TOPK_THREADS), (size_t)kp * 8, s, fhat, cand_ids, n_valid, ncand,
                     k, kp, ids, scores);
}

}  // namespace chimera
