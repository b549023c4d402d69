// k_score.hip - document scoring of the refined candidates and the final
// top-k (Sec. 3.2 document scoring: the complete score over all tokens of
// each survivor, on the GPU; Sec. 4.2 document score aggregation; Alg. 1,
// final topK).
//
// Token score of doc token t against query token j (Chamfer, Def. 1, on the
// decoded token c_cid(t) + w[code_t]):
//     s[j][t] = S[j][cid(t)] + sum_d Q_j[d] * w[code_t[d]]
// The first term is read from the per-query S^T table written by the probe;
// the second is a [32 doc tokens x 128] x [128 x 32 query tokens] bf16 MFMA
// product whose doc-token operand is decoded in registers from the packed
// codes through an LDS lookup table indexed by code byte (the bucket-weight
// counterpart of the LUT inner product of Sec. 4.1: one lookup yields 4
// (2-bit) or 2 (4-bit) bf16 weights).  The S term enters as the MFMA
// accumulator's initial value.  Each document's codes are one contiguous span
// (document-major layout).  The maximum over the document's tokens stays in
// registers and the sum over query tokens is an integer sum of exact keys.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

// 32x32x16 MFMA operand layout (A: 32 x 16, B: 16 x 32, D: 32 x 32):
//   A: lane l holds row l%32, contraction slots 8(l/32) .. +7
//   B: lane l holds col l%32, contraction slots 8(l/32) .. +7
//   D: lane l, register v holds row 8(v/4) + 4(l/32) + v%4, col l%32
// Rows are the 32 doc tokens of a tile, columns query tokens (column block
// cb: tokens 32cb .. 32cb+31).  Contraction slot (step s, half h, element i)
// is dimension 64h + 8s + i on both sides, so half h of the doc side decodes
// one contiguous half of its token's packed code.
//
// The limit of this kernel is the vector memory front end: the texture
// address unit spends 4 cycles on a 64-lane 32-bit load and 16 on a 64- or
// 128-bit one, and one load instruction that touches many cache lines
// serialises on L1 tag lookups.  The loads are shaped for both:
//   S^T:   D register v holds two doc tokens (one per half wave) for 32 query
//          tokens, so its initial value is one 32-bit gather of two full
//          128-byte S^T rows (2 cache lines, 4 cycles)
//   codes: one 128-bit load per 32-token tile (the tile's contiguous codes)
//   ids:   one 32-bit load per tile; lane l reads the id of the row that D
//          register l%16 holds in its half, so DPP row_newbcast:v hands
//          every lane the id of its row in register v
//
// Work split: a workgroup scores 4 * dpw candidates of one query, each wave
// dpw contiguous ones.  Workgroup b runs on XCD b % 8; with 8 or more
// queries, all workgroups of query q are given XCD q % 8 and queries are
// issued in order, so an XCD works on a few queries at a time and much of
// their S^T tables stays in its L2.  With fewer than 8 queries, every XCD
// takes chunks of every query.
//
// A wave's documents form one flat stream of 32-token tiles, software
// pipelined: while tile t is decoded and multiplied, the ids of tile t+2 and
// the codes and S^T rows of tile t+1 (whose addresses need tile t+1's ids,
// loaded one step earlier) are in flight.  Registers that are still being
// loaded alternate between two slots, so the loop is unrolled by two, and it
// has one exit (exits between the steps make the compiler drain every load
// in flight at the loop head).
//
// Addresses are a wave-uniform 64-bit base (scalar registers) plus a small
// 32-bit lane offset; loads are never predicated: a tile may read up to 31
// tokens past its document, which the index pads at the end of the token
// arrays.  Rows past the document read the S^T sentinel row ncent, which
// holds -inf, so they never win the maximum.

template <int NBITS>
struct RsCodes {
  uint32_t w[NBITS == 2 ? 4 : 8];
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

// y of lane 16*(l/16) + K, plus a, for every lane l: one DPP add
// (row_newbcast writes every lane, so the move needs no old value)
template <int K>
__device__ __forceinline__ uint32_t rs_row_bcast_add(uint32_t y, uint32_t a) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)y, 0x150 + K, 0xF, 0xF, true) + a;
}
// sum over the 32 lanes of each half wave, in lanes 31 and 63
__device__ __forceinline__ int rs_half_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);  // row_mirror
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1, 3
  return v;
}

template <int NBITS, int NCB>
struct RsWave {
  static constexpr int TQP = NCB * 32;
  static constexpr int CB = 16 * NBITS;  // code bytes per token
  const uint8_t *__restrict__ codes;
  const int32_t *__restrict__ cid;
  __amdgpu_buffer_rsrc_t st_rsrc;
  int64_t my_beg;
  int my_len, ndw, c, h, idrow, sentinel;
  uint32_t hcol, l4;  // 64 * ((l >> 4) & 1) and 4 * (l & 15): 4 * c = hcol + l4

  // Cursor on document u of the wave (u >= ndw: past the end; those lanes
  // hold an empty document at token 0, so the cursor keeps reading valid,
  // ignored tiles).
  __device__ __forceinline__ void set_doc(RsCur &cu, int u) const {
    cu.u = u;
    cu.base = 0;
    cu.len = __builtin_amdgcn_readlane(my_len, u & 63);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)my_beg, u & 63);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)my_beg >> 32), u & 63);
    cu.beg = (int64_t)(((uint64_t)hi << 32) | lo);
  }
  // next 32-token tile of the wave's document stream
  __device__ __forceinline__ void advance(RsCur &cu) const {
    const int nb = cu.base + 32;
    if (nb >= cu.len) set_doc(cu, cu.u + 1);
    else cu.base = nb;
  }
  // tokens of the tile inside its document: the buffer ranges below end
  // there, so rows past the document read 0 without touching memory
  __device__ __forceinline__ uint32_t rows(const RsCur &cu) const { return (uint32_t)min(32, cu.len - cu.base); }
  // id of tile row idrow (the row D register l%16 holds in this lane's half)
  __device__ __forceinline__ int32_t load_id(const RsCur &cu) const {
    const __amdgpu_buffer_rsrc_t r = rs_rsrc(cid + cu.beg + cu.base, 4 * rows(cu));
    return (int32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (uint32_t)(4 * idrow), 0, 0);
  }
  // this lane's half of token c's code: bytes CB/2 * h .. +CB/2
  __device__ __forceinline__ void load_codes(RsCodes<NBITS> &K, const RsCur &cu) const {
    const __amdgpu_buffer_rsrc_t r = rs_rsrc(codes + (cu.beg + cu.base) * CB, CB * rows(cu));
    const uint32_t off = (uint32_t)(c * CB + (CB / 2) * h);
#pragma unroll
    for (int p = 0; p < NBITS / 2; ++p) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16 * p, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) K.w[4 * p + e] = v[e];
    }
  }
  // S^T[id(row of register v)][32cb + c]; rows past the document take the
  // sentinel row
  __device__ __forceinline__ void gather(float (&st)[NCB][16], int32_t x, const RsCur &cu) const {
    x = idrow < cu.len - cu.base ? x : sentinel;  // the row count is scalar
    // byte offset of row x plus this lane's 16-lane group's first column;
    // lane l reads that of lane 16*(l/16) + V and adds its own 4 * (l%16)
    const uint32_t y = (uint32_t)x * (TQP * 4) + hcol;
#define CHIMERA_G(V)                                                                                  \
  {                                                                                                   \
    const uint32_t off = rs_row_bcast_add<V>(y, l4);                                                  \
    _Pragma("unroll") for (int cb = 0; cb < NCB; ++cb) st[cb][V] =                                    \
        __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(st_rsrc, off + 128 * cb, 0, 0));         \
  }
    CHIMERA_G(0) CHIMERA_G(1) CHIMERA_G(2) CHIMERA_G(3) CHIMERA_G(4) CHIMERA_G(5) CHIMERA_G(6) CHIMERA_G(7)
    CHIMERA_G(8) CHIMERA_G(9) CHIMERA_G(10) CHIMERA_G(11) CHIMERA_G(12) CHIMERA_G(13) CHIMERA_G(14) CHIMERA_G(15)
#undef CHIMERA_G
  }
};

template <int NBITS, int NCB>
__global__ __launch_bounds__(256) void k_residual_score(
    const uint16_t *__restrict__ Qs, int64_t nq, int Tq, const float *__restrict__ ST, int ncent,
    const int64_t *__restrict__ doc_off, const int32_t *__restrict__ cid, const uint8_t *__restrict__ codes,
    uint4 w_lo, uint4 w_hi, const int32_t *__restrict__ cand_ids, const int32_t *__restrict__ n_valid, int ncand,
    int lo, int hi, int dpw, int nchunks, int32_t *__restrict__ fhat) {
  constexpr int TQP = NCB * 32;
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
  __syncthreads();  // the only barrier

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // workgroup b runs on XCD b % 8: with 8 or more queries, the chunks of
  // query q go to XCD q % 8, queries in order
  const int b = blockIdx.x;
  const int64_t q = nq >= 8 ? (b & 7) + 8 * (int64_t)((b >> 3) / nchunks) : b / nchunks;
  const int chunk = nq >= 8 ? (b >> 3) % nchunks : b % nchunks;
  if (q >= nq) return;
  // candidates lo .. min(hi, n_valid) - 1 of query q
  const int nv = min(n_valid[q], hi) - lo;
  // this wave's documents: those candidates' d0 .. d0 + nd - 1
  const int d0 = (chunk * 4 + wave) * dpw;
  const int nd = min(dpw, nv - d0);
  if (nd <= 0) return;

  RsWave<NBITS, NCB> W;
  W.codes = codes;
  W.cid = cid;
  W.c = lane & 31;
  W.hcol = 64 * ((lane >> 4) & 1);
  W.l4 = 4 * (lane & 15);
  W.h = lane >> 5;
  // the row that D register k = l%16 holds in this lane's half
  W.idrow = 8 * ((lane & 15) >> 2) + 4 * W.h + (lane & 3);
  W.sentinel = ncent;
  W.ndw = nd;
  const int c = W.c, h = W.h;
  W.st_rsrc = rs_rsrc(ST + q * (int64_t)(ncent + 1) * TQP, (uint32_t)(ncent + 1) * TQP * 4);
  W.my_beg = 0;
  W.my_len = 0;
  if (lane < nd) {
    const int32_t V = cand_ids[q * ncand + lo + d0 + lane];
    W.my_beg = doc_off[V];
    W.my_len = (int)(doc_off[V + 1] - W.my_beg);
  }
  // query operand: column 32cb + c, dimensions 64h + 8s .. +7
  bf16x8 bq[NCB][8];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const uint4 *qp = (const uint4 *)(Qs + (q * TQP + 32 * cb + c) * 128 + 64 * h);
#pragma unroll
    for (int s = 0; s < 8; ++s) bq[cb][s] = as_bf16x8(qp[s]);
  }
  int32_t *fout = fhat + q * ncand + lo + d0;

  // cursors of tiles t (c0), t+1 (c1), t+2 (c2)
  RsCur c0, c1, c2;
  W.set_doc(c0, 0);
  c1 = c0;
  W.advance(c1);
  c2 = c1;
  W.advance(c2);

  int32_t id0, id1;                      // ids of tiles t+1 and t+2 (ring of 2)
  RsCodes<NBITS> k0, k1;                 // codes of tiles t and t+1 (ring of 2)
  float st0[NCB][16], st1[NCB][16];      // S^T values of tiles t and t+1 (ring of 2)
  {
    const int32_t idc = W.load_id(c0);
    W.load_codes(k0, c0);
    id0 = W.load_id(c1);
    W.gather(st0, idc, c0);
  }
  float mx[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) mx[cb] = -INFINITY;

  // One pipeline step.  In: kc/stc hold tile t; idn holds the ids of t+1.
  // Out: kn/stn hold tile t+1; idm holds the ids of t+2.
  auto step = [&](RsCodes<NBITS> &kc, float (&stc)[NCB][16], int32_t &idn, RsCodes<NBITS> &kn,
                  float (&stn)[NCB][16], int32_t &idm) {
    const int32_t x = idn;
    idm = W.load_id(c2);
    W.load_codes(kn, c1);
    W.gather(stn, x, c1);
    // every load of tile t+1 is issued before tile t's products, so that
    // the only wait below is for tile t itself
    __builtin_amdgcn_sched_barrier(0);
    const int len = c0.len, cbase = c0.base;
    f32x16 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[cb][v] = stc[cb][v];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      uint4 u;
      if (NBITS == 2) {
        // step s covers code bytes 2s and 2s+1 of this lane's 16 bytes
        const uint32_t word = kc.w[s >> 1];
        const uint2 lo = lut2[(word >> (16 * (s & 1))) & 255u];
        const uint2 hi = lut2[(word >> (16 * (s & 1) + 8)) & 255u];
        u = make_uint4(lo.x, lo.y, hi.x, hi.y);
      } else {
        // step s covers code bytes 4s .. 4s+3 (word s)
        const uint32_t word = kc.w[s];
        u = make_uint4(lut4[word & 255u], lut4[(word >> 8) & 255u], lut4[(word >> 16) & 255u], lut4[word >> 24]);
      }
      const bf16x8 a = as_bf16x8(u);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[cb][s], acc[cb], 0, 0, 0);
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      float m = mx[cb];
#pragma unroll
      for (int v = 0; v < 16; ++v) m = fmaxf(m, acc[cb][v]);
      mx[cb] = m;
    }
    if (cbase + 32 >= len && c0.u < W.ndw) {
      // last tile of document c0.u: maximum over its tokens (the rows: the
      // 16 registers and the two halves), then the exact integer sum over
      // query tokens (the columns)
      int key = 0;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        // the two half waves hold the maxima of different rows: one
        // permlane32 swap puts both in every lane
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx[cb]), __float_as_uint(mx[cb]), false,
                                                         false);
        const float m = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        if (32 * cb + c < Tq) key += to_key(m);
        mx[cb] = -INFINITY;
      }
      key = rs_half_sum(key);
      if (lane == 31) fout[c0.u] = key;
    }
    c0 = c1;
    c1 = c2;
    W.advance(c2);
  };

  do {
    step(k0, st0, id0, k1, st1, id1);
    step(k1, st1, id1, k0, st0, id0);
  } while (c0.u < W.ndw);
}

void launch_residual_score(const uint16_t *Qs, int64_t nq, int Tq, int TQP, const float *ST, int ncent,
                           const int64_t *doc_off, const int32_t *cid, const uint8_t *codes, int nbits,
                           const uint16_t *weights_host, const int32_t *cand_ids, const int32_t *n_valid, int ncand,
                           int lo, int hi, int32_t *fhat, hipStream_t s) {
  if (nq <= 0 || hi <= lo) return;
  uint32_t w[8] = {0};
  const int B = 1 << nbits;
  for (int u = 0; u < B; ++u) w[u >> 1] |= (uint32_t)weights_host[u] << (16 * (u & 1));
  const uint4 w_lo = make_uint4(w[0], w[1], w[2], w[3]), w_hi = make_uint4(w[4], w[5], w[6], w[7]);
  // documents per wave: 8 (measured best at 4096 candidates per query: more
  // documents per wave put more queries' S^T tables in flight per XCD, fewer
  // add per-wave setup), fewer for small batches so that the chip still gets
  // about 2048 workgroups
  const int span = hi - lo;
  const int dpw = (int)std::max<int64_t>(1, std::min<int64_t>(8, (int64_t)span * nq / (4 * 2048)));
  const int nchunks = (span + 4 * dpw - 1) / (4 * dpw);
  const int64_t blocks = (nq >= 8 ? (nq + 7) / 8 * 8 : nq) * nchunks;
#define CHIMERA_RS(NB, NC)                                                                                        \
  hipLaunchKernelGGL((k_residual_score<NB, NC>), dim3((unsigned)blocks), dim3(256), 0, s, Qs, nq, Tq, ST, ncent, \
                     doc_off, cid, codes, w_lo, w_hi, cand_ids, n_valid, ncand, lo, hi, dpw, nchunks, fhat)
  if (nbits == 2 && TQP == 32) CHIMERA_RS(2, 1);
  else if (nbits == 2) CHIMERA_RS(2, 2);
  else if (TQP == 32) CHIMERA_RS(4, 1);
  else CHIMERA_RS(4, 2);
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
  __shared__ int s_remaining, s_count, s_done;
  const int64_t q = blockIdx.x;
  const int n = n_valid[q];
  const int m = min(k, n);
  const int32_t *fh = fhat + q * ncand;
  const int32_t *ci = cand_ids + q * ncand;

  unsigned long long T = 0;  // every key >= T is taken
  if (n > k) {
    if (threadIdx.x == 0) { s_prefix = 0; s_pmask = 0; s_remaining = k; s_done = 0; }
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
      if (threadIdx.x < 64) {
        // wave 0 finds the bin holding the rem-th largest key: lane l covers
        // bins 255 - 4l .. 252 - 4l, counts above it come from a lane scan
        const int lane = threadIdx.x, rem = s_remaining;
        int local = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) local += hist[255 - 4 * lane - i];
        int incl = local;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int y = __shfl_up(incl, d, 64);
          if (lane >= d) incl += y;
        }
        int cum = incl - local;
        if (cum < rem && incl >= rem) {
          for (int i = 0; i < 4; ++i) {
            const int b = 255 - 4 * lane - i;
            if (cum + hist[b] >= rem) {
              s_remaining = rem - cum;
              s_prefix = prefix | ((unsigned long long)b << shift);
              s_pmask = pmask | (255ull << shift);
              // the whole bin is needed: every key >= the bin's base is taken
              s_done = hist[b] == rem - cum;
              break;
            }
            cum += hist[b];
          }
        }
      }
      __syncthreads();
      if (s_done) break;
    }
    T = s_prefix;  // keys are distinct: exactly k keys are >= T (the base of the last bin)
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
  // k up to 8192: 64 KiB of dynamic LDS beside the static state, above the
  // default per-workgroup limit
  static bool attr = [] {
    return hipFuncSetAttribute((const void *)k_topk, hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024) ==
           hipSuccess;
  }();
  (void)attr;
  hipLaunchKernelGGL(k_topk, dim3((unsigned)nq), dim3(TOPK_THREADS), (size_t)kp * 8, s, fhat, cand_ids, n_valid, ncand,
                     k, kp, ids, scores);
}

}  // namespace chimera
