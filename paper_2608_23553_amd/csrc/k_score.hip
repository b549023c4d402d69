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
#include "device_common.h"
#include "internal.h"

namespace chimera {

// 16x16x32 MFMA operand layout (A: 16 x 32, B: 32 x 16, D: 16 x 16):
//   A: lane l holds row l%16, contraction slots 8(l/16) .. +7
//   B: lane l holds col l%16, contraction slots 8(l/16) .. +7
//   D: lane l, register v holds row 4(l/16) + v, col l%16
// Contraction slot (step s, lane group g, element i) is dimension 32g + 8s + i
// for both operands: group g of the A side reads bytes of dimensions
// 32g .. 32g+31 of its token, a contiguous piece of the packed code.
template <int NBITS, int NCB>
__global__ __launch_bounds__(256) void k_residual_score(
    const uint16_t *__restrict__ Qs, int Tq, const float *__restrict__ ST, int ncent,
    const int64_t *__restrict__ doc_off, const int32_t *__restrict__ cid, const uint8_t *__restrict__ codes,
    uint4 w_lo, uint4 w_hi, const int32_t *__restrict__ cand_ids, const int32_t *__restrict__ n_valid, int ncand,
    int docs_per_block, int32_t *__restrict__ fhat) {
  constexpr int TQP = NCB * 16;
  constexpr int CODE_BYTES = 16 * NBITS;  // per token
  // 2-bit: byte -> 4 weights (two bf16x2 words); 4-bit: byte -> 2 weights
  __shared__ uint32_t lut[NBITS == 2 ? 512 : 256];
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
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int64_t q = blockIdx.y;
  const int nv = n_valid[q];
  const int i_end = min(nv, (int)(blockIdx.x + 1) * docs_per_block);

  bf16x8 bq[NCB][4];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const uint4 *qp = (const uint4 *)(Qs + ((q * TQP) + 16 * cb + n) * 128 + 32 * g);
#pragma unroll
    for (int s = 0; s < 4; ++s) bq[cb][s] = as_bf16x8(qp[s]);
  }
  const float *STq = ST + q * (int64_t)ncent * TQP;

  for (int i = blockIdx.x * docs_per_block + wave; i < i_end; i += 4) {
    const int32_t V = cand_ids[q * ncand + i];
    const int64_t t0 = doc_off[V];
    const int len = (int)(doc_off[V + 1] - t0);
    float mx[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) mx[cb] = -INFINITY;

    for (int base = 0; base < len; base += 16) {
      // ---- A operand: token base + n, dimensions 32g .. 32g+31
      const int tA = base + n;
      uint32_t cw[NBITS == 2 ? 2 : 4];
      if (tA < len) {
        const uint8_t *cp = codes + (t0 + tA) * CODE_BYTES + (CODE_BYTES / 4) * g;
        if (NBITS == 2) {
          const uint2 v = *(const uint2 *)cp;
          cw[0] = v.x; cw[1] = v.y;
        } else {
          const uint4 v = *(const uint4 *)cp;
          cw[0] = v.x; cw[1] = v.y; cw[2] = v.z; cw[3] = v.w;
        }
      } else {
#pragma unroll
        for (int w = 0; w < (NBITS == 2 ? 2 : 4); ++w) cw[w] = 0;
      }
      bf16x8 a[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        uint4 u;
        if (NBITS == 2) {
          // step s covers code bytes 2s and 2s+1 of this lane's 8 bytes
          const uint32_t word = cw[s >> 1];
          const uint32_t b0 = (word >> (16 * (s & 1))) & 255u, b1 = (word >> (16 * (s & 1) + 8)) & 255u;
          u.x = lut[2 * b0]; u.y = lut[2 * b0 + 1];
          u.z = lut[2 * b1]; u.w = lut[2 * b1 + 1];
        } else {
          // step s covers code bytes 4s .. 4s+3 (word s)
          const uint32_t word = cw[s];
          u.x = lut[word & 255u]; u.y = lut[(word >> 8) & 255u];
          u.z = lut[(word >> 16) & 255u]; u.w = lut[word >> 24];
        }
        a[s] = as_bf16x8(u);
      }
      // ---- accumulator init: S[j][cid(t)] for D rows t = base + 4g + v
      f32x4 acc[NCB];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int tC = base + 4 * g + v;
        if (tC < len) {
          const float *row = STq + (int64_t)cid[t0 + tC] * TQP + n;
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb][v] = row[16 * cb];
        } else {
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb][v] = -INFINITY;
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], bq[cb][s], acc[cb], 0, 0, 0);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        mx[cb] = fmaxf(mx[cb], fmaxf(fmaxf(acc[cb][0], acc[cb][1]), fmaxf(acc[cb][2], acc[cb][3])));
    }
    // segmented max: the four lane groups hold different doc tokens
    int key = 0;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      float m = mx[cb];
      m = fmaxf(m, shfl_xor(m, 16));
      m = fmaxf(m, shfl_xor(m, 32));
      if (16 * cb + n < Tq) key += to_key(m);
    }
    // sum over query tokens: integer, exact
    key += shfl_xor(key, 1);
    key += shfl_xor(key, 2);
    key += shfl_xor(key, 4);
    key += shfl_xor(key, 8);
    if (lane == 0) fhat[q * ncand + i] = key;
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
  const int docs_per_block = 64;
  dim3 grid((unsigned)((ncand + docs_per_block - 1) / docs_per_block), (unsigned)nq);
  if (grid.x == 0) return;
#define CHIMERA_RS(NB, NC)                                                                                        \
  hipLaunchKernelGGL((k_residual_score<NB, NC>), grid, dim3(256), 0, s, Qs, Tq, ST, ncent, doc_off, cid, codes, \
                     w_lo, w_hi, cand_ids, n_valid, ncand, docs_per_block, fhat)
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
