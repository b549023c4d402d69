// k_rabitq.hip - document scoring from RaBitQ 1-bit codes (Sec. 3.2 document
// scoring on the GPU: the complete 1-bit score over every token of each kept
// document; Sec. 2.2, Eqs. 5-6, the estimate from a code; Sec. 4.1, the
// binary inner product).
//
// For query token q and document token t with most significant bits b_t and
// factor g1_t (rabitq.cpp):
//     est(q, t) = g1_t * (<x, b_t> - sum(x) / 2),   x = H diag(s) q,
// which is g1_t * <x, b_t - 1/2>, the 1-bit form of Eq. 6.  The paper sums
// table entries over 4-bit chunks of b (Sec. 4.1) on the vector units; here
// the binary inner products of 32 query tokens with 32 document tokens are
// one bf16 MFMA product per 16 dimensions, with the bits expanded in
// registers to bf16 0 / 1 as the B operand.  x is a multiple of 2^-11 below
// 32 in magnitude (query tokens of norm below 2.8), so it is the exact sum of
// two bf16 values hi + lo, and <x, b> is the exact fp32 sum of two MFMA
// products (every partial sum is a multiple of 2^-11 below 2^12).  The
// subtraction is exact too; the multiply by g1 is the one fp32 rounding.
// The maximum over the document's tokens stays in registers; the sum over
// query tokens is an integer sum of keys rint(max * 2^22).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

// One wave per query row (256 threads: 4 rows): x = H diag(s) q in fp32
// (lane l holds dimensions 2l and 2l + 1; the butterflies of stride 2m > 1
// pair lanes l and l ^ m), split into bf16 hi and lo, and sum(x).
__global__ __launch_bounds__(256) void k_rq_prep(const uint16_t *__restrict__ Qs, int64_t rows,
                                                 const int8_t *__restrict__ signs, uint32_t *__restrict__ Qh,
                                                 uint32_t *__restrict__ Ql, float *__restrict__ qsum) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint32_t w = ((const uint32_t *)(Qs + row * 128))[lane];
  float x0 = __uint_as_float(w << 16) * (float)signs[2 * lane];
  float x1 = __uint_as_float(w & 0xFFFF0000u) * (float)signs[2 * lane + 1];
  float a = x0 + x1, b = x0 - x1;
  x0 = a;
  x1 = b;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const float y0 = __shfl_xor(x0, m, 64), y1 = __shfl_xor(x1, m, 64);
    if (lane & m) {
      x0 = y0 - x0;
      x1 = y1 - x1;
    } else {
      x0 = x0 + y0;
      x1 = x1 + y1;
    }
  }
  // hi = bf16 nearest (ties to even), lo = x - hi (exact in bf16)
  auto hi16 = [](float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u & 0xFFFF0000u;
  };
  const uint32_t h0 = hi16(x0), h1 = hi16(x1);
  const float l0 = x0 - __uint_as_float(h0), l1 = x1 - __uint_as_float(h1);
  Qh[row * 64 + lane] = (h0 >> 16) | h1;
  Ql[row * 64 + lane] = (__float_as_uint(l0) >> 16) | (__float_as_uint(l1) & 0xFFFF0000u);
  float sum = x0 + x1;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
  if (lane == 0) qsum[row] = sum;
}

// bf16 0 / 1 of bits 0..7 of `byte` (element i = bit i)
__device__ __forceinline__ bf16x8 rq_expand(uint32_t byte) {
  uint4 v;
  v.x = ((byte & 1u) ? 0x3F80u : 0u) | ((byte & 2u) ? 0x3F800000u : 0u);
  v.y = ((byte & 4u) ? 0x3F80u : 0u) | ((byte & 8u) ? 0x3F800000u : 0u);
  v.z = ((byte & 16u) ? 0x3F80u : 0u) | ((byte & 32u) ? 0x3F800000u : 0u);
  v.w = ((byte & 64u) ? 0x3F80u : 0u) | ((byte & 128u) ? 0x3F800000u : 0u);
  return as_bf16x8(v);
}

// Maximum over the 32 lanes of each half wave, in lanes 31 and 63 (lanes
// whose DPP source is off take -inf, the identity of max).
__device__ __forceinline__ float rq_half_max(float x) {
  const int ninf = __float_as_int(-INFINITY);
  int v = __float_as_int(x);
#define CHIMERA_MX(CTRL, ROWMASK) \
  v = __float_as_int(fmaxf(__int_as_float(v), __int_as_float(__builtin_amdgcn_update_dpp(ninf, v, CTRL, ROWMASK, 0xF, false))))
  CHIMERA_MX(0xB1, 0xF);   // quad_perm [1,0,3,2]
  CHIMERA_MX(0x4E, 0xF);   // quad_perm [2,3,0,1]
  CHIMERA_MX(0x141, 0xF);  // row_half_mirror
  CHIMERA_MX(0x140, 0xF);  // row_mirror
  CHIMERA_MX(0x142, 0xA);  // row_bcast:15 into rows 1, 3
#undef CHIMERA_MX
  return __int_as_float(v);
}

// A wave scores dpw consecutive kept documents (candidates c of query q,
// lo <= c < min(hi, n_valid[q])), holding the query operand in registers
// across them.  MFMA 32x32x16: rows are 32 query tokens (A, lane l holds row
// l % 32), columns 32 document tokens of a tile (B, lane l holds column
// l % 32); contraction slot (step s, half h, element i) is dimension
// 64h + 8s + i on both sides, so lane (col, h) reads bytes 8h .. 8h + 7 of its
// token's 16-byte code.  D register v of lane l is query row
// 8(v/4) + 4(l/32) + v%4, document token l % 32.  The estimate of row r and
// token t is g_t (acc - sum(x_r) / 2); its maximum over the document's tokens
// is taken per lane over the tiles, then across the 32 columns of each half
// wave.
template <int NCB>
__global__ __launch_bounds__(256) void k_rq_score(const uint32_t *__restrict__ Qh, const uint32_t *__restrict__ Ql,
                                                  const float *__restrict__ qsum, const int64_t *__restrict__ doc_off,
                                                  const uint8_t *__restrict__ bits, const float *__restrict__ g1,
                                                  const int32_t *__restrict__ cand_ids,
                                                  const int32_t *__restrict__ n_valid, int ncand, int lo, int hi,
                                                  int dpw, int32_t *__restrict__ fhat) {
  constexpr int TQP = 32 * NCB;
  const int lane = threadIdx.x & 63, col = lane & 31, h = lane >> 5;
  const int64_t q = blockIdx.y;
  const int c0 = lo + ((int)blockIdx.x * 4 + (int)(threadIdx.x >> 6)) * dpw;
  const int c1 = min(c0 + dpw, min(hi, n_valid[q]));
  if (c0 >= c1) return;  // wave-uniform
  bf16x8 ah[8], al[8];
  float half_sum[16];
  auto load_block = [&](int rb) {
    const int64_t qrow = q * TQP + rb * 32 + col;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      ah[s] = as_bf16x8(*(const uint4 *)(Qh + qrow * 64 + 32 * h + 4 * s));
      al[s] = as_bf16x8(*(const uint4 *)(Ql + qrow * 64 + 32 * h + 4 * s));
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) half_sum[v] = 0.5f * qsum[q * TQP + rb * 32 + 8 * (v >> 2) + 4 * h + (v & 3)];
  };
  // the integer key sum of one document over the current block's 32 rows
  auto score_doc = [&](int64_t beg, int len) -> long long {
    float mx[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) mx[v] = -INFINITY;
    for (int t0 = 0; t0 < len; t0 += 32) {
      // tokens past the document read the next ones (the arrays are padded)
      const int64_t tok = beg + t0 + col;
      const uint2 b = *(const uint2 *)(bits + tok * 16 + 8 * h);
      const float g = g1[tok];
      const bool valid = t0 + col < len;
      f32x16 acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 bb = rq_expand(((s < 4 ? b.x : b.y) >> (8 * (s & 3))) & 0xFFu);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[s], bb, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[s], bb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float e = g * (acc[v] - half_sum[v]);
        if (valid) mx[v] = fmaxf(mx[v], e);
      }
    }
    // each half holds 16 of the block's 32 rows: their maxima land in lanes
    // 31 and 63
    long long part = 0;
#pragma unroll
    for (int v = 0; v < 16; ++v) part += (long long)rintf(rq_half_max(mx[v]) * KEY_SCALE);
    const int lo32 = __builtin_amdgcn_readlane((int)(uint32_t)part, 31), hi32 = __builtin_amdgcn_readlane((int)(part >> 32), 31);
    const int lo63 = __builtin_amdgcn_readlane((int)(uint32_t)part, 63), hi63 = __builtin_amdgcn_readlane((int)(part >> 32), 63);
    return (long long)(((uint64_t)(uint32_t)hi32 << 32) | (uint32_t)lo32) +
           (long long)(((uint64_t)(uint32_t)hi63 << 32) | (uint32_t)lo63);
  };
  auto put = [&](int c, long long total) {
    if (lane == 0)
      fhat[q * ncand + c] = (int32_t)std::min<long long>(INT32_MAX, std::max<long long>(-INT32_MAX, total));
  };
  if constexpr (NCB == 1) {
    load_block(0);
    for (int c = c0; c < c1; ++c) {
      const int32_t doc = cand_ids[q * ncand + c];
      const int64_t beg = doc_off[doc];
      put(c, score_doc(beg, (int)(doc_off[doc + 1] - beg)));
    }
  } else {
    for (int c = c0; c < c1; ++c) {
      const int32_t doc = cand_ids[q * ncand + c];
      const int64_t beg = doc_off[doc];
      const int len = (int)(doc_off[doc + 1] - beg);
      long long total = 0;
#pragma unroll 1
      for (int rb = 0; rb < NCB; ++rb) {
        load_block(rb);
        total += score_doc(beg, len);
      }
      put(c, total);
    }
  }
}

void launch_rq_prep(const uint16_t *Qs, int64_t rows, const int8_t *signs, uint32_t *Qh, uint32_t *Ql, float *qsum,
                    hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_rq_prep, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, Qs, rows, signs, Qh, Ql, qsum);
}

void launch_rq_score(const uint32_t *Qh, const uint32_t *Ql, const float *qsum, int64_t nq, int TQP,
                     const int64_t *doc_off, const uint8_t *bits, const float *g1, const int32_t *cand_ids,
                     const int32_t *n_valid, int ncand, int lo, int hi, int32_t *fhat, hipStream_t s) {
  if (nq <= 0 || hi <= lo) return;
  // documents per wave: up to 8 (the query operand is loaded once per wave),
  // fewer for small batches so that the chip still gets about 2048
  // workgroups
  const int span = hi - lo;
  const int dpw = (int)std::max<int64_t>(1, std::min<int64_t>(8, (int64_t)span * nq / (4 * 2048)));
  const dim3 grid((unsigned)((span + 4 * dpw - 1) / (4 * dpw)), (unsigned)nq);
  if (TQP == 32)
    hipLaunchKernelGGL((k_rq_score<1>), grid, dim3(256), 0, s, Qh, Ql, qsum, doc_off, bits, g1, cand_ids, n_valid,
                       ncand, lo, hi, dpw, fhat);
  else
    hipLaunchKernelGGL((k_rq_score<2>), grid, dim3(256), 0, s, Qh, Ql, qsum, doc_off, bits, g1, cand_ids, n_valid,
                       ncand, lo, hi, dpw, fhat);
}

}  // namespace chimera
