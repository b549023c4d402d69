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
// int8 MFMA products, with the bits expanded in registers to bytes 0 / 1 as
// the B operand.  x is a multiple of 2^-11 below 32 in magnitude (query
// tokens of norm below 2.8), so X = 2048 x is an integer below 2^16 and the
// sum of three int8 limbs, X = a 2^14 + b 2^7 + c with 0 <= b, c < 128.  The
// three limb products are chained through the MFMA accumulator (Horner:
// shift by 7 bits between limbs), giving <X, b_t> exactly in int32; it is
// below 2^23, so the float of <x, b_t> = <X, b_t> 2^-11 is exact.  The
// subtraction is exact too; the multiply by g1 is the one fp32 rounding.
// The maximum over the document's tokens stays in registers; the sum over
// query tokens is an integer sum of keys rint(max * 2^22).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "internal.h"

namespace chimera {

typedef int v4i32 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

// One wave per query row (256 threads: 4 rows): x = H diag(s) q in fp32
// (lane l holds dimensions 2l and 2l + 1; the butterflies of stride 2m > 1
// pair lanes l and l ^ m), its int8 limbs (row r: limb a at bytes
// 384 r + d, b at 384 r + 128 + d, c at 384 r + 256 + d for dimension d), and
// sum(x).
__global__ __launch_bounds__(256) void k_rq_prep(const uint16_t *__restrict__ Qs, int64_t rows,
                                                 const int8_t *__restrict__ signs, uint8_t *__restrict__ Qi8,
                                                 float *__restrict__ qsum) {
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
  // X = 2048 x (exact integers), as limbs a (arithmetic shift), b, c
  const int X0 = (int)(x0 * 2048.0f), X1 = (int)(x1 * 2048.0f);
  uint16_t *q = (uint16_t *)(Qi8 + row * RQ_ROW_BYTES);
  q[lane] = (uint16_t)((uint32_t)(X0 >> 14) & 0xFFu) | (uint16_t)(((uint32_t)(X1 >> 14) & 0xFFu) << 8);
  q[64 + lane] = (uint16_t)((X0 >> 7) & 127) | (uint16_t)(((X1 >> 7) & 127) << 8);
  q[128 + lane] = (uint16_t)(X0 & 127) | (uint16_t)((X1 & 127) << 8);
  float sum = x0 + x1;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, 64);
  if (lane == 0) qsum[row] = sum;
}

// bytes 0 / 1 of the 16 bits of `w` (byte j of word k = bit 4k + j): each
// nibble's bits move to the low bit of a byte by one multiply, whose four
// shifted copies of the nibble do not overlap
__device__ __forceinline__ v4i32 rq_expand16(uint32_t w) {
  v4i32 v;
#pragma unroll
  for (int k = 0; k < 4; ++k) v[k] = (int)((((w >> (4 * k)) & 15u) * 0x00204081u) & 0x01010101u);
  return v;
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
// across them.  MFMA 32x32x32 int8: rows are 32 query tokens (A, lane l holds
// row l % 32), columns 32 document tokens of a tile (B, lane l holds column
// l % 32); step s of a limb feeds the 16 bytes of dimensions 64h + 16s .. +15
// on both sides (the same bytes of A and B meet in the product, whatever
// slots of the contraction the hardware gives them), so lane (col, h) reads
// bytes 8h .. 8h + 7 of its token's 16-byte code.  D register v of lane l is
// query row 8(v/4) + 4(l/32) + v%4, document token l % 32.  The estimate of
// row r and token t is g_t (<x_r, b_t> - sum(x_r) / 2); its maximum over the
// document's tokens is taken per lane over the tiles, then across the 32
// columns of each half wave.  With 32 query tokens the kernel is held to 4
// waves per SIMD (128 VGPRs and a 12-byte spill: 1.97 ms against 2.16 ms at
// 3 waves at 100k).
template <int NCB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NCB == 1 ? 4 : 1))) void k_rq_score(
    const uint8_t *__restrict__ Qi8, const float *__restrict__ qsum, const int64_t *__restrict__ doc_off,
    const uint8_t *__restrict__ bits, const float *__restrict__ g1, const int32_t *__restrict__ cand_ids,
    const int32_t *__restrict__ n_valid, int ncand, int lo, int hi, int dpw, int32_t *__restrict__ fhat) {
  constexpr int TQP = 32 * NCB;
  const int lane = threadIdx.x & 63, col = lane & 31, h = lane >> 5;
  const int64_t q = blockIdx.y;
  const int c0 = lo + ((int)blockIdx.x * 4 + (int)(threadIdx.x >> 6)) * dpw;
  const int c1 = min(c0 + dpw, min(hi, n_valid[q]));
  if (c0 >= c1) return;  // wave-uniform
  // limbs a, b, c of the query row: step s covers dimensions 64h + 16s .. +15
  v4i32 qa[4], qb[4], qc[4];
  float half_sum[16];
  auto load_block = [&](int rb) {
    const uint8_t *qr = Qi8 + (q * TQP + rb * 32 + col) * RQ_ROW_BYTES + 64 * h;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      qa[s] = *(const v4i32 *)(qr + 16 * s);
      qb[s] = *(const v4i32 *)(qr + 128 + 16 * s);
      qc[s] = *(const v4i32 *)(qr + 256 + 16 * s);
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
      // tokens past the document read the next ones (the arrays are padded);
      // a wave-uniform base and this lane's fixed offset
      const uint8_t *tb = bits + (beg + t0) * 16;
      const float *tg = g1 + beg + t0;
      const uint2 b = *(const uint2 *)(tb + (uint32_t)(col * 16 + 8 * h));
      const float g = tg[col];
      const bool valid = t0 + col < len;
      v4i32 bb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) bb[s] = rq_expand16((s < 2 ? b.x : b.y) >> (16 * (s & 1)));
      // <X, b> = ((<a, b> 2^7) + <b-limb, b>) 2^7 + <c, b>, chained through
      // the accumulator
      i32x16 acc;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = 0;
#pragma unroll
      for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(qa[s], bb[s], acc, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] <<= 7;
#pragma unroll
      for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(qb[s], bb[s], acc, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] <<= 7;
#pragma unroll
      for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(qc[s], bb[s], acc, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float e = g * ((float)acc[v] * (1.0f / 2048.0f) - half_sum[v]);
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

void launch_rq_prep(const uint16_t *Qs, int64_t rows, const int8_t *signs, uint8_t *Qi8, float *qsum, hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(k_rq_prep, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, Qs, rows, signs, Qi8, qsum);
}

void launch_rq_score(const uint8_t *Qi8, const float *qsum, int64_t nq, int TQP,
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
    hipLaunchKernelGGL((k_rq_score<1>), grid, dim3(256), 0, s, Qi8, qsum, doc_off, bits, g1, cand_ids, n_valid,
                       ncand, lo, hi, dpw, fhat);
  else
    hipLaunchKernelGGL((k_rq_score<2>), grid, dim3(256), 0, s, Qi8, qsum, doc_off, bits, g1, cand_ids, n_valid,
                       ncand, lo, hi, dpw, fhat);
}

}  // namespace chimera
