// rabitq.cpp - RaBitQ codes of document tokens, on the host (Sec. 2.2: the
// extended-bits RaBitQ quantiser; Sec. 3.1: B = 4 bits per dimension, split
// into the most significant bit, kept on the GPU, and the full code, kept in
// host memory).
//
// The random orthonormal rotation is P = H diag(s) / sqrt(D) (H the Sylvester
// Hadamard matrix, s the caller's random signs).  The factor 1/sqrt(D) and
// the norms of Eq. 2 cancel in every ratio used, so a token o (grid integers
// k) is rotated as xp = H diag(s) k, exactly, with the fast Walsh-Hadamard
// transform.  Its code is the codeword y of the half-integer grid
// {-(2^B-1)/2 .. (2^B-1)/2}^D of largest cosine with xp (ties: smallest
// |y|; a zero coordinate takes +1/2).  Rounding t * xp to that grid visits,
// as t grows, a chain of codewords that contains the best one, so the
// encoder walks the chain: each coordinate steps up at t = m / |xp_i|, and
// at every distinct step value the candidate is compared exactly (128-bit
// integers) with the best so far.  The estimate of <q, o> from a code
// (Eq. 5 with Eq. 2's norms, through Eq. 6) is
//     g * <H diag(s) q, 2y> * 2^-12,   g = |o|^2 / <P o, y>,
// and the stored factor is g = float(K2 / (A * 1024.0)) with K2 = sum k^2 and
// A = <xp, 2y> (one fp32 rounding).
#include <algorithm>
#include <cstring>
#include <vector>

#include "internal.h"

namespace chimera {

namespace {

// x <- H x in place (natural order: (H x)_i = sum_j (-1)^popcount(i & j) x_j)
void fwht(int64_t *x, int n) {
  for (int h = 1; h < n; h <<= 1)
    for (int i = 0; i < n; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        const int64_t a = x[j], b = x[j + h];
        x[j] = a + b;
        x[j + h] = a - b;
      }
}

struct Step {
  int64_t m, a;  // the coordinate steps up at t = m / a
  int i;
};

}  // namespace

void rabitq_encode_rows(const int16_t *k, int64_t n, int dim, const int8_t *signs, uint8_t *bits1, float *g1,
                        uint8_t *codes4, float *g4) {
  constexpr int B = 4, half = 1 << (B - 1);
  std::vector<int64_t> xp(dim);
  std::vector<int> lvl(dim), best(dim);
  std::vector<Step> steps;
  steps.reserve((size_t)dim * (half - 1));
  for (int64_t r = 0; r < n; ++r) {
    const int16_t *x = k + r * dim;
    int64_t k2 = 0;
    for (int d = 0; d < dim; ++d) {
      xp[d] = (int64_t)signs[d] * x[d];
      k2 += (int64_t)x[d] * x[d];
    }
    fwht(xp.data(), dim);
    // the chain of codewords: start at |y| = 1/2 everywhere
    int64_t A = 0, N = dim;
    steps.clear();
    for (int d = 0; d < dim; ++d) {
      const int64_t a = xp[d] < 0 ? -xp[d] : xp[d];
      A += a;
      lvl[d] = best[d] = 0;
      if (a)
        for (int m = 1; m < half; ++m) steps.push_back({m, a, d});
    }
    const int64_t a1 = A;  // <xp, 2 y1>, y1 = sign / 2
    std::sort(steps.begin(), steps.end(), [](const Step &u, const Step &v) {
      const int64_t l = u.m * v.a, rr = v.m * u.a;
      return l != rr ? l < rr : u.i < v.i;
    });
    int64_t bA = A, bN = N;
    for (size_t e = 0; e < steps.size();) {
      const Step &s0 = steps[e];
      while (e < steps.size() && steps[e].m * s0.a == s0.m * steps[e].a) {
        const int d = steps[e].i;
        A += 2 * steps[e].a;
        N += 8 * (int64_t)lvl[d] + 8;
        ++lvl[d];
        ++e;
      }
      if ((__int128)A * A * bN > (__int128)bA * bA * N) {
        bA = A;
        bN = N;
        std::copy(lvl.begin(), lvl.end(), best.begin());
      }
    }
    uint8_t *b1 = bits1 + r * (dim / 8);
    uint8_t *c4 = codes4 + r * (dim / 2);
    std::memset(b1, 0, dim / 8);
    for (int d = 0; d < dim; ++d) {
      const int code = xp[d] < 0 ? half - 1 - best[d] : half + best[d];
      if (code >= half) b1[d >> 3] |= (uint8_t)(1u << (d & 7));
      if (d & 1)
        c4[d >> 1] |= (uint8_t)(code << 4);
      else
        c4[d >> 1] = (uint8_t)code;
    }
    g1[r] = a1 ? (float)((double)k2 / ((double)a1 * 1024.0)) : 0.0f;
    g4[r] = bA ? (float)((double)k2 / ((double)bA * 1024.0)) : 0.0f;
  }
}

}  // namespace chimera
