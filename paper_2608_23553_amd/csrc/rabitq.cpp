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

}  // namespace

void rabitq_encode_rows(const int16_t *k, int64_t n, int dim, const int8_t *signs, uint8_t *bits1, float *g1,
                        uint8_t *codes4, float *g4) {
  constexpr int B = 4, half = 1 << (B - 1);
  std::vector<int64_t> xp(dim), av(dim);
  std::vector<int> lvl(dim), best(dim), ord(dim);
  std::vector<int> seq((size_t)dim * (half - 1));  // the chain's steps, in order
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
    int nz = 0;
    for (int d = 0; d < dim; ++d) {
      av[d] = xp[d] < 0 ? -xp[d] : xp[d];
      A += av[d];
      lvl[d] = best[d] = 0;
      if (av[d]) ord[nz++] = d;
    }
    const int64_t a1 = A;  // <xp, 2 y1>, y1 = sign / 2
    // Coordinate d steps from level m-1 to m at t = m / |xp_d| (m = 1 ..
    // half-1).  For a fixed m those times increase as |xp_d| decreases, so
    // with the coordinates in descending |xp| the steps form half-1 sorted
    // lists, merged here in order of t (exact comparisons of m / a as
    // m a' < m' a).  Steps of equal t are applied together before the
    // candidate is compared; their order among themselves does not matter.
    std::sort(ord.begin(), ord.begin() + nz, [&](int u, int v) { return av[u] != av[v] ? av[u] > av[v] : u < v; });
    int pos[half];
    for (int m = 1; m < half; ++m) pos[m] = 0;
    int64_t bA = A, bN = N;
    int total = nz * (half - 1), done = 0, ebest = 0;
    // the next step: the list whose head has the smallest t
    auto next = [&](int &mb) {
      mb = 0;
      for (int m = 1; m < half; ++m) {
        if (pos[m] >= nz) continue;
        if (!mb || (int64_t)m * av[ord[pos[mb]]] < (int64_t)mb * av[ord[pos[m]]]) mb = m;
      }
    };
    // the applied steps are recorded in seq and the best prefix is replayed
    // at the end
    while (done < total) {
      int m0;
      next(m0);
      const int64_t gm = m0, ga = av[ord[pos[m0]]];  // the group's time gm / ga
      for (;;) {
        int m;
        next(m);
        if (!m || (int64_t)m * ga != gm * av[ord[pos[m]]]) break;
        const int d = ord[pos[m]++];
        A += 2 * av[d];
        N += 8 * (int64_t)lvl[d] + 8;
        ++lvl[d];
        seq[done++] = d;
      }
      if ((__int128)A * A * bN > (__int128)bA * bA * N) {
        bA = A;
        bN = N;
        ebest = done;
      }
    }
    for (int e = 0; e < ebest; ++e) ++best[seq[e]];
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
