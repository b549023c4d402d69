// builder.cpp - offline index building (Sec. 3.1) and the index file format.
//
// The build takes centroids, document tokens and each token's centroid (its
// IVF assignment, Sec. 2.3) and produces:
//   * document-major per-token data: centroid id and packed residual codes,
//     each document's tokens contiguous (the document-reordered code copy of
//     Sec. 4.1, here the only copy);
//   * doc-level posting lists: for centroid c, the ascending distinct
//     documents owning a token assigned to c (Sec. 2.3 posting lists; the
//     candidate set of Sec. 3.2 only needs the documents);
//   * the residual quantiser: 2^b buckets cut at pooled empirical quantiles.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <memory>
#include <mutex>
#include <thread>

#include "internal.h"

namespace chimera {

// ------------------------------------------------------------------ grid
int32_t grid_k_of_float(float x) {
  float a = std::fabs(x);
  if (a < 0.0625f) return (int32_t)std::nearbyint(x * 2048.0f);
  uint32_t u;
  std::memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);  // bf16 round to nearest even
  u &= 0xFFFF0000u;
  float g;
  std::memcpy(&g, &u, 4);
  return (int32_t)std::nearbyint(g * 2048.0f);
}

float float_of_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

uint16_t bf16_of_grid_k(int32_t k) {
  float f = (float)k * (1.0f / 2048.0f);
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);  // exact for grid values
}

static unsigned hw_threads() {
  unsigned n = std::thread::hardware_concurrency();
  return n ? std::min(n, 32u) : 4u;
}

template <class F>
static void parallel_for(int64_t n, F f) {
  unsigned T = hw_threads();
  if (n < 4096 || T <= 1) { f(0, n); return; }
  std::vector<std::thread> th;
  int64_t per = (n + T - 1) / T;
  for (unsigned i = 0; i < T; ++i) {
    int64_t a = i * per, b = std::min(n, a + per);
    if (a >= b) break;
    th.emplace_back(f, a, b);
  }
  for (auto &t : th) t.join();
}

// ------------------------------------------------------------ checksums
// FNV-1a over little-endian 64-bit words, then the trailing bytes.
static uint64_t fnv64(const void *p, size_t n, uint64_t h = 14695981039346656037ull) {
  const uint8_t *b = (const uint8_t *)p;
  size_t w = n / 8;
  for (size_t i = 0; i < w; ++i) {
    uint64_t x;
    std::memcpy(&x, b + 8 * i, 8);
    h ^= x;
    h *= 1099511628211ull;
  }
  for (size_t i = 8 * w; i < n; ++i) {
    h ^= b[i];
    h *= 1099511628211ull;
  }
  return h;
}

// ------------------------------------------------------------ file format
// [0, 1024): header; then sections, each at a 256-byte aligned offset.
static const char kMagic[8] = {'C', 'H', 'I', 'M', 'I', 'D', 'X', '1'};
static const uint32_t kVersion = 1;
enum { SEC_CENT = 1, SEC_DOC_OFF, SEC_CID, SEC_CODES, SEC_CUT, SEC_WEIGHTS, SEC_IVF_OFF, SEC_IVF_DOC, NSEC = 8 };

struct FileSection {
  uint32_t id, pad;
  uint64_t offset, bytes, checksum;
};
struct FileHeader {
  char magic[8];
  uint32_t version, header_bytes;
  int32_t dim, nbits, ncent, max_doc_len;
  int64_t ndocs, ntok, nnz;
  uint32_t nsections, pad;
  FileSection sec[NSEC];
};
static_assert(sizeof(FileHeader) <= 1024, "header");

static void section_view(const HostIndex &h, int id, const void *&p, uint64_t &bytes) {
  switch (id) {
    case SEC_CENT: p = h.cent.data(); bytes = h.cent.size() * 2; break;
    case SEC_DOC_OFF: p = h.doc_off.data(); bytes = h.doc_off.size() * 8; break;
    case SEC_CID: p = h.cid.data(); bytes = h.cid.size() * 4; break;
    case SEC_CODES: p = h.codes.data(); bytes = h.codes.size(); break;
    case SEC_CUT: p = h.cut_k.data(); bytes = h.cut_k.size() * 4; break;
    case SEC_WEIGHTS: p = h.weights.data(); bytes = h.weights.size() * 2; break;
    case SEC_IVF_OFF: p = h.ivf_off.data(); bytes = h.ivf_off.size() * 8; break;
    default: p = h.ivf_doc.data(); bytes = h.ivf_doc.size() * 4; break;
  }
}

int save_index(const HostIndex &h, const char *path) {
  FILE *f = std::fopen(path, "wb");
  if (!f) return fail(CHIMERA_E_IO, "cannot open %s for writing", path);
  FileHeader hd;
  std::memset(&hd, 0, sizeof hd);
  std::memcpy(hd.magic, kMagic, 8);
  hd.version = kVersion;
  hd.header_bytes = 1024;
  hd.dim = h.dim; hd.nbits = h.nbits; hd.ncent = h.ncent; hd.max_doc_len = h.max_doc_len;
  hd.ndocs = h.ndocs; hd.ntok = h.ntok; hd.nnz = h.nnz;
  hd.nsections = NSEC;
  uint64_t off = 1024;
  for (int i = 0; i < NSEC; ++i) {
    const void *p; uint64_t bytes;
    section_view(h, i + 1, p, bytes);
    hd.sec[i].id = i + 1;
    hd.sec[i].offset = off;
    hd.sec[i].bytes = bytes;
    hd.sec[i].checksum = fnv64(p, bytes);
    off = (off + bytes + 255) / 256 * 256;
  }
  std::vector<char> head(1024, 0);
  std::memcpy(head.data(), &hd, sizeof hd);
  bool ok = std::fwrite(head.data(), 1, 1024, f) == 1024;
  static const char zeros[256] = {0};
  for (int i = 0; i < NSEC && ok; ++i) {
    const void *p; uint64_t bytes;
    section_view(h, i + 1, p, bytes);
    ok = std::fwrite(p, 1, bytes, f) == bytes;
    uint64_t end = hd.sec[i].offset + bytes, next = (end + 255) / 256 * 256;
    if (ok && next > end) ok = std::fwrite(zeros, 1, next - end, f) == next - end;
  }
  if (std::fclose(f) != 0) ok = false;
  if (!ok) return fail(CHIMERA_E_IO, "write to %s failed", path);
  return CHIMERA_OK;
}

int load_index(const char *path, HostIndex &h) {
  FILE *f = std::fopen(path, "rb");
  if (!f) return fail(CHIMERA_E_IO, "cannot open %s", path);
  std::unique_ptr<FILE, int (*)(FILE *)> guard(f, std::fclose);
  std::vector<char> head(1024);
  if (std::fread(head.data(), 1, 1024, f) != 1024) return fail(CHIMERA_E_FORMAT, "%s: truncated header", path);
  FileHeader hd;
  std::memcpy(&hd, head.data(), sizeof hd);
  if (std::memcmp(hd.magic, kMagic, 8) != 0) return fail(CHIMERA_E_FORMAT, "%s: bad magic", path);
  if (hd.version != kVersion) return fail(CHIMERA_E_FORMAT, "%s: version %u, expected %u", path, hd.version, kVersion);
  if (hd.header_bytes != 1024 || hd.nsections != NSEC)
    return fail(CHIMERA_E_FORMAT, "%s: bad header layout", path);
  if (hd.dim != CHIMERA_DIM || (hd.nbits != 2 && hd.nbits != 4) || hd.ncent < 1 || hd.ndocs < 0 || hd.ntok < 0 ||
      hd.nnz < 0 || hd.max_doc_len < 0)
    return fail(CHIMERA_E_FORMAT, "%s: bad sizes", path);
  h.dim = hd.dim; h.nbits = hd.nbits; h.ncent = hd.ncent; h.max_doc_len = hd.max_doc_len;
  h.ndocs = hd.ndocs; h.ntok = hd.ntok; h.nnz = hd.nnz;
  const uint64_t expect[NSEC] = {
      (uint64_t)h.ncent * h.dim * 2, (uint64_t)(h.ndocs + 1) * 8, (uint64_t)h.ntok * 4,
      (uint64_t)h.ntok * (uint64_t)h.code_bytes(), (uint64_t)((1 << h.nbits) - 1) * 4, (uint64_t)(1 << h.nbits) * 2,
      (uint64_t)(h.ncent + 1) * 8, (uint64_t)h.nnz * 4};
  for (int i = 0; i < NSEC; ++i)
    if (hd.sec[i].id != (uint32_t)(i + 1) || hd.sec[i].bytes != expect[i] || hd.sec[i].offset % 256 != 0)
      return fail(CHIMERA_E_FORMAT, "%s: section %d has wrong size or offset", path, i + 1);
  try {
    h.cent.resize(expect[0] / 2); h.doc_off.resize(expect[1] / 8); h.cid.resize(expect[2] / 4);
    h.codes.resize(expect[3]); h.cut_k.resize(expect[4] / 4); h.weights.resize(expect[5] / 2);
    h.ivf_off.resize(expect[6] / 8); h.ivf_doc.resize(expect[7] / 4);
  } catch (...) {
    return fail(CHIMERA_E_NOMEM, "%s: host allocation failed", path);
  }
  for (int i = 0; i < NSEC; ++i) {
    const void *p; uint64_t bytes;
    section_view(h, i + 1, p, bytes);
    if (std::fseek(f, (long)hd.sec[i].offset, SEEK_SET) != 0 ||
        std::fread(const_cast<void *>(p), 1, bytes, f) != bytes)
      return fail(CHIMERA_E_FORMAT, "%s: section %d truncated", path, i + 1);
    if (fnv64(p, bytes) != hd.sec[i].checksum) return fail(CHIMERA_E_FORMAT, "%s: section %d checksum mismatch", path, i + 1);
  }
  // structural checks the kernels rely on
  if (h.doc_off[0] != 0 || h.doc_off[h.ndocs] != h.ntok || h.ivf_off[0] != 0 || h.ivf_off[h.ncent] != h.nnz)
    return fail(CHIMERA_E_FORMAT, "%s: inconsistent offsets", path);
  for (int64_t v = 0; v < h.ndocs; ++v) {
    int64_t len = h.doc_off[v + 1] - h.doc_off[v];
    if (len < 1 || len > h.max_doc_len) return fail(CHIMERA_E_FORMAT, "%s: bad document length", path);
  }
  for (int32_t c = 0; c < h.ncent; ++c)
    if (h.ivf_off[c + 1] < h.ivf_off[c]) return fail(CHIMERA_E_FORMAT, "%s: bad posting offsets", path);
  for (int64_t t = 0; t < h.ntok; ++t)
    if ((uint32_t)h.cid[t] >= (uint32_t)h.ncent) return fail(CHIMERA_E_FORMAT, "%s: centroid id out of range", path);
  for (int64_t p = 0; p < h.nnz; ++p)
    if ((uint64_t)h.ivf_doc[p] >= (uint64_t)h.ndocs) return fail(CHIMERA_E_FORMAT, "%s: posting doc out of range", path);
  // the candidate walk relies on every list being strictly ascending
  for (int32_t c = 0; c < h.ncent; ++c)
    for (int64_t p = h.ivf_off[c] + 1; p < h.ivf_off[c + 1]; ++p)
      if (h.ivf_doc[p] <= h.ivf_doc[p - 1]) return fail(CHIMERA_E_FORMAT, "%s: posting list %d not ascending", path, c);
  return CHIMERA_OK;
}

void token_lists(const HostIndex &h, std::vector<int64_t> &tok_off, std::vector<int32_t> &ivf_tok,
                 std::vector<int32_t> &tok_doc) {
  tok_off.assign((size_t)h.ncent + 1, 0);
  for (int64_t t = 0; t < h.ntok; ++t) tok_off[(size_t)h.cid[t] + 1]++;
  for (int32_t c = 0; c < h.ncent; ++c) tok_off[c + 1] += tok_off[c];
  std::vector<int64_t> fill(tok_off.begin(), tok_off.end() - 1);
  ivf_tok.resize((size_t)h.ntok);
  for (int64_t t = 0; t < h.ntok; ++t) ivf_tok[fill[h.cid[t]]++] = (int32_t)t;  // ascending within a list
  tok_doc.resize((size_t)h.ntok);
  parallel_for(h.ndocs, [&](int64_t a, int64_t e) {
    for (int64_t v = a; v < e; ++v)
      for (int64_t t = h.doc_off[v]; t < h.doc_off[v + 1]; ++t) tok_doc[t] = (int32_t)v;
  });
}

int dense_lists(const HostIndex &h, std::vector<int8_t> &slot, std::vector<uint64_t> &doc_mask, int &ndense) {
  slot.assign(h.ncent, -1);
  doc_mask.clear();
  ndense = 0;
  std::vector<int32_t> cand;
  for (int32_t c = 0; c < h.ncent; ++c)
    if ((h.ivf_off[c + 1] - h.ivf_off[c]) * 16 > h.ndocs) cand.push_back(c);
  std::sort(cand.begin(), cand.end(), [&](int32_t a, int32_t b) {
    const int64_t la = h.ivf_off[a + 1] - h.ivf_off[a], lb = h.ivf_off[b + 1] - h.ivf_off[b];
    return la != lb ? la > lb : a < b;
  });
  if ((int)cand.size() > kMaxDense) cand.resize(kMaxDense);
  ndense = (int)cand.size();
  if (!ndense) return CHIMERA_OK;
  for (int i = 0; i < ndense; ++i) slot[cand[i]] = (int8_t)i;
  doc_mask.assign(h.ndocs, 0);
  parallel_for(h.ndocs, [&](int64_t a, int64_t e) {
    for (int64_t v = a; v < e; ++v) {
      uint64_t m = 0;
      for (int64_t t = h.doc_off[v]; t < h.doc_off[v + 1]; ++t) {
        const int sl = slot[h.cid[t]];
        if (sl >= 0) m |= 1ull << sl;
      }
      doc_mask[v] = m;
    }
  });
  // every dense list must hold exactly the documents whose mask has its bit
  std::vector<int64_t> count(ndense, 0);
  for (int64_t v = 0; v < h.ndocs; ++v)
    for (uint64_t m = doc_mask[v]; m; m &= m - 1) ++count[__builtin_ctzll(m)];
  for (int i = 0; i < ndense; ++i)
    if (count[i] != h.ivf_off[cand[i] + 1] - h.ivf_off[cand[i]])
      return fail(CHIMERA_E_FORMAT, "posting list %d does not match the token assignment", cand[i]);
  return CHIMERA_OK;
}

}  // namespace chimera

using namespace chimera;

// ---------------------------------------------------------------- builder
struct chimera_builder {
  HostIndex h;
  std::vector<int16_t> cent_k;   // grid integers [ncent][dim]
  std::vector<int64_t> hist;     // residual histogram, bins -4096..4096
  std::vector<int32_t> w_k;      // bucket weights, grid integers
  bool frozen = false;
  bool lists_built = false;
};

// bf16 bit patterns -> grid integers k = x * 2^11 (nearest, ties to even,
// which is grid_k_of_float for bf16 inputs: above 2^-4 a bf16 value is
// already a multiple of 2^-11).  Returns false if a value lies outside
// [-1, 1] (NaN included); out is then unspecified.
__attribute__((target_clones("avx512bw", "avx2", "default")))
static bool grid_rows(const uint16_t *bf16, int64_t n, int16_t *out) {
  bool ok = true;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t u = (uint32_t)bf16[i] << 16;
    float f;
    std::memcpy(&f, &u, 4);
    const bool in = std::fabs(f) <= 1.0f;
    // 1.5 * 2^23 has unit spacing: adding and removing it rounds f * 2^11
    // (exact, |f * 2^11| <= 2^11) to the nearest integer, ties to even
    const float r = (f * 2048.0f + 12582912.0f) - 12582912.0f;
    out[i] = (int16_t)(in ? r : 0.0f);
    ok &= in;
  }
  return ok;
}

// Residual histogram of ntok tokens: hist[r + 4096] counts residual
// components r = k_token - k_centroid.  Returns false on a value outside
// [-1, 1].
static bool residual_hist_rows(const uint16_t *tok, const int32_t *cids, int64_t ntok, const int16_t *cent_k,
                               int dim, int64_t *hist) {
  int16_t row[CHIMERA_DIM];
  for (int64_t t = 0; t < ntok; ++t) {
    if (!grid_rows(tok + t * dim, dim, row)) return false;
    const int16_t *c = cent_k + (size_t)cids[t] * dim;
    for (int d = 0; d < dim; ++d) hist[row[d] - c[d] + 4096]++;
  }
  return true;
}

// Packed codes of ntok tokens (2-bit: dim 4i+s in bits [2s, 2s+1] of byte i;
// 4-bit: dim 2i in the low nibble, 2i+1 in the high one).  code(r) is the
// number of cutoffs strictly below r.  Returns false on a value outside
// [-1, 1].
__attribute__((target_clones("avx512bw", "avx2", "default")))
static bool encode_rows(const uint16_t *tok, const int32_t *cids, int64_t ntok, const int16_t *cent_k, int dim,
                        const int16_t *cut, int ncut, int nbits, uint8_t *out) {
  int16_t row[CHIMERA_DIM];
  uint8_t code[CHIMERA_DIM];
  const int cb = dim * nbits / 8;
  for (int64_t t = 0; t < ntok; ++t) {
    if (!grid_rows(tok + t * dim, dim, row)) return false;
    const int16_t *c = cent_k + (size_t)cids[t] * dim;
    for (int d = 0; d < dim; ++d) row[d] = (int16_t)(row[d] - c[d]);
    for (int d = 0; d < dim; ++d) code[d] = 0;
    for (int i = 0; i < ncut; ++i)
      for (int d = 0; d < dim; ++d) code[d] += cut[i] < row[d];
    uint8_t *o = out + t * cb;
    if (nbits == 2)
      for (int i = 0; i < cb; ++i)
        o[i] = (uint8_t)(code[4 * i] | code[4 * i + 1] << 2 | code[4 * i + 2] << 4 | code[4 * i + 3] << 6);
    else
      for (int i = 0; i < cb; ++i) o[i] = (uint8_t)(code[2 * i] | code[2 * i + 1] << 4);
  }
  return true;
}

// floor(num * n / den)-th smallest residual (0-based, clamped to n-1)
static int32_t quantile_k(const std::vector<int64_t> &hist, int64_t n, int64_t num, int64_t den) {
  int64_t target = std::min<int64_t>((num * n) / den, n - 1), seen = 0;
  for (int b = 0; b < 8193; ++b) {
    seen += hist[b];
    if (seen > target) return b - 4096;
  }
  return 4096;
}

void chimera::ivf_lists(HostIndex &h) {
  std::vector<int64_t> last(h.ncent, -1), cnt(h.ncent + 1, 0);
  for (int64_t v = 0; v < h.ndocs; ++v)
    for (int64_t t = h.doc_off[v]; t < h.doc_off[v + 1]; ++t) {
      int32_t c = h.cid[t];
      if (last[c] != v) { last[c] = v; cnt[c + 1]++; }
    }
  for (int32_t c = 0; c < h.ncent; ++c) cnt[c + 1] += cnt[c];
  h.nnz = cnt[h.ncent];
  h.ivf_off = cnt;
  h.ivf_doc.assign(h.nnz, 0);
  std::fill(last.begin(), last.end(), -1);
  for (int64_t v = 0; v < h.ndocs; ++v)
    for (int64_t t = h.doc_off[v]; t < h.doc_off[v + 1]; ++t) {
      int32_t c = h.cid[t];
      if (last[c] != v) { last[c] = v; h.ivf_doc[cnt[c]++] = (int32_t)v; }
    }
}

static void build_lists(chimera_builder *b) {
  if (b->lists_built) return;
  chimera::ivf_lists(b->h);
  b->lists_built = true;
}

extern "C" {

int chimera_builder_create(const uint16_t *centroids_bf16, int32_t ncent, int32_t dim, int32_t nbits,
                           chimera_builder **out) {
  if (!out || !centroids_bf16) return fail(CHIMERA_E_INVAL, "null argument");
  if (dim != CHIMERA_DIM) return fail(CHIMERA_E_UNSUPPORTED, "dim %d: only %d is supported", dim, CHIMERA_DIM);
  if (nbits != 2 && nbits != 4) return fail(CHIMERA_E_INVAL, "nbits must be 2 or 4");
  if (ncent < 1) return fail(CHIMERA_E_INVAL, "ncent must be >= 1");
  chimera_builder *b = new (std::nothrow) chimera_builder;
  if (!b) return fail(CHIMERA_E_NOMEM, "builder allocation");
  try {
    b->h.ncent = ncent; b->h.dim = dim; b->h.nbits = nbits;
    b->cent_k.resize((size_t)ncent * dim);
    b->hist.assign(8193, 0);
    b->h.doc_off.assign(1, 0);
  } catch (...) {
    delete b;
    return fail(CHIMERA_E_NOMEM, "builder allocation");
  }
  if (!grid_rows(centroids_bf16, (int64_t)ncent * dim, b->cent_k.data())) {
    delete b;
    return fail(CHIMERA_E_INVAL, "centroid components must lie in [-1, 1]");
  }
  b->h.cent.resize((size_t)ncent * dim);
  for (size_t i = 0; i < b->cent_k.size(); ++i) b->h.cent[i] = bf16_of_grid_k(b->cent_k[i]);
  *out = b;
  return CHIMERA_OK;
}

int chimera_builder_add_residuals(chimera_builder *b, const uint16_t *tokens_bf16, const int32_t *cids,
                                  int64_t ntok) {
  if (!b || (ntok > 0 && (!tokens_bf16 || !cids)) || ntok < 0) return fail(CHIMERA_E_INVAL, "bad argument");
  if (b->frozen) return fail(CHIMERA_E_INVAL, "quantiser already frozen");
  const int dim = b->h.dim, ncent = b->h.ncent;
  for (int64_t t = 0; t < ntok; ++t)
    if ((uint32_t)cids[t] >= (uint32_t)ncent) return fail(CHIMERA_E_INVAL, "cid out of range at token %lld", (long long)t);
  // per-thread histograms, merged only when every token was valid, so a
  // rejected call leaves the builder as it was
  std::vector<std::vector<int64_t>> part;
  std::mutex mu;
  std::atomic<bool> bad{false};
  parallel_for(ntok, [&](int64_t a, int64_t e) {
    std::vector<int64_t> hloc(8193, 0);
    if (!residual_hist_rows(tokens_bf16 + a * dim, cids + a, e - a, b->cent_k.data(), dim, hloc.data())) bad = true;
    std::lock_guard<std::mutex> g(mu);
    part.push_back(std::move(hloc));
  });
  if (bad) return fail(CHIMERA_E_INVAL, "token components must lie in [-1, 1]");
  for (const auto &hp : part)
    for (int i = 0; i < 8193; ++i) b->hist[i] += hp[i];
  return CHIMERA_OK;
}

int chimera_builder_freeze_quantizer(chimera_builder *b) {
  if (!b) return fail(CHIMERA_E_INVAL, "null builder");
  if (b->frozen) return CHIMERA_OK;
  int64_t n = 0;
  for (int64_t x : b->hist) n += x;
  if (n == 0) return fail(CHIMERA_E_INVAL, "no residuals were added");
  const int B = 1 << b->h.nbits;
  b->h.cut_k.resize(B - 1);
  b->w_k.resize(B);
  b->h.weights.resize(B);
  for (int i = 1; i < B; ++i) b->h.cut_k[i - 1] = quantile_k(b->hist, n, i, B);
  for (int u = 0; u < B; ++u) {
    int32_t r = quantile_k(b->hist, n, 2 * u + 1, 2 * B);
    b->w_k[u] = grid_k_of_float((float)r / 2048.0f);  // exact: |r| <= 4096
    b->h.weights[u] = bf16_of_grid_k(b->w_k[u]);
  }
  b->frozen = true;
  return CHIMERA_OK;
}

int chimera_builder_add_docs(chimera_builder *b, const uint16_t *tokens_bf16, const int32_t *cids,
                             const int32_t *doc_lens, int64_t ndocs) {
  if (!b || ndocs < 0 || (ndocs > 0 && (!tokens_bf16 || !cids || !doc_lens))) return fail(CHIMERA_E_INVAL, "bad argument");
  if (!b->frozen) return fail(CHIMERA_E_INVAL, "freeze the quantiser before adding documents");
  HostIndex &h = b->h;
  const int dim = h.dim, nbits = h.nbits, ncut = (1 << nbits) - 1;
  const int64_t cb = h.code_bytes();
  int64_t rows = 0;
  int32_t longest = 0;
  for (int64_t i = 0; i < ndocs; ++i) {
    if (doc_lens[i] < 1) return fail(CHIMERA_E_INVAL, "document %lld has no token", (long long)i);
    rows += doc_lens[i];
    longest = std::max(longest, doc_lens[i]);
  }
  for (int64_t t = 0; t < rows; ++t)
    if ((uint32_t)cids[t] >= (uint32_t)h.ncent) return fail(CHIMERA_E_INVAL, "cid out of range at token %lld", (long long)t);
  const int64_t t0 = h.ntok;
  const size_t ndoc_off = h.doc_off.size();
  // every section grows first and is cut back if a token is rejected, so a
  // failed call leaves the builder exactly as it was
  auto roll_back = [&] {
    h.cid.resize(t0);
    h.codes.resize(t0 * cb);
    h.doc_off.resize(ndoc_off);
    if (h.rq) {
      h.rq_bits.resize(t0 * (dim / 8));
      h.rq_codes.resize(t0 * (dim / 2));
      h.rq_g1.resize(t0);
      h.rq_g4.resize(t0);
    }
  };
  try {
    h.cid.resize(t0 + rows);
    h.codes.resize((t0 + rows) * cb);
    h.doc_off.reserve(ndoc_off + ndocs);
    if (h.rq) {
      h.rq_bits.resize((t0 + rows) * (dim / 8));
      h.rq_codes.resize((t0 + rows) * (dim / 2));
      h.rq_g1.resize(t0 + rows);
      h.rq_g4.resize(t0 + rows);
    }
  } catch (...) {
    roll_back();
    return fail(CHIMERA_E_NOMEM, "host allocation for %lld tokens", (long long)rows);
  }
  int16_t cut[15];
  for (int i = 0; i < ncut; ++i) cut[i] = (int16_t)h.cut_k[i];
  std::atomic<bool> bad{false};
  parallel_for(rows, [&](int64_t a, int64_t e) {
    if (!encode_rows(tokens_bf16 + a * dim, cids + a, e - a, b->cent_k.data(), dim, cut, ncut, nbits,
                     h.codes.data() + (t0 + a) * cb))
      bad = true;
  });
  if (bad) {
    roll_back();
    return fail(CHIMERA_E_INVAL, "token components must lie in [-1, 1]");
  }
  if (h.rq) {  // the tokens are valid: their RaBitQ codes
    parallel_for(rows, [&](int64_t a, int64_t e) {
      std::vector<int16_t> kk((size_t)(e - a) * dim);
      grid_rows(tokens_bf16 + a * dim, (e - a) * dim, kk.data());
      rabitq_encode_rows(kk.data(), e - a, dim, h.rq_signs.data(), h.rq_bits.data() + (t0 + a) * (dim / 8),
                         h.rq_g1.data() + t0 + a, h.rq_codes.data() + (t0 + a) * (dim / 2), h.rq_g4.data() + t0 + a);
    });
  }
  std::memcpy(h.cid.data() + t0, cids, rows * 4);
  for (int64_t i = 0; i < ndocs; ++i) h.doc_off.push_back(h.doc_off.back() + doc_lens[i]);
  h.max_doc_len = std::max(h.max_doc_len, longest);
  h.ntok = t0 + rows;
  h.ndocs += ndocs;
  b->lists_built = false;
  return CHIMERA_OK;
}

int chimera_builder_rabitq(chimera_builder *b, const int8_t *signs) {
  if (!b || !signs) return fail(CHIMERA_E_INVAL, "null argument");
  if (b->h.ntok > 0) return fail(CHIMERA_E_INVAL, "enable RaBitQ codes before adding documents");
  for (int d = 0; d < b->h.dim; ++d)
    if (signs[d] != 1 && signs[d] != -1) return fail(CHIMERA_E_INVAL, "sign %d is %d, not +1 or -1", d, signs[d]);
  b->h.rq = true;
  b->h.rq_signs.assign(signs, signs + b->h.dim);
  return CHIMERA_OK;
}

int chimera_builder_reserve(chimera_builder *b, int64_t ndocs, int64_t ntok) {
  if (!b || ndocs < 0 || ntok < 0) return fail(CHIMERA_E_INVAL, "bad argument");
  HostIndex &h = b->h;
  try {
    h.doc_off.reserve((size_t)ndocs + 1);
    h.cid.reserve((size_t)ntok);
    h.codes.reserve((size_t)ntok * (size_t)h.code_bytes());
  } catch (...) {
    return fail(CHIMERA_E_NOMEM, "host allocation for %lld tokens", (long long)ntok);
  }
  return CHIMERA_OK;
}

int chimera_builder_quantizer(const chimera_builder *b, int32_t *cut_k, uint16_t *weights_bf16) {
  if (!b) return fail(CHIMERA_E_INVAL, "null builder");
  if (!b->frozen) return fail(CHIMERA_E_INVAL, "quantiser not frozen");
  if (cut_k) std::memcpy(cut_k, b->h.cut_k.data(), b->h.cut_k.size() * 4);
  if (weights_bf16) std::memcpy(weights_bf16, b->h.weights.data(), b->h.weights.size() * 2);
  return CHIMERA_OK;
}

int chimera_builder_save(const chimera_builder *b, const char *path) {
  if (!b || !path) return fail(CHIMERA_E_INVAL, "null argument");
  if (!b->frozen) return fail(CHIMERA_E_INVAL, "quantiser not frozen");
  if (b->h.rq) return fail(CHIMERA_E_UNSUPPORTED, "index files do not hold RaBitQ codes");
  build_lists(const_cast<chimera_builder *>(b));
  return save_index(b->h, path);
}

int chimera_builder_sections(const chimera_builder *b, int64_t *doc_off, int32_t *cid, uint8_t *codes,
                             int64_t *ivf_off, int32_t *ivf_doc) {
  if (!b) return fail(CHIMERA_E_INVAL, "null builder");
  build_lists(const_cast<chimera_builder *>(b));
  const HostIndex &h = b->h;
  if (doc_off) std::memcpy(doc_off, h.doc_off.data(), h.doc_off.size() * 8);
  if (cid) std::memcpy(cid, h.cid.data(), h.cid.size() * 4);
  if (codes) std::memcpy(codes, h.codes.data(), h.codes.size());
  if (ivf_off) std::memcpy(ivf_off, h.ivf_off.data(), h.ivf_off.size() * 8);
  if (ivf_doc) std::memcpy(ivf_doc, h.ivf_doc.data(), h.ivf_doc.size() * 4);
  return CHIMERA_OK;
}

int chimera_builder_rabitq_sections(const chimera_builder *b, uint8_t *bits1, float *g1, uint8_t *codes4,
                                    float *g4) {
  if (!b) return fail(CHIMERA_E_INVAL, "null builder");
  const HostIndex &h = b->h;
  if (!h.rq) return fail(CHIMERA_E_INVAL, "the builder has no RaBitQ codes");
  if (bits1) std::memcpy(bits1, h.rq_bits.data(), h.rq_bits.size());
  if (g1) std::memcpy(g1, h.rq_g1.data(), h.rq_g1.size() * 4);
  if (codes4) std::memcpy(codes4, h.rq_codes.data(), h.rq_codes.size());
  if (g4) std::memcpy(g4, h.rq_g4.data(), h.rq_g4.size() * 4);
  return CHIMERA_OK;
}

int chimera_builder_info(const chimera_builder *b, chimera_index_info *out) {
  if (!b || !out) return fail(CHIMERA_E_INVAL, "null argument");
  build_lists(const_cast<chimera_builder *>(b));
  const HostIndex &h = b->h;
  out->ndocs = h.ndocs; out->ntokens = h.ntok; out->nnz = h.nnz; out->ncent = h.ncent; out->dim = h.dim;
  out->nbits = h.nbits; out->max_doc_len = h.max_doc_len; out->device = -1; out->q_norm_limit = 0.0; out->ndeleted = 0;
  out->device_bytes = (int64_t)(h.cent.size() * 2 + h.doc_off.size() * 8 + h.cid.size() * 4 + h.codes.size() +
                                h.ivf_off.size() * 8 + h.ivf_doc.size() * 4);
  return CHIMERA_OK;
}

void chimera_builder_free(chimera_builder *b) { delete b; }

}  // extern "C"

namespace chimera {
const HostIndex *builder_host(const chimera_builder *b) {
  build_lists(const_cast<chimera_builder *>(b));
  return &b->h;
}
}  // namespace chimera
