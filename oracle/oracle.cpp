// CPU oracle for the EmbeddingBag training step.
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
// the benchmark's CPU-baseline leg may load or call this library; the product
// path never does.  It shares no source with the GPU library.
//
// Plain single-threaded loops, written from the paper's definitions:
//   * Section II: an embedding look-up over a minibatch is L = A^T W, where
//     column n of the sparse matrix A holds the multiplicity of every row
//     that bag n reads, and whole rows of W are read.
//   * Section III-A, Algorithm 1 (forward, sum pooling): Y[n] starts at zero
//     and accumulates W[I[s]] for s in [O[n], O[n+1]).
//   * Algorithm 2 (backward): the per-look-up gradient dW[s] = dY[bag of s].
//   * Algorithms 3/4 (sparse SGD update): every look-up adds alpha * dW[s]
//     to row I[s], with alpha = -lr; all contributions to a row are summed.
//     The fused backward+update (end of Section III-A) gives the same rows.
//   * Section VII (Split-SGD-BF16): an FP32 weight is kept as its 16 most
//     significant bits (a BF16 number, used by forward/backward) and its 16
//     least significant bits (used only by the update, which recombines the
//     two halves, applies SGD in FP32 and splits the result again).
//
// Accumulation is FP64, rounded once to FP32, so the reference value is the
// exact sum up to one rounding.  Readings of the paper's silent or garbled
// points (sizes of I and O in Algorithm 1, half-open loops, the update sign,
// empty bags, invalid inputs, truncation for the BF16 half) follow the
// project's design notes; each is restated beside the code that applies it.
//
// Build: g++ -O2 -std=c++17 -fno-fast-math -ffp-contract=off -shared -fPIC

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <vector>

namespace {

// Status codes of the EmbeddingBag boundary (same numbers as the library).
constexpr int kOk = 0;
constexpr int kErrInvalidArg = -1;
constexpr int kErrIndexRange = -3;
constexpr int kErrOffsets = -4;

constexpr int64_t kInt32Max = 2147483647;
// Indices and offsets are int32 (Algorithm 1's I[NS] and O[N+1], read as
// 32-bit integers), so a call holds at most 2^31 - 1 look-ups; more is an
// argument error.
constexpr int64_t kMaxIndices = kInt32Max;

// Argument checks, first in the fixed validation order.
int check_args(int32_t T, int32_t B, int32_t E, const int64_t* rows, int64_t NS) {
  if (T < 1 || T > 64) return kErrInvalidArg;
  if (E < 4 || E > 1024 || E % 4 != 0) return kErrInvalidArg;
  if (B < 0 || NS < 0 || NS > kMaxIndices) return kErrInvalidArg;
  if (rows == nullptr) return kErrInvalidArg;
  if (int64_t(T) * int64_t(B) + 1 > kInt32Max) return kErrInvalidArg;
  int64_t total = 0;
  for (int t = 0; t < T; ++t) {
    if (rows[t] < 1 || rows[t] > kInt32Max) return kErrInvalidArg;
    total += rows[t];
  }
  if (total > kInt32Max) return kErrInvalidArg;
  return kOk;
}

// Offsets: O has T*B + 1 entries, O[0] = 0, non-decreasing, O[T*B] = NS.
// (Algorithm 1's header swaps the sizes of I and O; the loops read O[n] and
// O[n+1] for n < N, so O has N + 1 entries and I has NS.)
int check_offsets(int64_t TB, const int32_t* O, int64_t NS) {
  if (O[0] != 0) return kErrOffsets;
  for (int64_t k = 0; k < TB; ++k)
    if (O[k] > O[k + 1]) return kErrOffsets;
  if (O[TB] != NS) return kErrOffsets;
  return kOk;
}

// Indices: every look-up of a bag of table t names a row in [0, M_t).
int check_indices(int32_t T, int32_t B, const int64_t* rows, const int32_t* I, const int32_t* O) {
  for (int64_t k = 0; k < int64_t(T) * B; ++k) {
    const int64_t m = rows[k / B];
    for (int64_t s = O[k]; s < O[k + 1]; ++s)
      if (I[s] < 0 || I[s] >= m) return kErrIndexRange;
  }
  return kOk;
}

int validate(int32_t T, int32_t B, int32_t E, const int64_t* rows, const int32_t* I,
             const int32_t* O, int64_t NS) {
  int rc = check_args(T, B, E, rows, NS);
  if (rc) return rc;
  if (O == nullptr || (NS > 0 && I == nullptr)) return kErrInvalidArg;
  rc = check_offsets(int64_t(T) * B, O, NS);
  if (rc) return rc;
  return check_indices(T, B, rows, I, O);
}

// The forward's output buffer: null is an argument error unless there is
// nothing to write (T*B = 0).  Checked after the sizes and the index and
// offsets pointers and before the data, so that the status matches the
// library's on the same arguments.
int check_out(int32_t T, int32_t B, int32_t E, const int64_t* rows, const int32_t* I,
              const int32_t* O, int64_t NS, const void* Y) {
  int rc = check_args(T, B, E, rows, NS);
  if (rc) return rc;
  if (O == nullptr || (NS > 0 && I == nullptr)) return kErrInvalidArg;
  if (int64_t(T) * B > 0 && Y == nullptr) return kErrInvalidArg;
  return kOk;
}

// The backward's gradient: null is an argument error when there is a
// look-up to update, checked before the data as the library does.
int check_grad(int32_t T, int32_t B, int32_t E, const int64_t* rows, const int32_t* I,
               const int32_t* O, int64_t NS, const void* dY) {
  int rc = check_args(T, B, E, rows, NS);
  if (rc) return rc;
  if (O == nullptr || (NS > 0 && I == nullptr)) return kErrInvalidArg;
  if (NS > 0 && dY == nullptr) return kErrInvalidArg;
  return kOk;
}

inline float bits_to_float(uint32_t u) {
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}
inline uint32_t float_to_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

// Row r of table t as FP32 values, either from an FP32 table or from the
// BF16 high half of a split table (the 16 most significant bits, shifted back
// into place; the low half is not read).
struct RowReader {
  const float* const* w = nullptr;
  const uint16_t* const* hi = nullptr;
  int32_t E = 0;
  float get(int t, int64_t r, int e) const {
    if (w) return w[t][r * E + e];
    return bits_to_float(uint32_t(hi[t][r * E + e]) << 16);
  }
};

// Algorithm 1 with FP64 accumulation: Y[k] = sum over the bag's look-ups of
// W_t[I[s]], zero for an empty bag; bag k = t*B + b belongs to table t.
int forward_impl(int32_t T, int32_t B, int32_t E, const int64_t* rows, const RowReader& W,
                 const int32_t* I, const int32_t* O, int64_t NS, float* Y) {
  int rc = check_out(T, B, E, rows, I, O, NS, Y);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  std::vector<double> acc(E);
  for (int64_t k = 0; k < int64_t(T) * B; ++k) {
    const int t = int(k / B);
    std::fill(acc.begin(), acc.end(), 0.0);
    for (int64_t s = O[k]; s < O[k + 1]; ++s)
      for (int e = 0; e < E; ++e) acc[e] += double(W.get(t, I[s], e));
    for (int e = 0; e < E; ++e) Y[k * E + e] = float(acc[e]);
  }
  return kOk;
}

// Look-ups grouped by table row: key[s] = rowbase[t] + I[s] where rowbase is
// the exclusive prefix sum of M_t, bag[s] = k for O[k] <= s < O[k+1]; a
// stable sort by key keeps the look-ups of one row in increasing s.
struct Dedup {
  std::vector<int64_t> rowbase;
  std::vector<uint32_t> key, bag, sorted_key, sorted_bag, unique_key;
  std::vector<int32_t> seg_off;
  std::vector<int64_t> perm;  // look-up position s of each sorted entry
};

void dedup_impl(int32_t T, int32_t B, const int64_t* rows, const int32_t* I, const int32_t* O,
                int64_t NS, Dedup& d) {
  d.rowbase.assign(T + 1, 0);
  for (int t = 0; t < T; ++t) d.rowbase[t + 1] = d.rowbase[t] + rows[t];
  d.key.resize(NS);
  d.bag.resize(NS);
  for (int64_t k = 0; k < int64_t(T) * B; ++k)
    for (int64_t s = O[k]; s < O[k + 1]; ++s) {
      d.bag[s] = uint32_t(k);
      d.key[s] = uint32_t(d.rowbase[k / B] + I[s]);
    }
  std::vector<int64_t> perm(NS);
  std::iota(perm.begin(), perm.end(), int64_t(0));
  std::stable_sort(perm.begin(), perm.end(),
                   [&](int64_t a, int64_t b) { return d.key[a] < d.key[b]; });
  d.perm = perm;
  d.sorted_key.resize(NS);
  d.sorted_bag.resize(NS);
  for (int64_t i = 0; i < NS; ++i) {
    d.sorted_key[i] = d.key[perm[i]];
    d.sorted_bag[i] = d.bag[perm[i]];
  }
  d.unique_key.clear();
  d.seg_off.clear();
  for (int64_t i = 0; i < NS; ++i)
    if (i == 0 || d.sorted_key[i] != d.sorted_key[i - 1]) {
      d.unique_key.push_back(d.sorted_key[i]);
      d.seg_off.push_back(int32_t(i));
    }
  d.seg_off.push_back(int32_t(NS));
}

int table_of_key(const Dedup& d, uint32_t key) {
  int t = 0;
  while (int64_t(key) >= d.rowbase[t + 1]) ++t;
  return t;
}

// Fused backward + SGD on the rows the batch touches: for row r of table t,
// G = sum over look-ups s with I[s] = r (in bags of t) of dY[bag(s)], and
// W_t[r] <- W_t[r] - lr * G; rows no look-up names keep their bits.
// The row is handed to `apply`, which does the FP32 (or split) write-back.
template <class Apply>
int backward_impl(const float* dY, int32_t T, int32_t B, int32_t E, const int64_t* rows,
                  const int32_t* I, const int32_t* O, int64_t NS, Apply apply) {
  int rc = check_grad(T, B, E, rows, I, O, NS, dY);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  Dedup d;
  dedup_impl(T, B, rows, I, O, NS, d);
  std::vector<double> acc(E);
  for (size_t u = 0; u < d.unique_key.size(); ++u) {
    std::fill(acc.begin(), acc.end(), 0.0);
    for (int64_t i = d.seg_off[u]; i < d.seg_off[u + 1]; ++i) {
      const float* g = dY + int64_t(d.sorted_bag[i]) * E;
      for (int e = 0; e < E; ++e) acc[e] += double(g[e]);
    }
    const int t = table_of_key(d, d.unique_key[u]);
    const int64_t r = int64_t(d.unique_key[u]) - d.rowbase[t];
    apply(t, r, acc.data());
  }
  return kOk;
}

}  // namespace

extern "C" {

int oracle_validate(int32_t T, int32_t B, int32_t E, const int64_t* rows, const int32_t* I,
                    const int32_t* O, int64_t NS) {
  return validate(T, B, E, rows, I, O, NS);
}

int oracle_forward(int32_t T, int32_t B, int32_t E, const int64_t* rows, const float* const* W,
                   const int32_t* I, const int32_t* O, int64_t NS, float* Y) {
  if (W == nullptr) return kErrInvalidArg;
  RowReader rd;
  rd.w = W;
  rd.E = E;
  return forward_impl(T, B, E, rows, rd, I, O, NS, Y);
}

int oracle_dedup(int32_t T, int32_t B, const int64_t* rows, const int32_t* I, const int32_t* O,
                 int64_t NS, uint32_t* sorted_keys, uint32_t* sorted_bags, uint32_t* unique_keys,
                 int32_t* seg_off, int64_t* num_unique) {
  int rc = validate(T, B, 4, rows, I, O, NS);
  if (rc) return rc;
  Dedup d;
  dedup_impl(T, B, rows, I, O, NS, d);
  std::copy(d.sorted_key.begin(), d.sorted_key.end(), sorted_keys);
  std::copy(d.sorted_bag.begin(), d.sorted_bag.end(), sorted_bags);
  std::copy(d.unique_key.begin(), d.unique_key.end(), unique_keys);
  std::copy(d.seg_off.begin(), d.seg_off.end(), seg_off);
  *num_unique = int64_t(d.unique_key.size());
  return kOk;
}

int oracle_backward_sgd(const float* dY, int32_t T, int32_t B, int32_t E, const int64_t* rows,
                        float* const* W, const int32_t* I, const int32_t* O, int64_t NS,
                        float lr) {
  if (W == nullptr) return kErrInvalidArg;
  return backward_impl(dY, T, B, E, rows, I, O, NS, [&](int t, int64_t r, const double* g) {
    float* w = W[t] + r * E;
    for (int e = 0; e < E; ++e) w[e] = float(double(w[e]) - double(lr) * g[e]);
  });
}

// Section VII storage: hi = 16 most significant bits (a BF16 number by
// truncation), lo = 16 least significant bits, as two separate arrays.
void oracle_split(const float* w, uint16_t* hi, uint16_t* lo, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t u = float_to_bits(w[i]);
    hi[i] = uint16_t(u >> 16);
    lo[i] = uint16_t(u & 0xFFFFu);
  }
}

void oracle_combine(const uint16_t* hi, const uint16_t* lo, float* w, int64_t n) {
  for (int64_t i = 0; i < n; ++i) w[i] = bits_to_float((uint32_t(hi[i]) << 16) | lo[i]);
}

// Count of bit patterns u in [start, start+count) with combine(split(u)) != u.
int64_t oracle_split_roundtrip_mismatches(uint64_t start, uint64_t count) {
  int64_t bad = 0;
  for (uint64_t v = start; v < start + count; ++v) {
    const float f = bits_to_float(uint32_t(v));
    uint16_t h, l;
    oracle_split(&f, &h, &l, 1);
    float g;
    oracle_combine(&h, &l, &g, 1);
    if (float_to_bits(g) != uint32_t(v)) ++bad;
  }
  return bad;
}

// Forward of Section VII: Algorithm 1 on the BF16 high halves only.
int oracle_forward_split(int32_t T, int32_t B, int32_t E, const int64_t* rows,
                         const uint16_t* const* hi, const int32_t* I, const int32_t* O, int64_t NS,
                         float* Y) {
  if (hi == nullptr) return kErrInvalidArg;
  RowReader rd;
  rd.hi = hi;
  rd.E = E;
  return forward_impl(T, B, E, rows, rd, I, O, NS, Y);
}

// Update of Section VII: recombine hi and lo into the FP32 weight, apply the
// FP32 update of oracle_backward_sgd, split the result again.
int oracle_backward_sgd_split(const float* dY, int32_t T, int32_t B, int32_t E,
                              const int64_t* rows, uint16_t* const* hi, uint16_t* const* lo,
                              const int32_t* I, const int32_t* O, int64_t NS, float lr) {
  if (hi == nullptr || lo == nullptr) return kErrInvalidArg;
  return backward_impl(dY, T, B, E, rows, I, O, NS, [&](int t, int64_t r, const double* g) {
    uint16_t* h = hi[t] + r * E;
    uint16_t* l = lo[t] + r * E;
    for (int e = 0; e < E; ++e) {
      float w;
      oracle_combine(h + e, l + e, &w, 1);
      w = float(double(w) - double(lr) * g[e]);
      oracle_split(&w, h + e, l + e, 1);
    }
  });
}

// ---- BF16 activations.  Section VII runs the forward and backward passes in
// ---- BF16 and keeps FP32 only for the weight update; a BF16 number is an
// ---- FP32 value whose 16 low bits are zero.

// FP32 -> BF16 by round to nearest, ties to even, from its definition: of the
// two BF16 neighbours of x (x truncated toward zero, and the next BF16 away
// from zero) take the nearer; on a tie the one whose last bit is 0.  Past the
// largest finite BF16 the upper neighbour is infinity, placed at 2^128 for the
// comparison (the value the next binade would start at), as IEEE 754 rounding
// does.  NaN stays NaN (quiet).
void oracle_bf16_round(const float* x, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    const float f = x[i];
    const uint32_t u = float_to_bits(f);
    if (std::isnan(f)) {
      out[i] = uint16_t((u >> 16) | 0x40u);
      continue;
    }
    const uint32_t down = u & 0xFFFF0000u;
    if (down == u) {  // already a BF16 number (zeros and infinities included)
      out[i] = uint16_t(down >> 16);
      continue;
    }
    const uint32_t up = down + 0x10000u;  // next in magnitude, same sign
    const double vd = double(bits_to_float(down));
    const double vu = (up & 0x7FFFFFFFu) == 0x7F800000u ? std::copysign(std::ldexp(1.0, 128), f)
                                                         : double(bits_to_float(up));
    const double dd = std::fabs(double(f) - vd), du = std::fabs(vu - double(f));
    uint32_t pick;
    if (dd < du)
      pick = down;
    else if (du < dd)
      pick = up;
    else
      pick = ((down >> 16) & 1u) == 0 ? down : up;
    out[i] = uint16_t(pick >> 16);
  }
}

// BF16 -> FP32 is exact: the 16 bits become the high half.
void oracle_bf16_widen(const uint16_t* h, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = bits_to_float(uint32_t(h[i]) << 16);
}

// Forward of Section VII with BF16 pooled outputs: the FP32 pooled sums of
// oracle_forward_split, each rounded to BF16.
int oracle_forward_split_bf16_act(int32_t T, int32_t B, int32_t E, const int64_t* rows,
                                  const uint16_t* const* hi, const int32_t* I, const int32_t* O,
                                  int64_t NS, uint16_t* Y) {
  if (hi == nullptr) return kErrInvalidArg;
  int rc = check_out(T, B, E, rows, I, O, NS, Y);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  std::vector<float> y(size_t(T) * size_t(B) * size_t(E), 0.0f);
  rc = oracle_forward_split(T, B, E, rows, hi, I, O, NS, y.data());
  if (rc) return rc;
  oracle_bf16_round(y.data(), Y, int64_t(y.size()));
  return kOk;
}

// Update of Section VII driven by a BF16 gradient of the pooled output: the
// gradient is widened to FP32, then oracle_backward_sgd_split applies.
int oracle_backward_sgd_split_bf16_act(const uint16_t* dY, int32_t T, int32_t B, int32_t E,
                                       const int64_t* rows, uint16_t* const* hi,
                                       uint16_t* const* lo, const int32_t* I, const int32_t* O,
                                       int64_t NS, float lr) {
  if (hi == nullptr || lo == nullptr) return kErrInvalidArg;
  int rc = check_grad(T, B, E, rows, I, O, NS, dY);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  const int64_t n = int64_t(T) * B * E;
  std::vector<float> g(static_cast<size_t>(n));
  if (n > 0 && dY != nullptr) oracle_bf16_widen(dY, g.data(), n);
  return oracle_backward_sgd_split(dY != nullptr ? g.data() : nullptr, T, B, E, rows, hi, lo, I,
                                   O, NS, lr);
}

// ---- Literal readings, kept only to show how far FP32 sequential order
// ---- lands from the FP64 definition (never used as the reference).

// Algorithm 1 as printed: FP32 accumulator, look-ups in increasing s.
int oracle_forward_literal(int32_t T, int32_t B, int32_t E, const int64_t* rows,
                           const float* const* W, const int32_t* I, const int32_t* O, int64_t NS,
                           float* Y) {
  if (W == nullptr) return kErrInvalidArg;
  int rc = check_out(T, B, E, rows, I, O, NS, Y);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  for (int64_t k = 0; k < int64_t(T) * B; ++k) {
    float* y = Y + k * E;
    for (int e = 0; e < E; ++e) y[e] = 0.0f;
    for (int64_t s = O[k]; s < O[k + 1]; ++s)
      for (int e = 0; e < E; ++e) y[e] += W[k / B][int64_t(I[s]) * E + e];
  }
  return kOk;
}

// Algorithm 2 (materialised dW[NS][E]) then Algorithm 3 applied one look-up
// at a time in increasing i, in FP32, with alpha = -lr.  Within one row this
// is also the order Algorithm 4's owning thread uses.
int oracle_backward_sgd_literal(const float* dY, int32_t T, int32_t B, int32_t E,
                                const int64_t* rows, float* const* W, const int32_t* I,
                                const int32_t* O, int64_t NS, float lr) {
  if (W == nullptr) return kErrInvalidArg;
  int rc = check_grad(T, B, E, rows, I, O, NS, dY);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  std::vector<float> dW(size_t(NS) * E, 0.0f);
  for (int64_t k = 0; k < int64_t(T) * B; ++k)
    for (int64_t s = O[k]; s < O[k + 1]; ++s)
      for (int e = 0; e < E; ++e) dW[s * E + e] += dY[k * E + e];
  const float alpha = -lr;
  for (int64_t k = 0; k < int64_t(T) * B; ++k)
    for (int64_t i = O[k]; i < O[k + 1]; ++i) {
      float* w = W[k / B] + int64_t(I[i]) * E;
      for (int e = 0; e < E; ++e) {
        const float step = alpha * dW[i * E + e];
        w[e] = w[e] + step;
      }
    }
  return kOk;
}

// ---- Weighted and mean pooling (Section II's general L = A^T W) ----------
// Column n of A holds a weight a_p for every row bag n reads.  With weights
// `a` (one per look-up; null means all ones) and sum pooling,
//   Y[k] = sum over s in bag k of a[s] * W_t[I[s]];
// mean pooling (mode 1, no weights) divides each bag's sum by its number of
// look-ups (an empty bag stays +0.0).  The backward is the transpose: row r
// of table t receives sum over its look-ups s of c_s * dY[bag(s)], with
// c_s = a[s] (sum) or 1 / |bag(s)| (mean), applied once with SGD.
constexpr int kPoolSum = 0;
constexpr int kPoolMean = 1;

int oracle_forward_weighted(int32_t T, int32_t B, int32_t E, const int64_t* rows,
                            const float* const* W, const int32_t* I, const int32_t* O, int64_t NS,
                            const float* a, int32_t mode, float* Y) {
  if (W == nullptr || (mode != kPoolSum && mode != kPoolMean) || (mode == kPoolMean && a))
    return kErrInvalidArg;
  int rc = check_out(T, B, E, rows, I, O, NS, Y);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  std::vector<double> acc(E);
  for (int64_t k = 0; k < int64_t(T) * B; ++k) {
    const int t = int(k / B);
    std::fill(acc.begin(), acc.end(), 0.0);
    for (int64_t s = O[k]; s < O[k + 1]; ++s) {
      const double c = a ? double(a[s]) : 1.0;
      for (int e = 0; e < E; ++e) acc[e] += c * double(W[t][int64_t(I[s]) * E + e]);
    }
    const int64_t n = O[k + 1] - O[k];
    for (int e = 0; e < E; ++e)
      Y[k * E + e] = float(mode == kPoolMean && n > 0 ? acc[e] / double(n) : acc[e]);
  }
  return kOk;
}

int oracle_backward_sgd_weighted(const float* dY, int32_t T, int32_t B, int32_t E,
                                 const int64_t* rows, float* const* W, const int32_t* I,
                                 const int32_t* O, int64_t NS, const float* a, int32_t mode,
                                 float lr) {
  if (W == nullptr || (mode != kPoolSum && mode != kPoolMean) || (mode == kPoolMean && a))
    return kErrInvalidArg;
  int rc = check_grad(T, B, E, rows, I, O, NS, dY);
  if (rc) return rc;
  rc = validate(T, B, E, rows, I, O, NS);
  if (rc) return rc;
  Dedup d;
  dedup_impl(T, B, rows, I, O, NS, d);
  std::vector<double> acc(E);
  for (size_t u = 0; u < d.unique_key.size(); ++u) {
    std::fill(acc.begin(), acc.end(), 0.0);
    for (int64_t i = d.seg_off[u]; i < d.seg_off[u + 1]; ++i) {
      const int64_t s = d.perm[i];
      const int64_t k = d.sorted_bag[i];
      double c = 1.0;
      if (a) c = double(a[s]);
      if (mode == kPoolMean) c = 1.0 / double(O[k + 1] - O[k]);
      const float* g = dY + k * E;
      for (int e = 0; e < E; ++e) acc[e] += c * double(g[e]);
    }
    const int t = table_of_key(d, d.unique_key[u]);
    float* w = W[t] + (int64_t(d.unique_key[u]) - d.rowbase[t]) * E;
    for (int e = 0; e < E; ++e) w[e] = float(double(w[e]) - double(lr) * acc[e]);
  }
  return kOk;
}

}  // extern "C"
