// Drives every entry point of the CPU oracle (oracle/oracle.cpp) over seeded
// random small cases, the edge cases of the method (empty bags, B = 0, one
// row per table, duplicate look-ups) and invalid inputs (indices out of
// range, bad offsets, bad sizes), so that a build with AddressSanitizer and
// UndefinedBehaviorSanitizer sees every path.  Exits 0 unless a sanitizer
// stops it or a call returns a status its inputs do not explain.
//
// Built and run by tests/test_oracle_sanitizers.py (g++ only, no GPU code).
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

extern "C" {
int oracle_validate(int32_t, int32_t, int32_t, const int64_t*, const int32_t*, const int32_t*,
                    int64_t);
int oracle_forward(int32_t, int32_t, int32_t, const int64_t*, const float* const*,
                   const int32_t*, const int32_t*, int64_t, float*);
int oracle_forward_literal(int32_t, int32_t, int32_t, const int64_t*, const float* const*,
                           const int32_t*, const int32_t*, int64_t, float*);
int oracle_forward_split(int32_t, int32_t, int32_t, const int64_t*, const uint16_t* const*,
                         const int32_t*, const int32_t*, int64_t, float*);
int oracle_forward_weighted(int32_t, int32_t, int32_t, const int64_t*, const float* const*,
                            const int32_t*, const int32_t*, int64_t, const float*, int32_t,
                            float*);
int oracle_forward_split_bf16_act(int32_t, int32_t, int32_t, const int64_t*,
                                  const uint16_t* const*, const int32_t*, const int32_t*,
                                  int64_t, uint16_t*);
int oracle_dedup(int32_t, int32_t, const int64_t*, const int32_t*, const int32_t*, int64_t,
                 uint32_t*, uint32_t*, uint32_t*, int32_t*, int64_t*);
int oracle_backward_sgd(const float*, int32_t, int32_t, int32_t, const int64_t*, float* const*,
                        const int32_t*, const int32_t*, int64_t, float);
int oracle_backward_sgd_literal(const float*, int32_t, int32_t, int32_t, const int64_t*,
                                float* const*, const int32_t*, const int32_t*, int64_t, float);
int oracle_backward_sgd_split(const float*, int32_t, int32_t, int32_t, const int64_t*,
                              uint16_t* const*, uint16_t* const*, const int32_t*,
                              const int32_t*, int64_t, float);
int oracle_backward_sgd_weighted(const float*, int32_t, int32_t, int32_t, const int64_t*,
                                 float* const*, const int32_t*, const int32_t*, int64_t,
                                 const float*, int32_t, float);
int oracle_backward_sgd_split_bf16_act(const uint16_t*, int32_t, int32_t, int32_t,
                                       const int64_t*, uint16_t* const*, uint16_t* const*,
                                       const int32_t*, const int32_t*, int64_t, float);
void oracle_split(const float*, uint16_t*, uint16_t*, int64_t);
void oracle_combine(const uint16_t*, const uint16_t*, float*, int64_t);
void oracle_bf16_round(const float*, uint16_t*, int64_t);
void oracle_bf16_widen(const uint16_t*, float*, int64_t);
int64_t oracle_split_roundtrip_mismatches(uint64_t, uint64_t);
}

namespace {

constexpr int kOk = 0, kErrInvalidArg = -1, kErrIndexRange = -3, kErrOffsets = -4;

struct Rng {  // SplitMix64 (Steele, Lea and Flood 2014)
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int below(int n) { return int(next() % uint64_t(n)); }
  float uniform() { return float(double(next() >> 11) * 0x1.0p-53 * 2.0 - 1.0); }
};

int failures = 0;

void expect(bool ok, const char* what, int trial) {
  if (!ok) {
    std::fprintf(stderr, "trial %d: %s\n", trial, what);
    ++failures;
  }
}

// One case: tables, bags, gradients; bad = 0 (valid), 1 (index out of range),
// 2 (offsets decreasing).
void run_case(Rng& g, int trial, int bad) {
  const int T = 1 + g.below(4);
  const int E = 4 * (1 + g.below(4));
  const int B = g.below(7);
  std::vector<int64_t> rows(T);
  for (auto& r : rows) r = 1 + g.below(40);
  std::vector<std::vector<float>> W(T);
  std::vector<std::vector<uint16_t>> hi(T), lo(T);
  for (int t = 0; t < T; ++t) {
    W[t].resize(size_t(rows[t]) * E);
    for (auto& w : W[t]) w = 0.1f * g.uniform();
    hi[t].resize(W[t].size());
    lo[t].resize(W[t].size());
    oracle_split(W[t].data(), hi[t].data(), lo[t].data(), int64_t(W[t].size()));
  }
  std::vector<int32_t> O(size_t(T) * B + 1, 0), I;
  for (int k = 0; k < T * B; ++k) {
    const int t = k / B;
    const int n = g.below(6);  // 0..5 look-ups, empty bags included
    for (int j = 0; j < n; ++j) {
      const bool dup = !I.empty() && j > 0 && g.below(3) == 0;
      I.push_back(dup ? I.back() : g.below(int(rows[t])));
    }
    O[k + 1] = int32_t(I.size());
  }
  const int64_t NS = int64_t(I.size());
  int expect_rc = kOk;
  if (bad == 1 && NS > 0) {
    I[size_t(g.below(int(NS)))] = int32_t(rows[0]) + 1000;
    expect_rc = kErrIndexRange;
  }
  if (bad == 2 && T * B >= 2 && O[T * B] > 0) {
    O[1] = O[T * B] + 1;  // O[1] > O[2] and beyond NS
    expect_rc = kErrOffsets;
  }
  std::vector<float> dY(size_t(T) * B * E), a(static_cast<size_t>(NS));
  for (auto& v : dY) v = g.uniform();
  for (auto& v : a) v = 0.5f + 0.5f * (g.uniform() + 1.0f);
  std::vector<uint16_t> dYb(dY.size()), Yb(dY.size());
  oracle_bf16_round(dY.data(), dYb.data(), int64_t(dY.size()));

  std::vector<const float*> wp(T);
  std::vector<float*> wm(T);
  std::vector<const uint16_t*> hp(T);
  std::vector<uint16_t*> hm(T), lm(T);
  for (int t = 0; t < T; ++t) {
    wp[t] = W[t].data();
    wm[t] = W[t].data();
    hp[t] = hi[t].data();
    hm[t] = hi[t].data();
    lm[t] = lo[t].data();
  }
  const int32_t* Ip = I.empty() ? nullptr : I.data();
  std::vector<float> Y(dY.size());
  const int v = oracle_validate(T, B, E, rows.data(), Ip, O.data(), NS);
  expect(v == expect_rc, "validate status", trial);
  const int rc[] = {
      oracle_forward(T, B, E, rows.data(), wp.data(), Ip, O.data(), NS, Y.data()),
      oracle_forward_literal(T, B, E, rows.data(), wp.data(), Ip, O.data(), NS, Y.data()),
      oracle_forward_split(T, B, E, rows.data(), hp.data(), Ip, O.data(), NS, Y.data()),
      oracle_forward_weighted(T, B, E, rows.data(), wp.data(), Ip, O.data(), NS, a.data(), 0,
                              Y.data()),
      oracle_forward_weighted(T, B, E, rows.data(), wp.data(), Ip, O.data(), NS, nullptr, 1,
                              Y.data()),
      oracle_forward_split_bf16_act(T, B, E, rows.data(), hp.data(), Ip, O.data(), NS,
                                    Yb.data()),
      oracle_backward_sgd(dY.data(), T, B, E, rows.data(), wm.data(), Ip, O.data(), NS, 0.1f),
      oracle_backward_sgd_literal(dY.data(), T, B, E, rows.data(), wm.data(), Ip, O.data(), NS,
                                  0.1f),
      oracle_backward_sgd_split(dY.data(), T, B, E, rows.data(), hm.data(), lm.data(), Ip,
                                O.data(), NS, 0.1f),
      oracle_backward_sgd_weighted(dY.data(), T, B, E, rows.data(), wm.data(), Ip, O.data(), NS,
                                   a.data(), 0, 0.1f),
      oracle_backward_sgd_weighted(dY.data(), T, B, E, rows.data(), wm.data(), Ip, O.data(), NS,
                                   nullptr, 1, 0.1f),
      oracle_backward_sgd_split_bf16_act(dYb.data(), T, B, E, rows.data(), hm.data(), lm.data(),
                                         Ip, O.data(), NS, 0.1f),
  };
  for (int r : rc) expect(r == expect_rc, "entry point status", trial);
  std::vector<uint32_t> sk(static_cast<size_t>(NS)), sb(static_cast<size_t>(NS)), uk(static_cast<size_t>(NS));
  std::vector<int32_t> so(static_cast<size_t>(NS) + 1);
  int64_t U = -1;
  const int d = oracle_dedup(T, B, rows.data(), Ip, O.data(), NS, sk.data(), sb.data(),
                             uk.data(), so.data(), &U);
  expect(d == expect_rc, "dedup status", trial);
  if (d == kOk) expect(U >= 0 && U <= NS && so[size_t(U)] == NS, "dedup segments", trial);
}

void invalid_arguments(int trial) {
  const int64_t rows[2] = {10, 10};
  const int32_t I[2] = {1, 2};
  const int32_t O[3] = {0, 1, 2};
  expect(oracle_validate(0, 1, 4, rows, I, O, 2) == kErrInvalidArg, "T = 0", trial);
  expect(oracle_validate(65, 1, 4, rows, I, O, 2) == kErrInvalidArg, "T = 65", trial);
  expect(oracle_validate(2, 1, 6, rows, I, O, 2) == kErrInvalidArg, "E % 4", trial);
  expect(oracle_validate(2, 1, 2048, rows, I, O, 2) == kErrInvalidArg, "E > 1024", trial);
  expect(oracle_validate(2, -1, 4, rows, I, O, 2) == kErrInvalidArg, "B < 0", trial);
  expect(oracle_validate(2, 1, 4, nullptr, I, O, 2) == kErrInvalidArg, "rows null", trial);
  expect(oracle_validate(2, 1, 4, rows, I, O, int64_t(1) << 31) == kErrInvalidArg, "NS", trial);
  float y[8];
  expect(oracle_forward(2, 1, 4, rows, nullptr, I, O, 2, y) == kErrInvalidArg, "W null", trial);
  expect(oracle_forward_weighted(2, 1, 4, rows, nullptr, I, O, 2, nullptr, 7, y) ==
             kErrInvalidArg, "pooling mode", trial);
  // A null output is an argument error only when there is something to write,
  // and argument errors come before data errors (as in the library).
  std::vector<float> w0(40, 0.5f), w1(40, 0.25f);
  const float* wc[2] = {w0.data(), w1.data()};
  float* wm[2] = {w0.data(), w1.data()};
  const int32_t Obad[3] = {0, 2, 1};
  const int32_t O0[1] = {0};
  expect(oracle_forward(2, 1, 4, rows, wc, I, O, 2, nullptr) == kErrInvalidArg, "Y null", trial);
  expect(oracle_forward(2, 1, 4, rows, wc, I, Obad, 2, nullptr) == kErrInvalidArg,
         "Y null before bad offsets", trial);
  expect(oracle_forward(2, 0, 4, rows, wc, nullptr, O0, 0, nullptr) == kOk, "B = 0, Y null", trial);
  expect(oracle_backward_sgd(nullptr, 2, 1, 4, rows, wm, I, Obad, 2, 0.1f) == kErrInvalidArg,
         "dY null before bad offsets", trial);
  expect(oracle_backward_sgd_literal(nullptr, 2, 1, 4, rows, wm, I, O, 2, 0.1f) == kErrInvalidArg,
         "dY null (literal)", trial);
  expect(oracle_backward_sgd(nullptr, 2, 0, 4, rows, wm, nullptr, O0, 0, 0.1f) == kOk,
         "no look-ups, dY null", trial);
}

}  // namespace

int main() {
  Rng g{20050468};
  for (int trial = 0; trial < 600; ++trial) run_case(g, trial, trial % 3);
  invalid_arguments(-1);
  // Split, combine, BF16 rounding and widening over special values and random patterns.
  std::vector<float> x = {0.0f, -0.0f, INFINITY, -INFINITY, NAN, 1e-45f, -1e-45f, 3.4e38f};
  for (int i = 0; i < 4096; ++i) {
    const uint32_t u = uint32_t(g.next());
    float f;
    std::memcpy(&f, &u, 4);
    x.push_back(f);
  }
  const int64_t n = int64_t(x.size());
  std::vector<uint16_t> h(x.size()), l(x.size()), r(x.size());
  std::vector<float> back(x.size()), wide(x.size());
  oracle_split(x.data(), h.data(), l.data(), n);
  oracle_combine(h.data(), l.data(), back.data(), n);
  expect(std::memcmp(back.data(), x.data(), x.size() * 4) == 0, "split round trip", -2);
  oracle_bf16_round(x.data(), r.data(), n);
  oracle_bf16_widen(r.data(), wide.data(), n);
  expect(oracle_split_roundtrip_mismatches(0xFFFF0000ull, 0x20000ull) == 0, "round trip range",
         -3);
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("oracle driver: all cases ran clean\n");
  return 0;
}
