// The paper's multi-core CPU designs, timed beside the GPU library for
// context on the same machine (they are neither the library nor the oracle,
// and share no code with either):
//   * the forward of Algorithm 1, the bags of all tables split over threads;
//   * the backward of Algorithms 2-3 fused (dW[s] is dY of the look-up's bag,
//     so it is never materialised) with the race-free update of Algorithm 4:
//     every thread owns one contiguous range of each table's rows, walks all
//     of the table's look-ups in order and applies those that name its rows.
// Arithmetic is FP32 in the paper's loop order (a bag's rows added in
// look-up order; a row's updates applied one look-up at a time, in order),
// so the results do not depend on the thread count.  The inputs are assumed
// valid (indices inside their table, offsets non-decreasing from 0 to the
// look-up count): only the argument shapes are checked.
#include <omp.h>
#include <stdint.h>

namespace {

bool shapes_ok(int32_t T, int32_t B, int32_t E, const void* W, const int32_t* I,
               const int32_t* O) {
  return T > 0 && B >= 0 && E > 0 && W != nullptr && O != nullptr &&
         (I != nullptr || int64_t(T) * B == 0);
}

}  // namespace

extern "C" {

int cpu_designs_threads() { return omp_get_max_threads(); }

// Y[t*B + b] = sum of W_t[I[s]] over the look-ups s of bag b of table t.
// Returns 0, or -1 for bad arguments.
int cpu_designs_forward(int32_t T, int32_t B, int32_t E, const float* const* W,
                        const int32_t* I, const int32_t* O, float* Y, int32_t threads) {
  if (!shapes_ok(T, B, E, W, I, O) || Y == nullptr || threads < 1) return -1;
  const int64_t bags = int64_t(T) * B;
#pragma omp parallel for schedule(static) num_threads(threads)
  for (int64_t k = 0; k < bags; ++k) {
    const float* table = W[k / B];
    float* y = Y + k * E;
    for (int32_t e = 0; e < E; ++e) y[e] = 0.0f;
    for (int32_t s = O[k]; s < O[k + 1]; ++s) {
      const float* row = table + int64_t(I[s]) * E;
      for (int32_t e = 0; e < E; ++e) y[e] += row[e];
    }
  }
  return 0;
}

// W_t[I[s]] += (-lr) * dY[t*B + b] for every look-up s of bag b of table t,
// thread p of P owning rows [M_t p / P, M_t (p + 1) / P) of table t.
// Returns 0, or -1 for bad arguments.
int cpu_designs_backward_sgd(int32_t T, int32_t B, int32_t E, const int64_t* rows,
                             float* const* W, const int32_t* I, const int32_t* O,
                             const float* dY, float lr, int32_t threads) {
  if (!shapes_ok(T, B, E, W, I, O) || rows == nullptr || dY == nullptr || threads < 1)
    return -1;
  const float step = -lr;
#pragma omp parallel num_threads(threads)
  {
    const int64_t P = omp_get_num_threads(), p = omp_get_thread_num();
    for (int32_t t = 0; t < T; ++t) {
      const int64_t first = rows[t] * p / P, last = rows[t] * (p + 1) / P;
      float* table = W[t];
      for (int64_t k = int64_t(t) * B; k < int64_t(t + 1) * B; ++k) {
        const float* g = dY + k * E;
        for (int32_t s = O[k]; s < O[k + 1]; ++s) {
          const int64_t r = I[s];
          if (r < first || r >= last) continue;
          float* row = table + r * E;
          for (int32_t e = 0; e < E; ++e) row[e] = row[e] + step * g[e];
        }
      }
    }
  }
  return 0;
}

}  // extern "C"
