// The paper's unfused update designs, on gfx950, as measured baselines for
// the fused sort-and-segment backward (which is the product path):
//   * Algorithm 2: the per-look-up gradient dW[s] = dY[bag(s)], materialised
//     as an NS x E array;
//   * Algorithm 3: W[I[s]] += alpha * dW[s] for every look-up, with hardware
//     FP32 atomics (alpha = -lr);
//   * Algorithms 2+3 fused the naive way: every look-up atomically adds
//     -lr * dY[bag] to its row (no dW);
//   * Algorithm 4: race-free update by row ownership: owner j (one wavefront)
//     owns the keys [K*j/n, K*(j+1)/n) of the global row space, scans all
//     look-ups in order and applies those it owns, one at a time.
// Atomics make the FP32 sum order scheduling-dependent; the owner update
// applies each row's look-ups in increasing s, like a sequential loop.
// A last kernel is no design of the paper but the floor of every update: the
// read and write-back of each touched row, once, with nothing summed.
#include <type_traits>

#include "common.hpp"

namespace embbag {
namespace {

__device__ __forceinline__ bool bag_range(const int32_t* O, int k, int NS, int* s0, int* s1) {
  *s0 = O[k];
  *s1 = O[k + 1];
  return *s0 >= 0 && *s1 <= NS && *s0 <= *s1;
}

// Algorithm 2: dW[s][:] = dY[k][:] for the look-ups s of bag k.
template <int LPR, int CPL>
__global__ __launch_bounds__(kBlock) void materialize_kernel(const float* __restrict__ dY,
                                                             const int32_t* __restrict__ O,
                                                             int32_t NS, int32_t TB, int32_t E,
                                                             float* __restrict__ dW,
                                                             int32_t* __restrict__ status) {
  constexpr int R = kWave / LPR;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int k = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * R + rg;
  if (k >= TB) return;
  int s0, s1;
  if (!bag_range(O, k, NS, &s0, &s1)) {
    if (rl == 0 && status) atomicMin(status, EMBBAG_ERR_OFFSETS);
    return;
  }
  const int E4 = E / 4;
  f4 g[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c4 = rl + j * LPR;
    if (c4 < E4) g[j] = *reinterpret_cast<const f4*>(dY + size_t(k) * E + c4 * 4);
  }
  for (int s = s0; s < s1; ++s) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) *reinterpret_cast<f4*>(dW + size_t(s) * E + c4 * 4) = g[j];
    }
  }
}

// Algorithm 3 (FUSED = false: reads dW[s]) or Algorithms 2+3 fused (reads
// dY[k] once per bag): atomic FP32 adds of -lr * gradient into each row.
template <int LPR, int CPL, bool FUSED>
__global__ __launch_bounds__(kBlock) void atomic_update_kernel(
    TableDesc d, const float* __restrict__ src, const int32_t* __restrict__ I,
    const int32_t* __restrict__ O, int32_t NS, int32_t B, float lr, int32_t* __restrict__ status) {
  constexpr int R = kWave / LPR;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int TB = d.num_tables * B;
  const int k = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * R + rg;
  if (k >= TB) return;
  int s0, s1;
  if (!bag_range(O, k, NS, &s0, &s1)) {
    if (rl == 0 && status) atomicMin(status, EMBBAG_ERR_OFFSETS);
    return;
  }
  const int t = k / B;
  const int E = d.dim, E4 = E / 4;
  float* w = static_cast<float*>(d.w[t]);
  f4 g[CPL];
  if constexpr (FUSED) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) g[j] = *reinterpret_cast<const f4*>(src + size_t(k) * E + c4 * 4);
    }
  }
  for (int s = s0; s < s1; ++s) {
    const int idx = I[s];
    if (uint32_t(idx) >= d.rows[t]) {
      if (rl == 0 && status) atomicMin(status, EMBBAG_ERR_INDEX_RANGE);
      continue;
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 >= E4) continue;
      f4 v = FUSED ? g[j] : *reinterpret_cast<const f4*>(src + size_t(s) * E + c4 * 4);
      float* p = w + size_t(idx) * E + c4 * 4;
      unsafeAtomicAdd(p + 0, -lr * v.x);
      unsafeAtomicAdd(p + 1, -lr * v.y);
      unsafeAtomicAdd(p + 2, -lr * v.z);
      unsafeAtomicAdd(p + 3, -lr * v.w);
    }
  }
}

// Algorithm 4: wavefront j owns global keys [K*j/n, K*(j+1)/n); it scans the
// look-ups 64 at a time (table from the per-table look-up ranges), and for
// each owned look-up, in increasing s, does W[row] += alpha * dW[s] in FP32.
template <int CPL>
__global__ __launch_bounds__(kWave) void owner_update_kernel(TableDesc d,
                                                             const float* __restrict__ dW,
                                                             const int32_t* __restrict__ I,
                                                             const int32_t* __restrict__ O,
                                                             int32_t NS, int32_t B,
                                                             int32_t owners, float lr) {
  const int lane = lane_id();
  const int j = blockIdx.x;
  const int T = d.num_tables;
  const int E = d.dim, E4 = E / 4;
  const uint64_t K = d.rowbase[T];
  const uint32_t klo = uint32_t(K * uint64_t(j) / uint64_t(owners));
  const uint32_t khi = uint32_t(K * uint64_t(j + 1) / uint64_t(owners));
  const float alpha = -lr;
  int t = 0;
  // unsigned: with num_indices = 2^31 - 1 the last window runs past it
  for (uint32_t base = 0; base < uint32_t(NS); base += kWave) {
    const uint32_t s = base + lane;
    // table of look-up s: tables own contiguous look-up ranges
    int tl = t;
    while (tl + 1 < T && int64_t(s) >= O[(tl + 1) * B]) ++tl;
    const int idx = s < uint32_t(NS) ? I[s] : -1;
    const bool ok = s < uint32_t(NS) && uint32_t(idx) < d.rows[tl];
    const uint32_t key = ok ? d.rowbase[tl] + uint32_t(idx) : 0u;
    uint64_t mine = __builtin_amdgcn_ballot_w64(ok && key >= klo && key < khi);
    while (mine) {
      const int l = __builtin_ctzll(mine);
      mine &= mine - 1;
      const uint32_t so = base + l;
      const int to = __builtin_amdgcn_readlane(tl, l);
      const uint32_t ro = uint32_t(__builtin_amdgcn_readlane(idx, l));
      float* w = static_cast<float*>(d.w[to]) + size_t(ro) * E;
#pragma unroll
      for (int jj = 0; jj < CPL; ++jj) {
        const int c4 = lane + jj * kWave;
        if (c4 >= E4) continue;
        const f4 g = *reinterpret_cast<const f4*>(dW + size_t(so) * E + c4 * 4);
        f4 v = *reinterpret_cast<f4*>(w + c4 * 4);
        v.x = v.x + alpha * g.x;
        v.y = v.y + alpha * g.y;
        v.z = v.z + alpha * g.z;
        v.w = v.w + alpha * g.w;
        *reinterpret_cast<f4*>(w + c4 * 4) = v;
      }
    }
    t = __builtin_amdgcn_readlane(tl, kWave - 1);
  }
}


// The update's data movement alone: the look-ups sorted by a prepared
// workspace are cut into the same chunks as the fused update's; a row group
// walks its chunk H look-ups at a time, and for each segment that begins
// there reads the row and writes it back unchanged (an SGD step with a zero
// gradient), all H reads in flight before the writes.  The chunks are walked
// in the fused update's order for FP32 gradients.  Split rows (Section VII)
// are read and written as their two halves, 16 bits per element each, as the
// split update moves them.
template <bool SPLIT>
struct TouchRow {
  using V = typename std::conditional<SPLIT, u2, f4>::type;
  V a, b;
  template <class D>
  static __device__ __forceinline__ TouchRow load(const D& tb, int t, uint32_t r, uint32_t E,
                                                   int c4) {
    TouchRow x;
    if constexpr (SPLIT) {
      const size_t off = size_t(r) * E + c4 * 4;
      x.a = __builtin_nontemporal_load(table_elem<const u2, uint16_t>(tb.w[t], off));
      x.b = __builtin_nontemporal_load(table_elem<const u2, uint16_t>(tb.lo[t], off));
    } else {
      x.a = __builtin_nontemporal_load(table_elem<const f4, float>(tb.w[t], size_t(r) * E + c4 * 4));
    }
    return x;
  }
  template <class D>
  __device__ __forceinline__ void store(const D& tb, int t, uint32_t r, uint32_t E, int c4) const {
    if constexpr (SPLIT) {
      const size_t off = size_t(r) * E + c4 * 4;
      __builtin_nontemporal_store(a, table_elem<u2, uint16_t>(tb.w[t], off));
      __builtin_nontemporal_store(b, table_elem<u2, uint16_t>(tb.lo[t], off));
    } else {
      __builtin_nontemporal_store(a, table_elem<f4, float>(tb.w[t], size_t(r) * E + c4 * 4));
    }
  }
};

template <int LPR, int CPL, bool SPLIT>
__global__ __launch_bounds__(kBlock) void touch_rows_kernel(
    TableDesc d, const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks,
    int32_t B, float inv_b, const int32_t* __restrict__ flags, uint32_t token, int32_t in_order) {
  __shared__ TableLds tl;
  if constexpr (LPR < kWave) {
    stage_tables(d, tl);
    __syncthreads();
  }
  const auto& tbl = table_view<(LPR < kWave)>(d, tl);
  if (flags[0] != 0 || uint32_t(flags[1]) != token) return;
  constexpr int R = kWave / LPR;
  constexpr int H = 8;
  const int E = d.dim, E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int blk = int(logical_block(in_order != 0));
  const int chunk = (blk * kWavesPerBlock + wave_id()) * R + rg;
  if (chunk >= nchunks) return;
  // unsigned: with num_indices = 2^31 - 1 the last group runs past it
  const uint32_t lo = uint32_t(chunk) * uint32_t(C);
  const uint32_t hi = min(lo + uint32_t(C), uint32_t(NS));
  uint32_t prev = lo > 0 ? key_of(sorted[lo - 1]) : kNoKey;
  for (uint32_t s = lo; s < hi; s += H) {
    bool head[H];
    int tb[H];
    uint32_t row[H];
#pragma unroll
    for (int u = 0; u < H; ++u) {
      const bool valid = s + u < hi;
      const uint64_t p = valid ? sorted[s + u] : 0ull;
      const uint32_t key = key_of(p);
      head[u] = valid && key != prev;
      prev = valid ? key : prev;
      tb[u] = head[u] ? table_of_bag(bag_of(p), B, inv_b) : 0;
      row[u] = head[u] ? key - tbl.rowbase[tb[u]] : 0u;
    }
    TouchRow<SPLIT> v[H][CPL];
#pragma unroll
    for (int u = 0; u < H; ++u) {
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = rl + j * LPR;
        if (head[u] && c4 < E4) v[u][j] = TouchRow<SPLIT>::load(tbl, tb[u], row[u], E, c4);
      }
    }
#pragma unroll
    for (int u = 0; u < H; ++u) {
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = rl + j * LPR;
        if (head[u] && c4 < E4) v[u][j].store(tbl, tb[u], row[u], E, c4);
      }
    }
  }
}

int grid_bags(int64_t TB, RowGeom g) {
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  return int((TB + per_block - 1) / per_block);
}

#define EMB_GEOM_SWITCH(g, MACRO) \
  switch (g.lpr) {                \
    case 1: MACRO(1, 1); break;   \
    case 2: MACRO(2, 1); break;   \
    case 4: MACRO(4, 1); break;   \
    case 8: MACRO(8, 1); break;   \
    case 16: MACRO(16, 1); break; \
    case 32: MACRO(32, 1); break; \
    default:                      \
      switch (g.cpl) {            \
        case 1: MACRO(64, 1); break; \
        case 2: MACRO(64, 2); break; \
        case 3: MACRO(64, 3); break; \
        default: MACRO(64, 4); break; \
      }                           \
  }

}  // namespace

hipError_t launch_materialize(const float* dY, const int32_t* O, int64_t NS, int32_t T, int32_t B,
                              int32_t E, float* dW, int32_t* status, hipStream_t st) {
  const int64_t TB = int64_t(T) * B;
  if (TB == 0) return hipSuccess;
  const RowGeom g = row_geom(E);
  const dim3 grid(grid_bags(TB, g));
#define EMB_MAT(L, C)                                                                        \
  hipLaunchKernelGGL((materialize_kernel<L, C>), grid, dim3(kBlock), 0, st, dY, O, int32_t(NS), \
                     int32_t(TB), E, dW, status)
  EMB_GEOM_SWITCH(g, EMB_MAT)
#undef EMB_MAT
  return hipGetLastError();
}

hipError_t launch_atomic_update(const TableDesc& d, const float* src, bool fused,
                                const int32_t* I, const int32_t* O, int64_t NS, int32_t B,
                                float lr, int32_t* status, hipStream_t st) {
  const int64_t TB = int64_t(d.num_tables) * B;
  if (TB == 0) return hipSuccess;
  const RowGeom g = row_geom(d.dim);
  const dim3 grid(grid_bags(TB, g));
#define EMB_ATOM(L, C)                                                                         \
  if (fused)                                                                                   \
    hipLaunchKernelGGL((atomic_update_kernel<L, C, true>), grid, dim3(kBlock), 0, st, d, src, I, \
                       O, int32_t(NS), B, lr, status);                                         \
  else                                                                                         \
    hipLaunchKernelGGL((atomic_update_kernel<L, C, false>), grid, dim3(kBlock), 0, st, d, src,   \
                       I, O, int32_t(NS), B, lr, status)
  EMB_GEOM_SWITCH(g, EMB_ATOM)
#undef EMB_ATOM
  return hipGetLastError();
}

hipError_t launch_owner_update(const TableDesc& d, const float* dW, const int32_t* I,
                               const int32_t* O, int64_t NS, int32_t B, int32_t owners, float lr,
                               hipStream_t st) {
  if (NS == 0) return hipSuccess;
  const int cpl = (d.dim / 4 + kWave - 1) / kWave;
#define EMB_OWN(C)                                                                              \
  hipLaunchKernelGGL((owner_update_kernel<C>), dim3(owners), dim3(kWave), 0, st, d, dW, I, O, \
                     int32_t(NS), B, owners, lr)
  switch (cpl) {
    case 1: EMB_OWN(1); break;
    case 2: EMB_OWN(2); break;
    case 3: EMB_OWN(3); break;
    default: EMB_OWN(4); break;
  }
#undef EMB_OWN
  return hipGetLastError();
}

hipError_t launch_touch_rows(const TableDesc& d, bool split, int32_t B, const BwdLayout& L,
                             char* ws, uint32_t token, hipStream_t st) {
  if (L.ns == 0) return hipSuccess;
  const uint64_t* sorted = sorted_buffer(L, ws);
  const int32_t* flags = reinterpret_cast<const int32_t*>(ws + L.off_flags);
  const float inv_b = 1.0f / float(B);
  const RowGeom g = row_geom(d.dim);
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  const dim3 grid(unsigned((L.nchunks + per_block - 1) / per_block));
  const int32_t in_order = apply_in_dispatch_order(grid.x, d.num_tables, B, d.dim, 4);
#define EMB_TOUCH(LL, CC)                                                                     \
  if (split)                                                                                  \
    hipLaunchKernelGGL((touch_rows_kernel<LL, CC, true>), grid, dim3(kBlock), 0, st, d, sorted, \
                       int32_t(L.ns), int32_t(L.chunk), int32_t(L.nchunks), B, inv_b, flags,    \
                       token, in_order);                                                      \
  else                                                                                        \
    hipLaunchKernelGGL((touch_rows_kernel<LL, CC, false>), grid, dim3(kBlock), 0, st, d,        \
                       sorted, int32_t(L.ns), int32_t(L.chunk), int32_t(L.nchunks), B, inv_b,   \
                       flags, token, in_order)
  EMB_GEOM_SWITCH(g, EMB_TOUCH)
#undef EMB_TOUCH
  return hipGetLastError();
}

}  // namespace embbag
