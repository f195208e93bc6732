// Forward of the EmbeddingBag step (Algorithm 1, sum pooling) for gfx950.
//
// Each "row group" of LPR lanes owns G consecutive bags of one table and walks
// their look-ups (contiguous in `indices`) as one list: U row loads are in
// flight per lane before any of them is summed, and a bag's FP32 sum is
// stored when the walk crosses the bag's end offset (empty bags store +0.0).
// Every lane holds CPL groups of 4 columns, so a row is read with 128-bit
// loads (64-bit for the BF16 halves of a split table).  Grids that fit the
// chip at once give each XCD one contiguous range of bags (one or two tables,
// whose hot rows then stay in that XCD's L2).  Larger grids whose tables'
// touched rows would not fit the MALL eight tables at a time walk the bags
// in dispatch order: all XCDs share the table in progress, and a row read
// again is served by the MALL instead of HBM.
//
// Once a group's offsets are validated its look-up positions are unsigned
// 32-bit: num_indices may be 2^31 - 1, and the walk reads index windows and
// load slots past a group's last look-up, which stays below 2^32.
#include "common.hpp"

namespace embbag {
namespace {

template <bool SPLIT>
__device__ __forceinline__ f4 load_row4(const void* base, uint32_t row, uint32_t E, int col4) {
  if constexpr (!SPLIT) {
    const float* p = static_cast<const float*>(base) + size_t(row) * E + col4 * 4;
    return *reinterpret_cast<const f4*>(p);
  } else {
    // BF16 high halves: element e is the 16 MSBs of an FP32 value.
    const uint16_t* p = static_cast<const uint16_t*>(base) + size_t(row) * E + col4 * 4;
    const u2 v = *reinterpret_cast<const u2*>(p);
    f4 r;
    r.x = __uint_as_float(v.x << 16);
    r.y = __uint_as_float(v.x & 0xFFFF0000u);
    r.z = __uint_as_float(v.y << 16);
    r.w = __uint_as_float(v.y & 0xFFFF0000u);
    return r;
  }
}

__device__ __forceinline__ d4 to_d4(const f4& v) {
  return d4{double(v.x), double(v.y), double(v.z), double(v.w)};
}

// FP32 -> BF16, round to nearest, ties to even (NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t b = __float_as_uint(f);
  if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x40u;
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Row groups that walk several bags are held to 6 waves per SIMD (80 VGPRs)
// for one float4 group per lane and plain sums, 5 for weighted or mean
// pooling (their coefficients take registers); wider rows take what they need.
template <int LPR, int CPL, bool SPLIT, bool MULTI, int MODE, bool YBF16>
__global__ __launch_bounds__(kBlock, MULTI ? (CPL == 1 && MODE == kPoolPlain ? 6 : (CPL == 1 ? 5 : 1)) : 1) void fwd_gather_sum(
    TableDesc d, const int32_t* __restrict__ I, const int32_t* __restrict__ O, int32_t NS,
    int32_t B, int32_t G, int32_t groups_per_table, int32_t items, void* __restrict__ Y,
    int32_t* __restrict__ status, const float* __restrict__ A, int32_t in_order) {
  constexpr int R = kWave / LPR;
  // Row loads in flight per lane: 10 when a wavefront reads one 1 KB row per
  // load and walks one bag (58 VGPRs, still 8 waves per SIMD); fewer as the
  // rows per lane grow.
  constexpr int U = CPL == 1 ? (LPR == kWave && !MULTI ? 10 : 8) : (CPL == 2 ? 4 : 2);
  const int E = d.dim;
  const int E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int blk = int(logical_block(in_order != 0));
  const int item = (blk * kWavesPerBlock + wave_id()) * R + rg;
  if (item >= items) return;

  const int TB = d.num_tables * B;
  const int t = item / groups_per_table;
  const int k0 = t * B + (item - t * groups_per_table) * G;
  const int k1 = MULTI ? min(k0 + G, (t + 1) * B) : k0 + 1;
  const uint32_t M = d.rows[t];
  const void* base = d.w[t];
  int err = 0;

  // Stores bag k's pooled row, the FP64 sum rounded once to FP32; mean
  // pooling divides by the bag's n look-ups first.  BF16 outputs are the FP32
  // values rounded to nearest even.
  auto store_bag = [&](int k, const d4* acc, int n) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      d4 a = acc[j];
      if constexpr (MODE == kPoolMean) {
        if (n > 0) a = a / double(n);
      }
      const f4 v = f4{float(a.x), float(a.y), float(a.z), float(a.w)};
      if (c4 >= E4) continue;
      if constexpr (YBF16) {
        u2 h;
        h.x = bf16_rne(v.x) | (bf16_rne(v.y) << 16);
        h.y = bf16_rne(v.z) | (bf16_rne(v.w) << 16);
        *reinterpret_cast<u2*>(static_cast<uint16_t*>(Y) + size_t(k) * E + c4 * 4) = h;
      } else {
        *reinterpret_cast<f4*>(static_cast<float*>(Y) + size_t(k) * E + c4 * 4) = v;
      }
    }
  };

  const int s0 = O[k0], s1 = O[k1];
  if ((k0 == 0 && s0 != 0) || (k1 == TB && s1 != NS)) err = EMBBAG_ERR_OFFSETS;
  bool bad = s0 < 0 || s1 > NS || s0 > s1;
  int k = k0;
  int bound = s1;
  int bstart = s0;  // first look-up of bag k
  // Several bags per row group: when their offsets O[k0..k1] fit one per
  // lane, they are loaded together here and each bag end is then read from
  // its lane instead of with a load of its own.
  const bool olanes = MULTI && G < LPR;
  int ov = 0;
  if constexpr (MULTI) {
    if (olanes && !bad && rl <= k1 - k0) ov = O[k0 + rl];
    bound = bad ? 0 : O[k0 + 1];
    bad = bad || bound < s0 || bound > s1;
  }

  d4 acc[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) acc[j] = d4{0.0, 0.0, 0.0, 0.0};

  // Indices arrive in windows of LPR look-ups, one per lane of the row group
  // (a coalesced load), the next window already in flight; each look-up's
  // index is then broadcast from its lane, so the row loads of an iteration
  // do not wait on index loads.  Past the end of the group a slot re-reads
  // the group's last row, and an index outside its table reads row 0: every
  // load is valid, and such slots are masked out of the sum.
  constexpr bool kWin = LPR >= U;
  // valid offsets: 0 <= s0 <= s1 <= NS
  const uint32_t u0 = uint32_t(s0), u1 = uint32_t(s1);
  uint32_t wbase = u0;
  int vcur = 0, vnext = 0;
  float acur = 0.f, anext = 0.f;  // per-look-up weights, same windows
  if constexpr (kWin) {
    if (!bad) {
      vcur = u0 + rl < u1 ? I[u0 + rl] : 0;
      vnext = u0 + LPR + rl < u1 ? I[u0 + LPR + rl] : 0;
      if constexpr (MODE == kPoolWeighted) {
        acur = u0 + rl < u1 ? A[u0 + rl] : 0.f;
        anext = u0 + LPR + rl < u1 ? A[u0 + LPR + rl] : 0.f;
      }
    }
  }

  for (uint32_t s = u0; s < u1 && !bad; s += U) {
    if constexpr (kWin) {
      if (s - wbase >= LPR) {
        wbase += LPR;
        vcur = vnext;
        vnext = wbase + LPR + rl < u1 ? I[wbase + LPR + rl] : 0;
        if constexpr (MODE == kPoolWeighted) {
          acur = anext;
          anext = wbase + LPR + rl < u1 ? A[wbase + LPR + rl] : 0.f;
        }
      }
    }
    f4 v[U][CPL];
    bool use[U];
    float wt[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t ss = min(s + u, u1 - 1);
      int idx;
      if constexpr (kWin) {
        if constexpr (LPR == kWave) {
          // U need not divide LPR: the last slots of an iteration may lie in
          // the next window, which is already loaded (off < LPR + U <= 2 LPR).
          const int off = int(ss - wbase);
          idx = off < LPR ? __builtin_amdgcn_readlane(vcur, off)
                          : __builtin_amdgcn_readlane(vnext, off - LPR);
          if constexpr (MODE == kPoolWeighted)
            wt[u] = __int_as_float(off < LPR
                                       ? __builtin_amdgcn_readlane(__float_as_int(acur), off)
                                       : __builtin_amdgcn_readlane(__float_as_int(anext), off - LPR));
        } else {
          static_assert(LPR % U == 0, "a window must hold whole iterations");
          idx = __shfl(vcur, rg * LPR + int(ss - wbase), kWave);
          if constexpr (MODE == kPoolWeighted) wt[u] = __shfl(acur, rg * LPR + int(ss - wbase), kWave);
        }
      } else {
        idx = I[ss];
        if constexpr (MODE == kPoolWeighted) wt[u] = A[ss];
      }
      const bool ok = uint32_t(idx) < M;
      if (!ok) err = min(err, EMBBAG_ERR_INDEX_RANGE);
      use[u] = ok && s + u < u1;
      const uint32_t row = ok ? uint32_t(idx) : 0u;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = min(rl + j * LPR, E4 - 1);
        v[u][j] = load_row4<SPLIT>(base, row, E, c4);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (MULTI) {
        const uint32_t ss = s + u;
        if (ss >= u1 || bad) break;
        // Crossing the end of bag k (and of any empty bags after it).  While
        // ss < s1 = O[k1] and O is non-decreasing up to s1, k + 1 < k1 here.
        while (ss >= uint32_t(bound)) {
          store_bag(k, acc, bound - bstart);
          bstart = bound;
#pragma unroll
          for (int j = 0; j < CPL; ++j) acc[j] = d4{0.0, 0.0, 0.0, 0.0};
          ++k;
          const int nb = olanes ? __shfl(ov, rg * LPR + (k + 1 - k0), kWave) : O[k + 1];
          if (nb < bound || nb > s1) {
            bad = true;
            break;
          }
          bound = nb;
        }
        if (bad) break;
      }
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        if constexpr (MODE == kPoolWeighted)
          acc[j] = use[u] ? acc[j] + double(wt[u]) * to_d4(v[u][j]) : acc[j];
        else
          acc[j] = use[u] ? acc[j] + to_d4(v[u][j]) : acc[j];
      }
    }
  }
  if (!bad) {
    store_bag(k, acc, s1 - bstart);
    if constexpr (MULTI) {
      // Remaining bags of the group hold no look-ups: O[k'] == s1 for them all.
      for (int kk = k + 1; kk < k1; ++kk) {
        if (O[kk] != s1) bad = true;
#pragma unroll
        for (int j = 0; j < CPL; ++j) acc[j] = d4{0.0, 0.0, 0.0, 0.0};
        store_bag(kk, acc, 0);
      }
    }
  }
  if (bad) err = EMBBAG_ERR_OFFSETS;
  if (err != 0 && rl == 0 && status != nullptr) atomicMin(status, err);
}

// T*B == 0: the only data check left is offsets[0] == 0 == num_indices.
__global__ void fwd_empty_check(const int32_t* __restrict__ O, int32_t NS,
                                int32_t* __restrict__ status) {
  if (threadIdx.x == 0 && status != nullptr && (O[0] != 0 || NS != 0))
    atomicMin(status, EMBBAG_ERR_OFFSETS);
}

template <bool SPLIT, int MODE, bool YBF16, int LPR, int CPL>
void launch_one(dim3 grid, hipStream_t st, const TableDesc& d, const int32_t* I, const int32_t* O,
                int32_t NS, int32_t B, int32_t G, int32_t gpt, int32_t items, void* Y,
                int32_t* status, const float* A, int32_t in_order) {
  if (G > 1)
    hipLaunchKernelGGL((fwd_gather_sum<LPR, CPL, SPLIT, true, MODE, YBF16>), grid, dim3(kBlock), 0,
                       st, d, I, O, NS, B, G, gpt, items, Y, status, A, in_order);
  else
    hipLaunchKernelGGL((fwd_gather_sum<LPR, CPL, SPLIT, false, MODE, YBF16>), grid, dim3(kBlock),
                       0, st, d, I, O, NS, B, G, gpt, items, Y, status, A, in_order);
}

template <bool SPLIT, int MODE, bool YBF16 = false>
bool dispatch(RowGeom g, dim3 grid, hipStream_t st, const TableDesc& d, const int32_t* I,
              const int32_t* O, int32_t NS, int32_t B, int32_t G, int32_t gpt, int32_t items,
              void* Y, int32_t* status, const float* A, int32_t in_order) {
#define EMB_FWD(L, C)                                                                   \
  launch_one<SPLIT, MODE, YBF16, L, C>(grid, st, d, I, O, NS, B, G, gpt, items, Y, status, A, \
                                       in_order)
  switch (g.lpr) {
    case 1: EMB_FWD(1, 1); return true;
    case 2: EMB_FWD(2, 1); return true;
    case 4: EMB_FWD(4, 1); return true;
    case 8: EMB_FWD(8, 1); return true;
    case 16: EMB_FWD(16, 1); return true;
    case 32: EMB_FWD(32, 1); return true;
    case 64:
      switch (g.cpl) {
        case 1: EMB_FWD(64, 1); return true;
        case 2: EMB_FWD(64, 2); return true;
        case 3: EMB_FWD(64, 3); return true;
        case 4: EMB_FWD(64, 4); return true;
      }
  }
#undef EMB_FWD
  return false;
}

}  // namespace

hipError_t launch_forward(const TableDesc& d, bool split, int32_t B, const int32_t* I,
                          const int32_t* O, int64_t NS, void* Y, bool y_bf16, int32_t* status,
                          const PoolArgs& pool, hipStream_t st) {
  const int64_t TB = int64_t(d.num_tables) * B;
  if (TB == 0) {
    hipLaunchKernelGGL(fwd_empty_check, dim3(1), dim3(kWave), 0, st, O, int32_t(NS), status);
    return hipGetLastError();
  }
  // Bags per row group: enough look-ups per group to keep ~16 row loads per
  // lane in flight when bags are short (P = 1 for the MLPerf-style tables).
  const int64_t avg = NS / TB;
  int G = avg >= 16 ? 1 : int(16 / (avg > 0 ? avg : 1));
  G = G > 64 ? 64 : G;
  G = G > B ? B : G;
  const int gpt = (B + G - 1) / G;
  const int64_t items = int64_t(d.num_tables) * gpt;
  const RowGeom g = row_geom(d.dim);
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  const dim3 grid(unsigned((items + per_block - 1) / per_block));
  const int32_t ns = int32_t(NS), it = int32_t(items);
  // A table's touched rows are at most its look-ups' rows.
  const int64_t row_bytes = int64_t(d.dim) * (split ? 2 : 4);
  const int32_t in_order = dispatch_order(grid.x, d.num_tables, NS / d.num_tables * row_bytes);
  bool ok = false;
  if (split && y_bf16)
    ok = dispatch<true, kPoolPlain, true>(g, grid, st, d, I, O, ns, B, G, gpt, it, Y, status,
                                          nullptr, in_order);
  else if (split)
    ok = dispatch<true, kPoolPlain>(g, grid, st, d, I, O, ns, B, G, gpt, it, Y, status, nullptr,
                                    in_order);
  else if (pool.mode == kPoolWeighted)
    ok = dispatch<false, kPoolWeighted>(g, grid, st, d, I, O, ns, B, G, gpt, it, Y, status,
                                        pool.weights, in_order);
  else if (pool.mode == kPoolMean)
    ok = dispatch<false, kPoolMean>(g, grid, st, d, I, O, ns, B, G, gpt, it, Y, status, nullptr,
                                    in_order);
  else
    ok = dispatch<false, kPoolPlain>(g, grid, st, d, I, O, ns, B, G, gpt, it, Y, status, nullptr,
                                     in_order);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace embbag
