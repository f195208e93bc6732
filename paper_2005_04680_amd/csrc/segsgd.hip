// Backward fused with the sparse SGD update (Algorithms 2-3, fused as the end
// of Section III-A describes), for gfx950, without float atomics.
//
// Input: the look-ups sorted by row key (ties in look-up order), as
// (key << 32 | bag) words.  The sorted list is cut into fixed chunks of C
// look-ups, one per row group of LPR lanes.  A row group walks its chunk,
// gathers dY[bag] for each look-up (U row loads in flight per lane) and adds
// it to an FP64 accumulator; when the key changes, the finished segment is
//   * applied, W[row] <- W[row] - lr * G, if it began and ended inside the
//     chunk (the W row was requested with the look-up that began it), or
//   * with 64-lane rows, applied as well if it began in the chunk and ends
//     within the next chunk's first 64 look-ups: the wavefront walks on to
//     its end, and the next chunk starts its walk after it, so short segments
//     need no carry;
//   * otherwise parked as a partial sum in the carry buffer: slot 2c for the
//     chunk's first segment, slot 2c+1 for its last one.
// A second kernel gives every other segment that crosses a chunk boundary to
// the chunk where it begins; that chunk adds its own partial and the partials
// of the following chunks, in chunk order, and applies the row once.  Every
// touched row is therefore read and written exactly once, with a sum order
// that does not depend on scheduling (the result is bit-reproducible).
//
// Locality: each XCD owns one contiguous range of chunks, so the dY rows it
// gathers at any time belong to one or two tables, unless eight tables' dY
// would fill more than half of the MALL: then the chunks are walked in
// dispatch order, and all XCDs gather from the dY of the table in progress,
// which the MALL holds.  The W rows, touched once, are read and written with
// non-temporal hints so they do not evict dY.
//
// Sorted positions are unsigned 32-bit: num_indices may be 2^31 - 1, and the
// walks look at most 64 look-ups and two groups past a chunk's end, which
// stays below 2^32.
#include <type_traits>

#include "common.hpp"

namespace embbag {
namespace {

// Row update for FP32 tables: w <- fl(w - lr * G), G in FP64.
struct Fp32Rows {
  struct Pre {
    f4 w;
  };
  template <class D>
  static __device__ __forceinline__ Pre load(const D& d, int t, uint32_t r, uint32_t E, int c4) {
    return {__builtin_nontemporal_load(table_elem<const f4, float>(d.w[t], size_t(r) * E + c4 * 4))};
  }
  template <class D>
  static __device__ __forceinline__ void store(const D& d, int t, uint32_t r, uint32_t E, int c4,
                                               const Pre& p, const d4& g, double lr) {
    f4 o;
    o.x = float(double(p.w.x) - lr * g.x);
    o.y = float(double(p.w.y) - lr * g.y);
    o.z = float(double(p.w.z) - lr * g.z);
    o.w = float(double(p.w.w) - lr * g.w);
    __builtin_nontemporal_store(o, table_elem<f4, float>(d.w[t], size_t(r) * E + c4 * 4));
  }
};

// Row update for split tables (Section VII): recombine hi/lo into the FP32
// weight, apply the FP32 update, split the result again.
struct SplitRows {
  struct Pre {
    u2 hi, lo;
  };
  template <class D>
  static __device__ __forceinline__ Pre load(const D& d, int t, uint32_t r, uint32_t E, int c4) {
    const size_t off = size_t(r) * E + c4 * 4;
    return {__builtin_nontemporal_load(table_elem<const u2, uint16_t>(d.w[t], off)),
            __builtin_nontemporal_load(table_elem<const u2, uint16_t>(d.lo[t], off))};
  }
  static __device__ __forceinline__ float upd(uint32_t hi16, uint32_t lo16, double g, double lr) {
    const float w = __uint_as_float((hi16 << 16) | lo16);
    return float(double(w) - lr * g);
  }
  template <class D>
  static __device__ __forceinline__ void store(const D& d, int t, uint32_t r, uint32_t E, int c4,
                                               const Pre& p, const d4& g, double lr) {
    const uint32_t w0 = __float_as_uint(upd(p.hi.x & 0xFFFFu, p.lo.x & 0xFFFFu, g.x, lr));
    const uint32_t w1 = __float_as_uint(upd(p.hi.x >> 16, p.lo.x >> 16, g.y, lr));
    const uint32_t w2 = __float_as_uint(upd(p.hi.y & 0xFFFFu, p.lo.y & 0xFFFFu, g.z, lr));
    const uint32_t w3 = __float_as_uint(upd(p.hi.y >> 16, p.lo.y >> 16, g.w, lr));
    u2 hi, lo;
    hi.x = (w0 >> 16) | (w1 & 0xFFFF0000u);
    hi.y = (w2 >> 16) | (w3 & 0xFFFF0000u);
    lo.x = (w0 & 0xFFFFu) | (w1 << 16);
    lo.y = (w2 & 0xFFFFu) | (w3 << 16);
    const size_t off = size_t(r) * E + c4 * 4;
    __builtin_nontemporal_store(hi, table_elem<u2, uint16_t>(d.w[t], off));
    __builtin_nontemporal_store(lo, table_elem<u2, uint16_t>(d.lo[t], off));
  }
};

// Four gradient values of dY row `bag` as loaded (FP32, or BF16 bit patterns);
// BF16 values are widened exactly only when summed, so that the loads of a
// group stay in flight together.
template <bool GBF16>
struct Dy {
  using Raw = typename std::conditional<GBF16, u2, f4>::type;
  static __device__ __forceinline__ Raw load(const void* dY, uint32_t bag, uint32_t E, int c4) {
    if constexpr (!GBF16)
      return *reinterpret_cast<const f4*>(static_cast<const float*>(dY) + size_t(bag) * E + c4 * 4);
    else
      return *reinterpret_cast<const u2*>(static_cast<const uint16_t*>(dY) + size_t(bag) * E +
                                          c4 * 4);
  }
  static __device__ __forceinline__ Raw zero() {
    if constexpr (!GBF16)
      return f4{0.f, 0.f, 0.f, 0.f};
    else
      return u2{0u, 0u};
  }
  static __device__ __forceinline__ f4 value(const Raw& r) {
    if constexpr (!GBF16)
      return r;
    else
      return f4{__uint_as_float(r.x << 16), __uint_as_float(r.x & 0xFFFF0000u),
                __uint_as_float(r.y << 16), __uint_as_float(r.y & 0xFFFF0000u)};
  }
};

__device__ __forceinline__ d4 widen(const f4& v) {
  return d4{double(v.x), double(v.y), double(v.z), double(v.w)};
}

template <int CPL>
__device__ __forceinline__ void store_carry(double* carry, int64_t slot, int E, int rl, int lpr,
                                            const d4* acc) {
  double* c = carry + slot * E;
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c4 = rl + j * lpr;
    if (c4 < E / 4) *reinterpret_cast<d4*>(c + c4 * 4) = acc[j];
  }
}

// Look-up coefficients of the gradient sum (Section II's weights a_p): 1 for
// plain sums, the look-up's weight for weighted sums (the weights sorted
// along with the look-ups, so read in sorted order), 1/|bag| for means.
struct PoolDev {
  const float* svals;
  const int32_t* offsets;
};


// Lane i's copy of a 64-bit word held one per lane (i the same across the
// wavefront).
__device__ __forceinline__ uint64_t word_of_lane(uint64_t w, int i) {
  const uint32_t l = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(w)), i));
  const uint32_t h = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(w >> 32)), i));
  return (uint64_t(h) << 32) | l;
}

template <int LPR, int CPL, class Rows, int MODE, bool GBF16>
__global__ __launch_bounds__(kBlock) void segment_sgd(
    TableDesc d, const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks,
    const void* __restrict__ dY, int32_t B, float inv_b, float lr,
    double* __restrict__ carry, const int32_t* __restrict__ flags, uint32_t token, PoolDev pd,
    int32_t in_order) {
  __shared__ TableLds tl;
  if constexpr (LPR < kWave) {
    stage_tables(d, tl);
    __syncthreads();
  }
  const auto& tb = table_view<(LPR < kWave)>(d, tl);
  // A data error, or no sort result for these sizes: no table writes.
  if (flags[0] != 0 || uint32_t(flags[1]) != token) return;
  constexpr int R = kWave / LPR;
  // look-ups in flight per row group: fewer when a wave holds several row
  // groups (their (key, bag) words no longer share scalar registers)
  constexpr int U = CPL == 1 ? (LPR == kWave ? 8 : 4) : (CPL == 2 ? 4 : 2);
  const int E = d.dim;
  const int E4 = E / 4;  // float4 groups per row
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int blk = int(logical_block(in_order != 0));
  const int chunk = (blk * kWavesPerBlock + wave_id()) * R + rg;
  if (chunk >= nchunks) return;
  const uint32_t lo = uint32_t(chunk) * uint32_t(C);
  const uint32_t hi0 = min(lo + uint32_t(C), uint32_t(NS));
  const double lrd = double(lr);
  constexpr bool kW = MODE == kPoolWeighted;
  // With 64 lanes per row (one row group per wavefront), a segment that
  // crosses into the next chunk and ends within its first 64 look-ups is
  // walked to its end here; with several row groups per wavefront the longer
  // walk would hold up the others, and every crossing segment is carried.
  constexpr bool kWin = LPR == kWave;

  const uint32_t kprev = lo > 0 ? key_of(sorted[lo - 1]) : kNoKey;
  const uint32_t knext0 = hi0 < uint32_t(NS) ? key_of(sorted[hi0]) : kNoKey;
  uint32_t hi = hi0, knext = knext0;  // end of the walk, key just past it
  uint32_t s0 = lo;                   // start of the walk
  bool first_open;                    // first segment walked began before s0
  bool is_first = true;
  // Software pipeline: the (key, bag) words of the next U look-ups are loaded
  // while the current ones are summed; for the current U look-ups, the dY rows
  // (skipped when a look-up repeats the previous (key, bag) pair: its row is
  // still in registers) and the W rows of the segments that start among them
  // are all requested before the first of them is used.
  // Weighted bags: each look-up's weight is loaded one group ahead, with its
  // word (the weights were sorted along with the look-ups).
  uint64_t pn[U];
  float an[U];
  if constexpr (kWin) {
    // Requested with the keys above: the key before the previous chunk, the
    // words of the chunk's first 64 look-ups and the keys of the 64 past its
    // end, one per lane.
    const uint32_t klast = key_of(sorted[hi0 - 1]);
    const uint32_t kpp = lo > uint32_t(C) ? key_of(sorted[lo - uint32_t(C) - 1]) : kNoKey;
    const uint64_t wlead = lo + lane < hi0 ? sorted[lo + lane] : ~0ull;
    const float alead = kW && lo + lane < hi0 ? pd.svals[lo + lane] : 0.f;
    const uint32_t kpast = hi0 + lane < uint32_t(NS) ? key_of(sorted[hi0 + lane]) : kNoKey;
    // The last segment began in this chunk, continues in the next and ends
    // within its first 64 look-ups: the walk goes on to its end, and the
    // segment is applied here.
    if (knext0 == klast && kprev != klast) {
      const uint64_t m = __builtin_amdgcn_ballot_w64(kpast != klast);
      if (m != 0ull) {
        const int e = int(__builtin_ctzll(m));
        hi = hi0 + uint32_t(e);
        knext = uint32_t(__builtin_amdgcn_readlane(int(kpast), e));
      }
    }
    // The first segment began in the previous chunk and ends within this
    // chunk's first 64 look-ups: the previous chunk applied it, and the walk
    // starts after it.
    first_open = kprev == key_of(word_of_lane(wlead, 0));
    if (first_open && kpp != kprev) {
      const uint64_t m = __builtin_amdgcn_ballot_w64(key_of(wlead) != kprev);
      if (m != 0ull) {
        s0 = lo + uint32_t(__builtin_ctzll(m));
        if (s0 >= hi0) return;  // the whole chunk was that segment
        first_open = false;
        is_first = false;  // a segment left open at the end takes slot 2c+1
      }
    }
    // the first U words from the lanes that hold them
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t q = s0 + uint32_t(u);
      const int i = int(q - lo);
      if (i < kWave) {
        pn[u] = q < hi ? word_of_lane(wlead, i) : 0ull;
        if constexpr (kW)
          an[u] = q < hi ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alead), i)) : 0.f;
      } else {
        pn[u] = q < hi ? sorted[q] : 0ull;
        if constexpr (kW) an[u] = q < hi ? pd.svals[q] : 0.f;
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) pn[u] = lo + u < hi0 ? sorted[lo + u] : 0ull;
    if constexpr (kW) {
#pragma unroll
      for (int u = 0; u < U; ++u) an[u] = lo + u < hi0 ? pd.svals[lo + u] : 0.f;
    }
    first_open = kprev == key_of(pn[0]);
  }
  const uint64_t p0 = pn[0];
  uint32_t cur = key_of(p0);
  int ct = table_of_bag(bag_of(p0), B, inv_b);

  d4 acc[CPL];
  f4 glast[CPL];
  typename Rows::Pre pre[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    acc[j] = d4{0.0, 0.0, 0.0, 0.0};
    glast[j] = f4{0.f, 0.f, 0.f, 0.f};
    const int c4 = rl + j * LPR;
    if (!first_open && c4 < E4) pre[j] = Rows::load(tb, ct, cur - tb.rowbase[ct], E, c4);
  }

  auto apply = [&](uint32_t key, int t) {
    const uint32_t r = key - tb.rowbase[t];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) Rows::store(tb, t, r, E, c4, pre[j], acc[j], lrd);
    }
  };

  uint64_t plast = p0;  // look-up before the current group (none before s0: p0 itself)
  for (uint32_t s = s0; s < hi; s += U) {
    uint64_t p[U];
    uint32_t bg[U];
    float aw[U];
    int32_t ob0[U], ob1[U];
    bool dup[U], nseg[U];
    typename Dy<GBF16>::Raw g[U][CPL];
    typename Rows::Pre wp[U][CPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      p[u] = pn[u];
      if constexpr (kW) aw[u] = an[u];
      bg[u] = s + u < hi ? bag_of(p[u]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t pq = u == 0 ? plast : p[u - 1];
      const bool valid = s + u < hi;
      // a repeat of the previous look-up's (key, bag): its dY row is reused
      dup[u] = valid && p[u] == pq && !(s == s0 && u == 0);
      nseg[u] = valid && key_of(p[u]) != key_of(pq);
    }
    if constexpr (MODE == kPoolMean) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        ob0[u] = s + u < hi ? pd.offsets[bg[u]] : 0;
        ob1[u] = s + u < hi ? pd.offsets[bg[u] + 1] : 1;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ld = s + u < hi && !dup[u];
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = rl + j * LPR;
        g[u][j] = (ld && c4 < E4) ? Dy<GBF16>::load(dY, bg[u], E, c4) : Dy<GBF16>::zero();
      }
      if (nseg[u]) {
        const int tu = table_of_bag(bg[u], B, inv_b);
        const uint32_t ru = key_of(p[u]) - tb.rowbase[tu];
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          const int c4 = rl + j * LPR;
          if (c4 < E4) wp[u][j] = Rows::load(tb, tu, ru, E, c4);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) pn[u] = s + U + u < hi ? sorted[s + U + u] : 0ull;
    if constexpr (kW) {
#pragma unroll
      for (int u = 0; u < U; ++u) an[u] = s + U + u < hi ? pd.svals[s + U + u] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s + u >= hi) break;
      if (nseg[u]) {
        if (is_first && first_open)
          store_carry<CPL>(carry, 2 * int64_t(chunk), E, rl, LPR, acc);
        else
          apply(cur, ct);
        cur = key_of(p[u]);
        ct = table_of_bag(bg[u], B, inv_b);
        is_first = false;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          acc[j] = d4{0.0, 0.0, 0.0, 0.0};
          pre[j] = wp[u][j];
        }
      }
      double c = 1.0;
      if constexpr (kW) c = double(aw[u]);
      if constexpr (MODE == kPoolMean) c = 1.0 / double(ob1[u] - ob0[u]);
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        if (!dup[u]) glast[j] = Dy<GBF16>::value(g[u][j]);
        if constexpr (MODE == kPoolPlain)
          acc[j] += widen(glast[j]);
        else
          acc[j] += c * widen(glast[j]);
      }
    }
    plast = p[U - 1];
  }

  const bool last_open = knext == cur;  // last segment continues in the next chunk
  if (is_first && (first_open || last_open)) {
    store_carry<CPL>(carry, 2 * int64_t(chunk), E, rl, LPR, acc);
  } else if (!is_first && last_open) {
    store_carry<CPL>(carry, 2 * int64_t(chunk) + 1, E, rl, LPR, acc);
  } else {
    apply(cur, ct);
  }
}

// Groups of kCarryGroup chunks that one segment fills entirely (the look-up
// before the group and the one after it have the same key, so, the look-ups
// being sorted, every look-up in between has it too): their partials (slot 2c
// of each chunk) are summed in chunk order once, so that a long segment's
// fixup adds one value per such group instead of one per chunk.  gflag[g]
// says whether group g is filled (written for every group).
template <int LPR, int CPL>
__global__ __launch_bounds__(kBlock) void carry_group(
    const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks, int32_t E,
    int32_t ngroups, const double* __restrict__ carry, double* __restrict__ gsum,
    int32_t* __restrict__ gflag, const int32_t* __restrict__ flags, uint32_t token) {
  if (flags[0] != 0 || uint32_t(flags[1]) != token) return;
  constexpr int R = kWave / LPR;
  const int E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int g = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * R + rg;
  if (g >= ngroups) return;
  const int64_t c0 = int64_t(g) * kCarryGroup;
  const int64_t first = c0 * C, after = (c0 + kCarryGroup) * C;
  const bool full = c0 > 0 && c0 + kCarryGroup <= nchunks && after < NS &&
                    key_of(sorted[first - 1]) == key_of(sorted[after]);
  if (rl == 0) gflag[g] = full ? 1 : 0;
  if (!full) return;
  // The partials are requested GU at a time (all 16 for one float4 group per
  // lane, 2 for three or four) and added in chunk order.
  constexpr int GU = CPL == 1 ? kCarryGroup : (CPL == 2 ? kCarryGroup / 2 : kCarryGroup / 8);
  d4 acc[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) acc[j] = d4{0.0, 0.0, 0.0, 0.0};
#pragma unroll 1
  for (int u0 = 0; u0 < kCarryGroup; u0 += GU) {
    d4 v[GU][CPL];
#pragma unroll
    for (int u = 0; u < GU; ++u) {
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = rl + j * LPR;
        v[u][j] = c4 < E4 ? *reinterpret_cast<const d4*>(carry + 2 * (c0 + u0 + u) * E + c4 * 4)
                          : d4{0.0, 0.0, 0.0, 0.0};
      }
    }
#pragma unroll
    for (int u = 0; u < GU; ++u) {
#pragma unroll
      for (int j = 0; j < CPL; ++j) acc[j] += v[u][j];
    }
  }
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c4 = rl + j * LPR;
    if (c4 < E4) *reinterpret_cast<d4*>(gsum + int64_t(g) * E + c4 * 4) = acc[j];
  }
}

// Segments carried across chunk boundaries: the chunk where one begins sums
// the partials in chunk order (a filled group's pre-summed value in place of
// its chunks) and applies the row.  With 64 lanes per row a wavefront takes a
// group of kCarryGroup chunks, finds which of them start such a segment (all
// boundary words requested at once, one chunk per lane) and fixes those up
// one after another: with short segments applied by the update, most groups
// hold none and few hold more than two.  Narrower rows take one chunk per
// row group.
template <int LPR, int CPL, class Rows, int MODE>
__global__ __launch_bounds__(kBlock) void segment_fixup(
    TableDesc d, const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks,
    int32_t B, float inv_b, float lr, const double* __restrict__ carry,
    const double* __restrict__ gsum, const int32_t* __restrict__ gflag,
    const int32_t* __restrict__ flags, uint32_t token, PoolDev pd) {
  __shared__ TableLds tl;
  if constexpr (LPR < kWave) {
    stage_tables(d, tl);
    __syncthreads();
  }
  const auto& tb = table_view<(LPR < kWave)>(d, tl);
  if (flags[0] != 0 || uint32_t(flags[1]) != token) return;
  constexpr int R = kWave / LPR;
  constexpr int UF = CPL == 1 ? 8 : (CPL == 2 ? 4 : 2);
  const int E = d.dim, E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int ngroups = (nchunks + kCarryGroup - 1) / kCarryGroup;
  // Bit q of `need`: chunk base + q starts a segment left to this kernel.
  int base;
  uint32_t need;
  if constexpr (LPR == kWave) {
    // A wavefront takes a group of kCarryGroup chunks; chunk q needs a fix-up
    // if its last segment continues in the next chunk, began in this one, and
    // goes on past the next chunk's first 64 look-ups (one ending earlier was
    // applied whole by the update).  Lane q examines chunk q.
    base = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * kCarryGroup;
    if (base >= nchunks) return;
    const int c = base + lane;
    const uint32_t lo = uint32_t(c) * uint32_t(C);
    const uint32_t hi = lo + uint32_t(C);
    const bool ok = lane < kCarryGroup && c < nchunks && hi < uint32_t(NS);
    const uint64_t wl = ok ? sorted[hi - 1] : 0ull;
    const uint64_t wn = ok ? sorted[hi] : ~0ull;
    const uint64_t wb = ok && lo > 0 ? sorted[lo - 1] : ~0ull;
    const uint64_t wx =
        ok && hi + uint32_t(kWave - 1) < uint32_t(NS) ? sorted[hi + uint32_t(kWave - 1)] : ~0ull;
    const uint32_t kl = key_of(wl);
    need = uint32_t(__builtin_amdgcn_ballot_w64(key_of(wn) == kl && key_of(wb) != kl &&
                                                key_of(wx) == kl));
  } else {
    // A row group takes one chunk; it needs a fix-up if its last segment
    // continues in the next chunk and began in this one.
    base = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * R + rg;
    if (base >= nchunks) return;
    const uint32_t lo = uint32_t(base) * uint32_t(C);
    const uint32_t hi = min(lo + uint32_t(C), uint32_t(NS));
    if (hi >= uint32_t(NS)) return;
    // the words around both ends of the chunk, requested together
    const uint64_t wl = sorted[hi - 1], wn = sorted[hi];
    const uint64_t wb = lo > 0 ? sorted[lo - 1] : ~0ull;
    const uint32_t kl = key_of(wl);
    need = key_of(wn) == kl && key_of(wb) != kl ? 1u : 0u;
  }
  constexpr bool kLaneFlags = LPR >= 16;
  constexpr int NF = kLaneFlags ? LPR : UF;  // flags read per step
  while (need != 0) {
    const int chunk = base + __builtin_ctz(need);
    need &= need - 1u;
    const uint32_t lo = uint32_t(chunk) * uint32_t(C);
    const uint32_t hi = lo + uint32_t(C);
    const uint32_t kl = key_of(sorted[hi - 1]);
    const uint32_t kf = key_of(sorted[lo]);
    const int ct = table_of_bag(bag_of(sorted[hi - 1]), B, inv_b);
    const uint32_t r = kl - tb.rowbase[ct];
    const int64_t own = kf != kl ? 2 * int64_t(chunk) + 1 : 2 * int64_t(chunk);

    d4 acc[CPL];
    typename Rows::Pre pre[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) {
        acc[j] = *reinterpret_cast<const d4*>(carry + own * E + c4 * 4);
        pre[j] = Rows::load(tb, ct, r, E, c4);
      } else {
        acc[j] = d4{0.0, 0.0, 0.0, 0.0};
      }
    }
    // Chunks chunk+1, chunk+2, ... belong to the segment while the chunk
    // before continues it.  At a group boundary the filled groups that follow
    // are taken whole (the segment then continues past each): the flags of
    // the next groups (one per lane of the row group when it has at least 16
    // lanes, else UF), then the sums of the leading filled ones, UF at a time,
    // are requested and added in order.  Otherwise up to UF chunks, not
    // crossing the next group boundary (their first-segment partials and the
    // key just past them), are loaded per step.
    int unfilled = -1;  // a group known not to be filled
    bool inside = true;
    int c2 = chunk + 1;
    while (inside) {
      const int gi = c2 / kCarryGroup, off = c2 % kCarryGroup;
      if (off == 0 && c2 < nchunks && gi != unfilled) {
        int nf = 0;  // filled groups in a row from gi (at most NF)
        if constexpr (kLaneFlags) {
          const int f = gi + rl < ngroups ? gflag[gi + rl] : 0;
          const uint64_t m = __builtin_amdgcn_ballot_w64(f != 0);
          uint64_t mine;
          if constexpr (LPR == kWave)
            mine = m;
          else
            mine = (m >> (rg * LPR)) & ((1ull << LPR) - 1ull);
          nf = ~mine == 0ull ? kWave : int(__builtin_ctzll(~mine));
        } else {
#pragma unroll
          for (int u = 0; u < UF; ++u) {
            const int f = gi + u < ngroups ? gflag[gi + u] : 0;
            nf += (nf == u && f != 0) ? 1 : 0;
          }
        }
        if (nf < NF) unfilled = gi + nf;
        if (nf > 0) {
          for (int u0 = 0; u0 < nf; u0 += UF) {
            d4 gs[UF][CPL];
#pragma unroll
            for (int u = 0; u < UF; ++u) {
#pragma unroll
              for (int j = 0; j < CPL; ++j) {
                const int c4 = rl + j * LPR;
                gs[u][j] = (u0 + u < nf && c4 < E4)
                               ? *reinterpret_cast<const d4*>(gsum + int64_t(gi + u0 + u) * E + c4 * 4)
                               : d4{0.0, 0.0, 0.0, 0.0};
              }
            }
#pragma unroll
            for (int u = 0; u < UF; ++u) {
              if (u0 + u >= nf) break;
#pragma unroll
              for (int j = 0; j < CPL; ++j) acc[j] += gs[u][j];
            }
          }
          c2 += nf * kCarryGroup;
          continue;
        }
      }
      const int n = kCarryGroup - off < UF ? kCarryGroup - off : UF;
      d4 part[UF][CPL];
      uint32_t kn[UF];
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        const int cu = c2 + u;
        const bool ok = u < n && cu < nchunks;
        const int64_t nxt = int64_t(cu + 1) * C;
        kn[u] = (ok && nxt < NS) ? key_of(sorted[nxt]) : kNoKey;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          const int c4 = rl + j * LPR;
          part[u][j] = (ok && c4 < E4) ? *reinterpret_cast<const d4*>(carry + 2 * int64_t(cu) * E + c4 * 4)
                                       : d4{0.0, 0.0, 0.0, 0.0};
        }
      }
#pragma unroll
      for (int u = 0; u < UF; ++u) {
        if (!inside || u >= n) break;
#pragma unroll
        for (int j = 0; j < CPL; ++j) acc[j] += part[u][j];
        inside = kn[u] == kl;
      }
      c2 += n;
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) Rows::store(tb, ct, r, E, c4, pre[j], acc[j], double(lr));
    }
  }
}

template <class Rows, int MODE, bool GBF16>
bool launch_seg(RowGeom g, int blocks, hipStream_t st, const TableDesc& d, const uint64_t* sorted,
                int32_t NS, int32_t C, int32_t nchunks, const void* dY, int32_t B, float inv_b,
                float lr, double* carry, const int32_t* flags, uint32_t token, PoolDev pd,
                int32_t in_order) {
#define EMB_SEG(L, CC)                                                                     \
  hipLaunchKernelGGL((segment_sgd<L, CC, Rows, MODE, GBF16>), dim3(blocks), dim3(kBlock), 0, st, \
                     d, sorted, NS, C, nchunks, dY, B, inv_b, lr, carry, flags, token, pd,      \
                     in_order)
  switch (g.lpr) {
    case 1: EMB_SEG(1, 1); return true;
    case 2: EMB_SEG(2, 1); return true;
    case 4: EMB_SEG(4, 1); return true;
    case 8: EMB_SEG(8, 1); return true;
    case 16: EMB_SEG(16, 1); return true;
    case 32: EMB_SEG(32, 1); return true;
    case 64:
      switch (g.cpl) {
        case 1: EMB_SEG(64, 1); return true;
        case 2: EMB_SEG(64, 2); return true;
        case 3: EMB_SEG(64, 3); return true;
        case 4: EMB_SEG(64, 4); return true;
      }
  }
#undef EMB_SEG
  return false;
}

bool launch_group(RowGeom g, hipStream_t st, const uint64_t* sorted, int32_t NS, int32_t C,
                  int32_t nchunks, int32_t E, int32_t ngroups, const double* carry, double* gsum,
                  int32_t* gflag, const int32_t* flags, uint32_t token) {
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  const int blocks = (ngroups + per_block - 1) / per_block;
  if (blocks == 0) return true;
#define EMB_GRP(L, CC)                                                                        \
  hipLaunchKernelGGL((carry_group<L, CC>), dim3(blocks), dim3(kBlock), 0, st, sorted, NS, C, \
                     nchunks, E, ngroups, carry, gsum, gflag, flags, token)
  switch (g.lpr) {
    case 1: EMB_GRP(1, 1); return true;
    case 2: EMB_GRP(2, 1); return true;
    case 4: EMB_GRP(4, 1); return true;
    case 8: EMB_GRP(8, 1); return true;
    case 16: EMB_GRP(16, 1); return true;
    case 32: EMB_GRP(32, 1); return true;
    case 64:
      switch (g.cpl) {
        case 1: EMB_GRP(64, 1); return true;
        case 2: EMB_GRP(64, 2); return true;
        case 3: EMB_GRP(64, 3); return true;
        case 4: EMB_GRP(64, 4); return true;
      }
  }
#undef EMB_GRP
  return false;
}

template <class Rows, int MODE>
bool launch_fix(RowGeom g, int blocks, hipStream_t st, const TableDesc& d, const uint64_t* sorted,
                int32_t NS, int32_t C, int32_t nchunks, int32_t B, float inv_b, float lr,
                const double* carry, const double* gsum, const int32_t* gflag,
                const int32_t* flags, uint32_t token, PoolDev pd) {
#define EMB_FIX(L, CC)                                                                       \
  hipLaunchKernelGGL((segment_fixup<L, CC, Rows, MODE>), dim3(blocks), dim3(kBlock), 0, st, d, \
                     sorted, NS, C, nchunks, B, inv_b, lr, carry, gsum, gflag, flags, token, pd)
  switch (g.lpr) {
    case 1: EMB_FIX(1, 1); return true;
    case 2: EMB_FIX(2, 1); return true;
    case 4: EMB_FIX(4, 1); return true;
    case 8: EMB_FIX(8, 1); return true;
    case 16: EMB_FIX(16, 1); return true;
    case 32: EMB_FIX(32, 1); return true;
    case 64:
      switch (g.cpl) {
        case 1: EMB_FIX(64, 1); return true;
        case 2: EMB_FIX(64, 2); return true;
        case 3: EMB_FIX(64, 3); return true;
        case 4: EMB_FIX(64, 4); return true;
      }
  }
#undef EMB_FIX
  return false;
}

template <class Rows, int MODE, bool GBF16 = false>
bool launch_apply(const TableDesc& d, int32_t B, const void* dY, float lr, const BwdLayout& L,
                  char* ws, uint32_t token, PoolDev pd, hipStream_t st) {
  const uint64_t* sorted = sorted_buffer(L, ws);
  double* carry = reinterpret_cast<double*>(ws + L.off_carry);
  double* gsum = reinterpret_cast<double*>(ws + L.off_gsum);
  int32_t* gflag = reinterpret_cast<int32_t*>(ws + L.off_gflag);
  const int32_t* flags = reinterpret_cast<const int32_t*>(ws + L.off_flags);
  const float inv_b = 1.0f / float(B);
  const RowGeom g = row_geom(d.dim);
  // a segment's end is looked for within 64 look-ups of a chunk boundary,
  // which must stay inside the neighbouring chunk
  if (g.lpr == kWave && L.chunk < 2 * int64_t(kWave)) return false;
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  const int blocks = int((L.nchunks + per_block - 1) / per_block);
  const int32_t NS = int32_t(L.ns), C = int32_t(L.chunk), nch = int32_t(L.nchunks);
  const int32_t in_order = apply_in_dispatch_order(blocks, d.num_tables, B, d.dim, GBF16 ? 2 : 4);
  const int fix_blocks =
      g.lpr == kWave ? int((L.ngroups + kWavesPerBlock - 1) / kWavesPerBlock) : blocks;
  return launch_seg<Rows, MODE, GBF16>(g, blocks, st, d, sorted, NS, C, nch, dY, B, inv_b, lr,
                                       carry, flags, token, pd, in_order) &&
         launch_group(g, st, sorted, NS, C, nch, d.dim, int32_t(L.ngroups), carry, gsum, gflag,
                      flags, token) &&
         launch_fix<Rows, MODE>(g, fix_blocks, st, d, sorted, NS, C, nch, B, inv_b, lr, carry,
                                gsum, gflag, flags, token, pd);
}

}  // namespace

hipError_t launch_segment_sgd(const TableDesc& d, bool split, int32_t B, const void* dY,
                              bool dy_bf16, float lr, const BwdLayout& L, char* ws,
                              uint32_t token, const PoolArgs& pool, hipStream_t st) {
  if (L.ns == 0) return hipSuccess;
  PoolDev pd{sorted_values(L, ws), pool.offsets};
  bool ok;
  if (split && dy_bf16)
    ok = launch_apply<SplitRows, kPoolPlain, true>(d, B, dY, lr, L, ws, token, pd, st);
  else if (split)
    ok = launch_apply<SplitRows, kPoolPlain>(d, B, dY, lr, L, ws, token, pd, st);
  else if (pool.mode == kPoolWeighted)
    ok = launch_apply<Fp32Rows, kPoolWeighted>(d, B, dY, lr, L, ws, token, pd, st);
  else if (pool.mode == kPoolMean)
    ok = launch_apply<Fp32Rows, kPoolMean>(d, B, dY, lr, L, ws, token, pd, st);
  else
    ok = launch_apply<Fp32Rows, kPoolPlain>(d, B, dY, lr, L, ws, token, pd, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace embbag
