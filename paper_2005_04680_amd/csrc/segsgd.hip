// Backward fused with the sparse SGD update (Algorithms 2-3, fused as the end
// of Section III-A describes), for gfx950, without float atomics.
//
// Input: the look-ups sorted by row key (ties in look-up order), as
// (key << 32 | bag) words.  The sorted list is cut into fixed chunks of C
// look-ups, one per row group of LPR lanes.  A row group walks its chunk,
// gathers dY[bag] for each look-up (U row loads in flight per lane) and adds
// it to an FP64 accumulator; when the key changes, the finished segment is
//   * applied, W[row] <- W[row] - lr * G, if it began and ended inside the
//     chunk (the W row was prefetched when the segment began), or
//   * parked as a partial sum in the carry buffer: slot 2c for the chunk's
//     first segment, slot 2c+1 for its last one.
// A second kernel gives every segment that crosses chunk boundaries to the
// chunk where it begins; that chunk adds its own partial and the partials
// of the following chunks, in chunk order, and applies the row once.  Every
// touched row is therefore read and written exactly once, with a sum order
// that does not depend on scheduling (the result is bit-reproducible).
#include "common.hpp"

namespace embbag {
namespace {

// Row update for FP32 tables: w <- fl(w - lr * G), G in FP64.
struct Fp32Rows {
  struct Pre {
    f4 w;
  };
  static __device__ __forceinline__ Pre load(const TableDesc& d, int t, uint32_t r, int E, int c4) {
    return {*reinterpret_cast<const f4*>(static_cast<const float*>(d.w[t]) + size_t(r) * E + c4 * 4)};
  }
  static __device__ __forceinline__ void store(const TableDesc& d, int t, uint32_t r, int E, int c4,
                                               const Pre& p, const d4& g, double lr) {
    f4 o;
    o.x = float(double(p.w.x) - lr * g.x);
    o.y = float(double(p.w.y) - lr * g.y);
    o.z = float(double(p.w.z) - lr * g.z);
    o.w = float(double(p.w.w) - lr * g.w);
    *reinterpret_cast<f4*>(static_cast<float*>(d.w[t]) + size_t(r) * E + c4 * 4) = o;
  }
};

// Row update for split tables (Section VII): recombine hi/lo into the FP32
// weight, apply the FP32 update, split the result again.
struct SplitRows {
  struct Pre {
    u2 hi, lo;
  };
  static __device__ __forceinline__ Pre load(const TableDesc& d, int t, uint32_t r, int E, int c4) {
    const size_t off = size_t(r) * E + c4 * 4;
    return {*reinterpret_cast<const u2*>(static_cast<const uint16_t*>(d.w[t]) + off),
            *reinterpret_cast<const u2*>(static_cast<const uint16_t*>(d.lo[t]) + off)};
  }
  static __device__ __forceinline__ float upd(uint32_t hi16, uint32_t lo16, double g, double lr) {
    const float w = __uint_as_float((hi16 << 16) | lo16);
    return float(double(w) - lr * g);
  }
  static __device__ __forceinline__ void store(const TableDesc& d, int t, uint32_t r, int E, int c4,
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
    *reinterpret_cast<u2*>(static_cast<uint16_t*>(d.w[t]) + off) = hi;
    *reinterpret_cast<u2*>(static_cast<uint16_t*>(d.lo[t]) + off) = lo;
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

template <int LPR, int CPL, class Rows>
__global__ __launch_bounds__(kBlock) void segment_sgd(
    TableDesc d, const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks,
    const float* __restrict__ dY, int32_t B, float lr, double* __restrict__ carry,
    const int32_t* __restrict__ flags) {
  if (flags[0] != 0) return;  // data error: no table writes
  constexpr int R = kWave / LPR;
  constexpr int U = CPL == 1 ? 8 : (CPL == 2 ? 4 : 2);
  const int E = d.dim, E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int blk = int(xcd_remap(blockIdx.x, gridDim.x));
  const int chunk = (blk * kWavesPerBlock + wave_id()) * R + rg;
  if (chunk >= nchunks) return;
  const int lo = chunk * C, hi = min(lo + C, NS);
  const double lrd = double(lr);

  const uint32_t kprev = lo > 0 ? key_of(sorted[lo - 1]) : kNoKey;
  const uint32_t knext = hi < NS ? key_of(sorted[hi]) : kNoKey;
  const uint64_t p0 = sorted[lo];
  uint32_t cur = key_of(p0);
  int ct = int(bag_of(p0) / uint32_t(B));
  const bool first_open = kprev == cur;  // first segment began in an earlier chunk
  bool is_first = true;

  d4 acc[CPL];
  typename Rows::Pre pre[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    acc[j] = d4{0.0, 0.0, 0.0, 0.0};
    const int c4 = rl + j * LPR;
    if (!first_open && c4 < E4) pre[j] = Rows::load(d, ct, cur - d.rowbase[ct], E, c4);
  }

  for (int s = lo; s < hi; s += U) {
    uint64_t p[U];
    f4 g[U][CPL];
#pragma unroll
    for (int u = 0; u < U; ++u) p[u] = s + u < hi ? sorted[s + u] : 0ull;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float* gy = dY + size_t(bag_of(p[u])) * E;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c4 = rl + j * LPR;
        g[u][j] = (s + u < hi && c4 < E4) ? *reinterpret_cast<const f4*>(gy + c4 * 4)
                                          : f4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s + u >= hi) break;
      const uint32_t key = key_of(p[u]);
      if (key != cur) {
        if (is_first && first_open) {
          store_carry<CPL>(carry, 2 * int64_t(chunk), E, rl, LPR, acc);
        } else {
          const uint32_t r = cur - d.rowbase[ct];
#pragma unroll
          for (int j = 0; j < CPL; ++j) {
            const int c4 = rl + j * LPR;
            if (c4 < E4) Rows::store(d, ct, r, E, c4, pre[j], acc[j], lrd);
          }
        }
        cur = key;
        ct = int(bag_of(p[u]) / uint32_t(B));
        is_first = false;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          acc[j] = d4{0.0, 0.0, 0.0, 0.0};
          const int c4 = rl + j * LPR;
          if (c4 < E4) pre[j] = Rows::load(d, ct, cur - d.rowbase[ct], E, c4);
        }
      }
#pragma unroll
      for (int j = 0; j < CPL; ++j) acc[j] += widen(g[u][j]);
    }
  }

  const bool last_open = knext == cur;  // last segment continues in the next chunk
  if (is_first && (first_open || last_open)) {
    store_carry<CPL>(carry, 2 * int64_t(chunk), E, rl, LPR, acc);
  } else if (!is_first && last_open) {
    store_carry<CPL>(carry, 2 * int64_t(chunk) + 1, E, rl, LPR, acc);
  } else {
    const uint32_t r = cur - d.rowbase[ct];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c4 = rl + j * LPR;
      if (c4 < E4) Rows::store(d, ct, r, E, c4, pre[j], acc[j], lrd);
    }
  }
}

// Segments that cross chunk boundaries: the chunk where one begins sums the
// partials in chunk order and applies the row.
template <int LPR, int CPL, class Rows>
__global__ __launch_bounds__(kBlock) void segment_fixup(
    TableDesc d, const uint64_t* __restrict__ sorted, int32_t NS, int32_t C, int32_t nchunks,
    int32_t B, float lr, const double* __restrict__ carry, const int32_t* __restrict__ flags) {
  if (flags[0] != 0) return;
  constexpr int R = kWave / LPR;
  constexpr int UF = CPL == 1 ? 8 : (CPL == 2 ? 4 : 2);
  const int E = d.dim, E4 = E / 4;
  const int lane = lane_id();
  const int rg = lane / LPR, rl = lane % LPR;
  const int chunk = (int(blockIdx.x) * kWavesPerBlock + wave_id()) * R + rg;
  if (chunk >= nchunks) return;
  const int lo = chunk * C, hi = min(lo + C, NS);
  if (hi >= NS) return;
  const uint32_t kl = key_of(sorted[hi - 1]);
  if (key_of(sorted[hi]) != kl) return;             // last segment ends here
  const uint32_t kf = key_of(sorted[lo]);
  if (kf == kl && lo > 0 && key_of(sorted[lo - 1]) == kl) return;  // began earlier
  const int ct = int(bag_of(sorted[hi - 1]) / uint32_t(B));
  const uint32_t r = kl - d.rowbase[ct];
  const int64_t own = kf != kl ? 2 * int64_t(chunk) + 1 : 2 * int64_t(chunk);

  d4 acc[CPL];
  typename Rows::Pre pre[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c4 = rl + j * LPR;
    if (c4 < E4) {
      acc[j] = *reinterpret_cast<const d4*>(carry + own * E + c4 * 4);
      pre[j] = Rows::load(d, ct, r, E, c4);
    } else {
      acc[j] = d4{0.0, 0.0, 0.0, 0.0};
    }
  }
  // Chunks chunk+1, chunk+2, ... belong to the segment while the chunk before
  // continues it; UF chunks (their first-segment partials and the key just
  // past them) are loaded per step.
  bool inside = true;
  for (int c2 = chunk + 1; inside; c2 += UF) {
    d4 part[UF][CPL];
    uint32_t kn[UF];
#pragma unroll
    for (int u = 0; u < UF; ++u) {
      const int cu = c2 + u;
      const bool ok = cu < nchunks;
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
      if (!inside) break;
#pragma unroll
      for (int j = 0; j < CPL; ++j) acc[j] += part[u][j];
      inside = kn[u] == kl;
    }
  }
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c4 = rl + j * LPR;
    if (c4 < E4) Rows::store(d, ct, r, E, c4, pre[j], acc[j], double(lr));
  }
}

template <class Rows, int LPR, int CPL>
void launch_pair(int blocks_seg, int blocks_fix, hipStream_t st, const TableDesc& d,
                 const uint64_t* sorted, int32_t NS, int32_t C, int32_t nchunks, const float* dY,
                 int32_t B, float lr, double* carry, const int32_t* flags) {
  hipLaunchKernelGGL((segment_sgd<LPR, CPL, Rows>), dim3(blocks_seg), dim3(kBlock), 0, st, d,
                     sorted, NS, C, nchunks, dY, B, lr, carry, flags);
  hipLaunchKernelGGL((segment_fixup<LPR, CPL, Rows>), dim3(blocks_fix), dim3(kBlock), 0, st, d,
                     sorted, NS, C, nchunks, B, lr, carry, flags);
}

template <class Rows>
bool dispatch(RowGeom g, int bs, int bf, hipStream_t st, const TableDesc& d,
              const uint64_t* sorted, int32_t NS, int32_t C, int32_t nchunks, const float* dY,
              int32_t B, float lr, double* carry, const int32_t* flags) {
#define EMB_SEG(L, CC) launch_pair<Rows, L, CC>(bs, bf, st, d, sorted, NS, C, nchunks, dY, B, lr, carry, flags)
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

}  // namespace

hipError_t launch_segment_sgd(const TableDesc& d, bool split, int32_t B, const float* dY,
                              float lr, const uint64_t* sorted, const BwdLayout& L, char* ws,
                              hipStream_t st) {
  if (L.ns == 0) return hipSuccess;
  double* carry = reinterpret_cast<double*>(ws + L.off_carry);
  const int32_t* flags = reinterpret_cast<const int32_t*>(ws + L.off_flags);
  const RowGeom g = row_geom(d.dim);
  const int per_block = kWavesPerBlock * (kWave / g.lpr);
  const int blocks = int((L.nchunks + per_block - 1) / per_block);
  const bool ok = split ? dispatch<SplitRows>(g, blocks, blocks, st, d, sorted, int32_t(L.ns),
                                              int32_t(L.chunk), int32_t(L.nchunks), dY, B, lr,
                                              carry, flags)
                        : dispatch<Fp32Rows>(g, blocks, blocks, st, d, sorted, int32_t(L.ns),
                                             int32_t(L.chunk), int32_t(L.nchunks), dY, B, lr,
                                             carry, flags);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace embbag
