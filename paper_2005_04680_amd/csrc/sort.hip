// Integer work of the backward on gfx950: bag ids, keys, validation, a stable
// LSD radix sort of (key, bag) pairs, and (for the checking entry point) the
// unique keys with their segment offsets.
//
// A look-up s of bag k (table t = k / B) gets key = rowbase[t] + indices[s];
// it travels as one 64-bit word (key << 32 | k), so a stable sort on the key
// bits alone keeps the look-ups of one row in increasing s.  The sort is
// reduce-then-scan, one pass per digit of BITS = 6..10 bits (as few passes as
// the key width allows: 3 for 27- or 28-bit keys): a per-tile digit
// histogram, a scan per digit over the tiles, and a scatter in which every
// tile (1024, 2048 or 4096 keys: the largest that still gives two tiles per
// compute unit and two keys per digit value) is ranked in LDS (wavefront
// ballots give each lane its rank among equal digits) and written out in
// digit order, so that the global stores form runs of consecutive addresses.
// No kernel waits on another workgroup.
//
// Look-up positions are unsigned 32-bit: num_indices may be 2^31 - 1, and a
// tile's last slots run past it (by less than a tile), which stays below 2^32.
#include "common.hpp"

namespace embbag {
namespace {

// Inclusive scan across a wavefront (64 lanes).
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t n = __shfl_up(v, off, kWave);
    if (lane >= off) v += n;
  }
  return v;
}

// Exclusive scan of one value per thread over a 256-thread block; returns the
// exclusive prefix and writes the block total to *total.  `scratch` holds
// kWavesPerBlock + 1 words of LDS.  Every thread must call it.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch,
                                                         uint32_t* total) {
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const uint32_t inc = wave_inclusive_scan(v);
  if (lane == kWave - 1) scratch[w] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const uint32_t s = scratch[i];
    before += i < w ? s : 0u;
    all += s;
  }
  __syncthreads();
  *total = all;
  return before + inc - v;
}

// Scan of the per-tile digit counts: four digits (one 16-byte word of a
// tile's row) per block, kScanPer consecutive tiles per thread and round.
constexpr int kScanPer = 16;
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

// Digits handled per thread when a block walks all the digits of a radix.
template <int BITS>
struct Radix {
  static constexpr int R = 1 << BITS;
  static constexpr int DPT = R > kBlock ? R / kBlock : 1;
};

// Loads per thread requested before the first is used (the offsets in
// build_keys, the status words in the first scan).
constexpr int kOq = 8;

// Bags, keys and the first digit's histogram for one tile; offsets checks for
// a slice of the bags; one status word per block.  With per-look-up weights
// A, vals[s] = A[s] starts the value array that the sort carries along.
template <int BITS, int IPT>
__global__ __launch_bounds__(kBlock) void build_keys(
    TableDesc d, const int32_t* __restrict__ I, const int32_t* __restrict__ O, int32_t NS,
    int32_t B, float inv_b, int32_t TB, int32_t ntiles, int32_t vb, uint64_t* __restrict__ out,
    uint32_t* __restrict__ hist, int32_t* __restrict__ parts, const float* __restrict__ A,
    float* __restrict__ vals) {
  constexpr int R = Radix<BITS>::R;
  constexpr int TILE = kBlock * IPT;
  __shared__ uint32_t lbag[TILE];
  __shared__ uint32_t lhist[R];
  __shared__ int32_t lerr;
  __shared__ int32_t krange[2];
  // the tables' row counts and key bases, read per look-up (a per-lane index
  // into the kernel arguments would be a vector load for every look-up)
  __shared__ uint32_t srows[kMaxTables];
  __shared__ uint32_t srowbase[kMaxTables];
  const int tid = threadIdx.x;
  const int blk = blockIdx.x;
  const uint32_t s_lo = uint32_t(blk) * TILE;
  const uint32_t s_hi = min(s_lo + TILE, uint32_t(NS));
  // The tile's indices are requested first, so that they arrive while the
  // bag search below runs.
  int32_t rv[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const uint32_t s = s_lo + i * kBlock + tid;
    rv[i] = s < s_hi ? I[s] : 0;
  }
  int err = 0;
  if (tid == 0) lerr = 0;
  for (int i = tid; i < R; i += kBlock) lhist[i] = 0;
  if (tid < d.num_tables) {
    srows[tid] = d.rows[tid];
    srowbase[tid] = d.rowbase[tid];
  }
  __syncthreads();

  // Offsets: O[0] == 0, O non-decreasing, O[TB] == NS, all within [0, NS].
  // kOq offsets per thread are requested before any is checked (with one
  // look-up per bag a block checks thousands of them).
  // 64-bit: with both NS and T*B near 2^31, blk * vb passes 2^31 - 1.
  const int64_t kb0 = int64_t(blk) * vb, kb1 = min(kb0 + vb, int64_t(TB) + 1);
  for (int64_t k0 = kb0 + tid; k0 < kb1; k0 += kBlock * kOq) {
    int oa[kOq], ob[kOq];
#pragma unroll
    for (int q = 0; q < kOq; ++q) {
      const int64_t k = k0 + q * kBlock;
      oa[q] = k < kb1 ? O[k] : 0;
      ob[q] = k < kb1 && k < TB ? O[k + 1] : 0;
    }
#pragma unroll
    for (int q = 0; q < kOq; ++q) {
      const int64_t k = k0 + q * kBlock;
      if (k >= kb1) break;
      const int o = oa[q];
      if (o < 0 || o > NS || (k == 0 && o != 0) || (k == TB && o != NS)) err = EMBBAG_ERR_OFFSETS;
      if (k < TB && ob[q] < o) err = EMBBAG_ERR_OFFSETS;
    }
  }

  if (s_lo < s_hi) {  // uniform over the block
    for (int i = tid; i < TILE; i += kBlock) lbag[i] = 0;
    const int w = tid / kWave;
    if (w < 2) {
      // Last bag k in [0, TB - 1] with O[k] <= x, for the tile's first
      // (wave 0) and last (wave 1) look-up: a 64-way search, each lane
      // probing one of 64 evenly spaced bags of the current range per round
      // (ceil(log64 TB) dependent loads).  O[lo] <= x holds for valid O; a bad
      // O still leaves the range inside [0, TB - 1].
      const int lane = lane_id();
      const int x = int(w == 0 ? s_lo : s_hi - 1);
      int lo = 0, hi = TB - 1;
      while (lo < hi) {
        const int step = int((int64_t(hi) - lo + kWave) / kWave);  // ceil((hi - lo + 1) / 64)
        const int64_t k = lo + int64_t(lane) * step;
        const uint64_t m = __builtin_amdgcn_ballot_w64(k <= hi && O[k] <= x);
        const int j = m != 0 ? 63 - __builtin_clzll(m) : 0;
        lo = lo + j * step;
        hi = int(min(int64_t(lo) + step - 1, int64_t(hi)));
      }
      if (lane == 0) krange[w] = lo;
    }
    __syncthreads();
    // Expand bag ids over the tile's look-ups (kOq bags per thread requested
    // together).
    const int k1 = krange[1];
    for (int64_t k0 = krange[0] + tid; k0 <= k1; k0 += kBlock * kOq) {
      int oa[kOq], ob[kOq];
#pragma unroll
      for (int q = 0; q < kOq; ++q) {
        const int64_t k = k0 + q * kBlock;
        oa[q] = k <= k1 ? O[k] : 0;
        ob[q] = k <= k1 ? O[k + 1] : 0;
      }
#pragma unroll
      for (int q = 0; q < kOq; ++q) {
        const int64_t k = k0 + q * kBlock;
        if (k > k1) break;
        const int a = max(oa[q], int(s_lo)), b = min(ob[q], int(s_hi));
        for (int s = a; s < b; ++s) lbag[s - int(s_lo)] = uint32_t(k);
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const uint32_t s = s_lo + i * kBlock + tid;
      uint32_t key = 0;
      if (s < s_hi) {
        const uint32_t k = min(lbag[s - s_lo], uint32_t(TB - 1));
        const int t = table_of_bag(k, B, inv_b);
        int32_t r = rv[i];
        if (uint32_t(r) >= srows[t]) {
          err = min(err, EMBBAG_ERR_INDEX_RANGE);
          r = 0;
        }
        key = srowbase[t] + uint32_t(r);
        out[s] = (uint64_t(key) << 32) | k;
        if (A != nullptr) vals[s] = A[s];
      }
      if (s < s_hi) atomicAdd(&lhist[key & (R - 1)], 1u);
    }
    __syncthreads();
    for (int i = tid; i < R; i += kBlock) hist[size_t(blk) * R + i] = lhist[i];
  }
  if (err != 0) atomicMin(&lerr, err);
  __syncthreads();
  if (tid == 0) parts[blk] = lerr;
}

// Digit histogram of one tile of the current arrangement.
template <int BITS, int IPT>
__global__ __launch_bounds__(kBlock) void radix_upsweep(const uint64_t* __restrict__ src,
                                                        int32_t NS, int shift, int32_t ntiles,
                                                        uint32_t* __restrict__ hist) {
  constexpr int R = Radix<BITS>::R;
  __shared__ uint32_t lhist[R];
  const int tid = threadIdx.x, blk = blockIdx.x;
  for (int i = tid; i < R; i += kBlock) lhist[i] = 0;
  __syncthreads();
  // The keys arrive in the previous pass's order, so equal digits often
  // come in runs (every copy of a hot row is adjacent): within a wavefront,
  // the first lane of each run of equal digits adds the run's length.
  // All of the thread's keys are requested before the first is counted.
  const uint32_t base = uint32_t(blk) * (kBlock * IPT);
  const int lane = lane_id();
  uint32_t kv[IPT];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const uint32_t s = base + i * kBlock + tid;
    kv[i] = s < uint32_t(NS) ? key_of(src[s]) : 0u;
  }
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const uint32_t s = base + i * kBlock + tid;
    const uint32_t dg = s < uint32_t(NS) ? (kv[i] >> shift) & (R - 1) : uint32_t(R);
    const uint32_t left = __shfl_up(dg, 1, kWave);
    const bool head = lane == 0 || dg != left;
    const uint64_t heads = __builtin_amdgcn_ballot_w64(head);
    if (head && dg < uint32_t(R)) {
      const uint64_t after = lane == kWave - 1 ? 0ull : heads >> (lane + 1);
      const uint32_t len = after ? uint32_t(__builtin_ctzll(after)) + 1u : uint32_t(kWave - lane);
      atomicAdd(&lhist[dg], len);
    }
  }
  __syncthreads();
  for (int i = tid; i < R; i += kBlock) hist[size_t(blk) * R + i] = lhist[i];
}

// Block g < radix / 4 (after the XCD remap): for digits [4g, 4g + 4), the
// exclusive scan of the
// tile counts in tile order (hist is [tile][radix], rewritten in place: one
// 16-byte word per tile) and the digit totals.  Thread tid takes kScanPer
// consecutive tiles of each round of kBlock * kScanPer tiles.  The last
// block (first pass only) folds the per-block status words into this call's
// verdict and lowers the caller's status word.
__global__ __launch_bounds__(kBlock) void radix_scan(uint32_t* __restrict__ hist, int32_t ntiles,
                                                     int32_t radix,
                                                     uint32_t* __restrict__ totals,
                                                     const int32_t* __restrict__ parts,
                                                     int32_t nparts, int32_t* __restrict__ flags,
                                                     int32_t* __restrict__ d_status,
                                                     uint32_t token) {
  __shared__ u4 wsum[kWavesPerBlock];
  __shared__ int32_t lerr;
  const int tid = threadIdx.x;
  if (int(blockIdx.x) == radix / 4) {
    if (tid == 0) lerr = 0;
    __syncthreads();
    int e = 0;  // kOq words per thread requested before any is folded
    for (int i0 = tid; i0 < nparts; i0 += kBlock * kOq) {
      int v[kOq];
#pragma unroll
      for (int q = 0; q < kOq; ++q) v[q] = i0 + q * kBlock < nparts ? parts[i0 + q * kBlock] : 0;
#pragma unroll
      for (int q = 0; q < kOq; ++q) e = min(e, v[q]);
    }
    if (e != 0) atomicMin(&lerr, e);
    __syncthreads();
    if (tid == 0) {
      flags[0] = lerr;
      flags[1] = int32_t(token);
      if (lerr != 0 && d_status != nullptr) atomicMin(d_status, lerr);
    }
    return;
  }
  const int lane = lane_id(), w = tid / kWave;
  // Each XCD takes one contiguous range of the digit groups, so that the
  // blocks sharing a cache line of a tile's row share that XCD's L2.
  const uint32_t g = xcd_remap(blockIdx.x, uint32_t(radix / 4));
  u4* col = reinterpret_cast<u4*>(hist) + g;  // tile t's word: col[t * radix / 4]
  const size_t stride = size_t(radix / 4);
  u4 running = u4{0u, 0u, 0u, 0u};
  for (int base = 0; base < ntiles; base += kBlock * kScanPer) {
    const int t0 = base + tid * kScanPer;
    u4 v[kScanPer];
    u4 sum = u4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      v[q] = t0 + q < ntiles ? col[size_t(t0 + q) * stride] : u4{0u, 0u, 0u, 0u};
      sum += v[q];
    }
    // exclusive scan of `sum` over the block, four counts at once
    u4 inc = sum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      u4 n;
      n.x = __shfl_up(inc.x, off, kWave);
      n.y = __shfl_up(inc.y, off, kWave);
      n.z = __shfl_up(inc.z, off, kWave);
      n.w = __shfl_up(inc.w, off, kWave);
      if (lane >= off) inc += n;
    }
    if (lane == kWave - 1) wsum[w] = inc;
    __syncthreads();
    u4 before = u4{0u, 0u, 0u, 0u}, all = u4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i) {
      const u4 x = wsum[i];
      if (i < w) before += x;
      all += x;
    }
    __syncthreads();  // wsum is rewritten by the next round
    u4 ex = running + before + inc - sum;
#pragma unroll
    for (int q = 0; q < kScanPer; ++q) {
      if (t0 + q < ntiles) col[size_t(t0 + q) * stride] = ex;
      ex += v[q];
    }
    running += all;
  }
  if (tid == 0) reinterpret_cast<u4*>(totals)[g] = running;
}

// Stable scatter of one tile by the digit at `shift` (with VALS, the value
// of each key moves with it: vsrc[i] goes where src[i] goes).
// Four tiles per compute unit fit when the digits have at most 9 bits and no
// values travel along (LDS below 40 KB), three with values (below 53 KB):
// registers are then held to 128 or 168.
template <int BITS, int IPT, bool VALS>
__global__ __launch_bounds__(kBlock, BITS <= 9 ? (VALS ? 3 : 4) : 1) void radix_downsweep(
    const uint64_t* __restrict__ src, uint64_t* __restrict__ dst, int32_t NS, int shift,
    int32_t ntiles, const uint32_t* __restrict__ hist, const uint32_t* __restrict__ totals,
    const float* __restrict__ vsrc, float* __restrict__ vdst) {
  constexpr int R = Radix<BITS>::R;
  constexpr int DPT = Radix<BITS>::DPT;
  constexpr int TILE = kBlock * IPT;
  __shared__ uint64_t buf[TILE];
  __shared__ float vbuf[VALS ? TILE : 1];
  // Per-wave digit counts, then each wave's first position for a digit in
  // the locally sorted tile (at most TILE: 16 bits); once the tile is
  // sorted in LDS, the same memory holds each digit's global offset.
  union WaveDigits {
    uint16_t whist[kWavesPerBlock][R];
    uint32_t gofs[R];
  };
  __shared__ WaveDigits wd;
  auto& whist = wd.whist;
  __shared__ uint32_t scratch[kWavesPerBlock + 1];
  const int tid = threadIdx.x;
  // Each XCD takes one contiguous range of tiles: the runs that neighbouring
  // tiles write for one digit meet in cache lines of the same L2.
  const int blk = int(xcd_remap(blockIdx.x, gridDim.x));
  const int lane = lane_id();
  const int w = tid / kWave;

  // Wave w owns keys [w*64*IPT, (w+1)*64*IPT) of the tile, item i of lane l
  // being key w*64*IPT + i*64 + l: ranking item by item keeps the original
  // order.  The tile is requested first; the digit bases are computed while
  // it is in flight.
  const uint32_t wbase = uint32_t(blk) * TILE + w * (kWave * IPT);
  uint64_t item[IPT];
  float val[VALS ? IPT : 1];
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const uint32_t pos = wbase + i * kWave + lane;
    item[i] = pos < uint32_t(NS) ? src[pos] : ~0ull;
    if constexpr (VALS) val[i] = pos < uint32_t(NS) ? vsrc[pos] : 0.f;
  }

  // Global start of each digit's run for this tile (thread tid owns digits
  // [tid*DPT, tid*DPT + DPT)), kept as gbase - (start of the digit's run in
  // the locally sorted tile) once that start is known.
  uint32_t gb[DPT];
  {
    // the tile's own counts are requested with the totals (they do not
    // depend on the scan)
    uint32_t v[DPT], th[DPT], sum = 0;
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int dg = tid * DPT + i;
      v[i] = dg < R ? totals[dg] : 0u;
      th[i] = dg < R ? hist[size_t(blk) * R + dg] : 0u;
    }
#pragma unroll
    for (int i = 0; i < DPT; ++i) sum += v[i];
    uint32_t tot;
    uint32_t ex = block_exclusive_scan(sum, scratch, &tot);
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int dg = tid * DPT + i;
      gb[i] = dg < R ? ex + th[i] : 0u;
      ex += v[i];
    }
  }
  for (int i = tid; i < kWavesPerBlock * R; i += kBlock) (&whist[0][0])[i] = 0;
  __syncthreads();

  uint32_t dig[IPT];
  uint32_t rank[IPT];
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const bool valid = wbase + i * kWave + lane < uint32_t(NS);
    const uint32_t dg = (key_of(item[i]) >> shift) & (R - 1);
    dig[i] = dg;
    uint64_t peers = __builtin_amdgcn_ballot_w64(valid);
    // One digit across the wavefront (a run of equal keys, common after the
    // first pass): every valid lane is a peer.  Otherwise match bit by bit.
    const uint32_t d0 = __builtin_amdgcn_readfirstlane(dg);
    if (__builtin_amdgcn_ballot_w64(valid && dg != d0) != 0) {
      uint32_t plo = uint32_t(peers), phi = uint32_t(peers >> 32);
#pragma unroll
      for (int b = 0; b < BITS; ++b) {
        // keep the lanes whose bit b equals this lane's: peers & ~(m ^ s), s
        // all ones where the bit is set; one three-input logic op per half
        // (truth table 0x90 = f(0xF0, 0xCC, 0xAA) for f(a, b, c) = a & ~(b ^ c))
        const int32_t sb = __builtin_amdgcn_sbfe(int32_t(dg), b, 1);  // 0 or -1
        const uint64_t m = __builtin_amdgcn_ballot_w64(sb != 0);
        plo = __builtin_amdgcn_bitop3_b32(plo, uint32_t(m), uint32_t(sb), 0x90);
        phi = __builtin_amdgcn_bitop3_b32(phi, uint32_t(m >> 32), uint32_t(sb), 0x90);
      }
      peers = (uint64_t(phi) << 32) | plo;
    }
    const uint32_t lrank = uint32_t(__popcll(peers & below));
    const uint32_t cnt = uint32_t(__popcll(peers));
    const uint32_t prior = whist[w][dg];
    rank[i] = prior + lrank;
    if (valid && lrank == 0) whist[w][dg] = uint16_t(prior + cnt);
  }
  __syncthreads();
  uint32_t go[DPT];  // global offset of each owned digit's run, minus its local start
  {
    // Per digit: offsets of each wave's run inside the tile's digit run, and
    // the start of each digit's run in the locally sorted tile.
    uint32_t run[DPT], sum = 0;
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int dg = tid * DPT + i;
      uint32_t r = 0;
      if (dg < R) {
#pragma unroll
        for (int ww = 0; ww < kWavesPerBlock; ++ww) {
          const uint32_t c = whist[ww][dg];
          whist[ww][dg] = uint16_t(r);
          r += c;
        }
      }
      run[i] = r;
      sum += r;
    }
    uint32_t tot;
    uint32_t ex = block_exclusive_scan(sum, scratch, &tot);
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int dg = tid * DPT + i;
      if (dg < R) {
#pragma unroll
        for (int ww = 0; ww < kWavesPerBlock; ++ww) whist[ww][dg] = uint16_t(whist[ww][dg] + ex);
      }
      go[i] = gb[i] - ex;  // modulo 2^32: go + local position = global position
      ex += run[i];
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    if (wbase + i * kWave + lane < uint32_t(NS)) {
      const uint32_t at = whist[w][dig[i]] + rank[i];
      buf[at] = item[i];
      if constexpr (VALS) vbuf[at] = val[i];
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < DPT; ++i) {
    const int dg = tid * DPT + i;
    if (dg < R) wd.gofs[dg] = go[i];
  }
  __syncthreads();
  // The locally sorted tile, written out in order: each digit's keys land in
  // consecutive addresses.
  const int nvalid = min(TILE, NS - blk * TILE);
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int j = i * kBlock + tid;
    if (j < nvalid) {
      const uint64_t it = buf[j];
      const uint32_t to = wd.gofs[(key_of(it) >> shift) & (R - 1)] + uint32_t(j);
      dst[to] = it;
      if constexpr (VALS) vdst[to] = vbuf[j];
    }
  }
}

// ---- unique keys and segment offsets (checking entry point only) ----------

// Unpacks one tile and counts its segment heads.
template <int IPT>
__global__ __launch_bounds__(kBlock) void unique_count(const uint64_t* __restrict__ sorted,
                                                       int32_t NS, uint32_t* __restrict__ skeys,
                                                       uint32_t* __restrict__ sbags,
                                                       uint32_t* __restrict__ counts) {
  __shared__ uint32_t scratch[kWavesPerBlock + 1];
  const int tid = threadIdx.x, blk = blockIdx.x;
  uint32_t c = 0;
  for (int i = 0; i < IPT; ++i) {
    const uint32_t s = uint32_t(blk) * (kBlock * IPT) + i * kBlock + tid;
    if (s < uint32_t(NS)) {
      const uint64_t p = sorted[s];
      skeys[s] = key_of(p);
      sbags[s] = bag_of(p);
      c += (s == 0 || key_of(sorted[s - 1]) != key_of(p)) ? 1u : 0u;
    }
  }
  uint32_t tot;
  block_exclusive_scan(c, scratch, &tot);
  if (tid == 0) counts[blk] = tot;
}

// Exclusive scan of the per-tile head counts (one block); writes U and seg_off[U].
__global__ __launch_bounds__(kBlock) void unique_scan(uint32_t* __restrict__ counts,
                                                      int32_t ntiles, int32_t NS,
                                                      int32_t* __restrict__ seg_off,
                                                      int32_t* __restrict__ d_num_unique) {
  __shared__ uint32_t scratch[kWavesPerBlock + 1];
  const int tid = threadIdx.x;
  uint32_t running = 0;
  for (int base = 0; base < ntiles; base += kBlock) {
    const int i = base + tid;
    const uint32_t v = i < ntiles ? counts[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, scratch, &tot);
    if (i < ntiles) counts[i] = running + ex;
    running += tot;
  }
  if (tid == 0) {
    *d_num_unique = int32_t(running);
    seg_off[running] = NS;
  }
}

// Writes unique_keys[u] and seg_off[u] for the heads of one tile, in order.
template <int IPT>
__global__ __launch_bounds__(kBlock) void unique_write(const uint64_t* __restrict__ sorted,
                                                       int32_t NS,
                                                       const uint32_t* __restrict__ tile_off,
                                                       uint32_t* __restrict__ ukeys,
                                                       int32_t* __restrict__ seg_off) {
  __shared__ uint32_t scratch[kWavesPerBlock + 1];
  const int tid = threadIdx.x, blk = blockIdx.x;
  uint32_t running = tile_off[blk];
  for (int i = 0; i < IPT; ++i) {
    const uint32_t s = uint32_t(blk) * (kBlock * IPT) + i * kBlock + tid;
    bool head = false;
    uint32_t key = 0;
    if (s < uint32_t(NS)) {
      key = key_of(sorted[s]);
      head = s == 0 || key_of(sorted[s - 1]) != key;
    }
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(head ? 1u : 0u, scratch, &tot);
    if (head) {
      ukeys[running + ex] = key;
      seg_off[running + ex] = int32_t(s);
    }
    running += tot;
  }
}

template <int BITS, int IPT>
hipError_t sort_passes(const TableDesc& d, int32_t B, const int32_t* I, const int32_t* O,
                       int64_t NS, const BwdLayout& L, char* ws, int32_t* d_status,
                       uint32_t token, const float* A, hipStream_t st) {
  constexpr int R = Radix<BITS>::R;
  const int32_t TB = d.num_tables * B;
  uint64_t* a = reinterpret_cast<uint64_t*>(ws + L.off_a);
  uint64_t* b = reinterpret_cast<uint64_t*>(ws + L.off_b);
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.off_hist);
  uint32_t* totals = reinterpret_cast<uint32_t*>(ws + L.off_tot);
  int32_t* parts = reinterpret_cast<int32_t*>(ws + L.off_parts);
  int32_t* flags = reinterpret_cast<int32_t*>(ws + L.off_flags);
  const int nkb = int(L.nkeyblocks);
  const int vb = int((int64_t(TB) + 1 + nkb - 1) / nkb);
  const int ntiles = int(L.ntiles);
  const float inv_b = B > 0 ? 1.0f / float(B) : 0.0f;
  float* va = reinterpret_cast<float*>(ws + L.off_va);
  float* vb_ = reinterpret_cast<float*>(ws + L.off_vb);
  hipLaunchKernelGGL((build_keys<BITS, IPT>), dim3(nkb), dim3(kBlock), 0, st, d, I, O,
                     int32_t(NS), B, inv_b, TB, ntiles, vb, a, hist, parts, A, va);
  // Status verdict (block R of the first scan, or alone when nothing is sorted).
  const int passes = NS > 0 ? L.passes : 0;
  if (passes == 0) {
    hipLaunchKernelGGL(radix_scan, dim3(R / 4 + 1), dim3(kBlock), 0, st, hist, 0, R,
                       totals, parts, nkb, flags, d_status, token);
    return hipGetLastError();
  }
  uint64_t* src = a;
  uint64_t* dst = b;
  float* vsrc = va;
  float* vdst = vb_;
  for (int p = 0; p < passes; ++p) {
    const int shift = p * BITS;
    if (p > 0)
      hipLaunchKernelGGL((radix_upsweep<BITS, IPT>), dim3(ntiles), dim3(kBlock), 0, st, src,
                         int32_t(NS), shift, ntiles, hist);
    hipLaunchKernelGGL(radix_scan, dim3(R / 4 + (p == 0 ? 1 : 0)), dim3(kBlock), 0, st,
                       hist, ntiles, R, totals, parts, nkb, flags, d_status, token);
    if (A != nullptr)
      hipLaunchKernelGGL((radix_downsweep<BITS, IPT, true>), dim3(ntiles), dim3(kBlock), 0, st,
                         src, dst, int32_t(NS), shift, ntiles, hist, totals, vsrc, vdst);
    else
      hipLaunchKernelGGL((radix_downsweep<BITS, IPT, false>), dim3(ntiles), dim3(kBlock), 0, st,
                         src, dst, int32_t(NS), shift, ntiles, hist, totals, nullptr, nullptr);
    uint64_t* tmp = src;
    src = dst;
    dst = tmp;
    float* vt = vsrc;
    vsrc = vdst;
    vdst = vt;
  }
  return hipGetLastError();
}

template <int BITS>
hipError_t sort_ipt(const TableDesc& d, int32_t B, const int32_t* I, const int32_t* O, int64_t NS,
                    const BwdLayout& L, char* ws, int32_t* d_status, uint32_t token,
                    const float* A, hipStream_t st) {
  switch (L.ipt) {
    case 4: return sort_passes<BITS, 4>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 8: return sort_passes<BITS, 8>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 16: return sort_passes<BITS, 16>(d, B, I, O, NS, L, ws, d_status, token, A, st);
  }
  return hipErrorInvalidValue;
}

template <int IPT>
void unique_launch(const uint64_t* sorted, const BwdLayout& L, uint32_t* counts,
                   uint32_t* sorted_keys, uint32_t* sorted_bags, uint32_t* unique_keys,
                   int32_t* seg_off, int32_t* d_num_unique, hipStream_t st) {
  const int ntiles = int(L.ntiles);
  hipLaunchKernelGGL(unique_count<IPT>, dim3(ntiles), dim3(kBlock), 0, st, sorted, int32_t(L.ns),
                     sorted_keys, sorted_bags, counts);
  hipLaunchKernelGGL(unique_scan, dim3(1), dim3(kBlock), 0, st, counts, ntiles, int32_t(L.ns),
                     seg_off, d_num_unique);
  hipLaunchKernelGGL(unique_write<IPT>, dim3(ntiles), dim3(kBlock), 0, st, sorted, int32_t(L.ns),
                     counts, unique_keys, seg_off);
}

}  // namespace

hipError_t launch_sort(const TableDesc& d, int32_t B, const int32_t* I, const int32_t* O,
                       int64_t NS, const BwdLayout& L, char* ws, int32_t* d_status,
                       uint32_t token, const float* A, hipStream_t st) {
  switch (L.bits) {
    case 6: return sort_ipt<6>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 7: return sort_ipt<7>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 8: return sort_ipt<8>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 9: return sort_ipt<9>(d, B, I, O, NS, L, ws, d_status, token, A, st);
    case 10: return sort_ipt<10>(d, B, I, O, NS, L, ws, d_status, token, A, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_unique(const uint64_t* sorted, const BwdLayout& L, char* ws,
                         uint32_t* sorted_keys, uint32_t* sorted_bags, uint32_t* unique_keys,
                         int32_t* seg_off, int32_t* d_num_unique, hipStream_t st) {
  uint32_t* counts = reinterpret_cast<uint32_t*>(ws + L.off_uniq);
  if (L.ns == 0) {
    hipLaunchKernelGGL(unique_scan, dim3(1), dim3(kBlock), 0, st, counts, 0, 0, seg_off,
                       d_num_unique);
    return hipGetLastError();
  }
  switch (L.ipt) {
    case 4: unique_launch<4>(sorted, L, counts, sorted_keys, sorted_bags, unique_keys, seg_off,
                             d_num_unique, st); break;
    case 8: unique_launch<8>(sorted, L, counts, sorted_keys, sorted_bags, unique_keys, seg_off,
                             d_num_unique, st); break;
    case 16: unique_launch<16>(sorted, L, counts, sorted_keys, sorted_bags, unique_keys, seg_off,
                               d_num_unique, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace embbag
