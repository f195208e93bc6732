// Internal definitions shared by the gfx950 kernels and the host launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "embbag.h"

namespace embbag {

constexpr int kMaxTables = 64;
constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kBlock = 256;        // threads per workgroup (4 waves)
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kNumXcd = 8;         // MI355X: 8 XCDs, each with its own L2
constexpr int kNumCu = 256;        // compute units (32 per XCD)
constexpr int kMaxBlocksPerCu = 8; // 32 wavefronts per CU, 4 per block
constexpr int64_t kMallBytes = int64_t(256) << 20;  // Infinity Cache (MALL)

// Radix sort geometry: digits of 6..10 bits, tiles of 256 threads x 4, 8 or
// 16 keys.
constexpr int kMaxRadixBits = 10;
constexpr int kMaxRadix = 1 << kMaxRadixBits;
constexpr int kMaxItemsPerThread = 16;  // radix tile: kBlock * (4, 8 or 16) keys
constexpr int kCarryGroup = 16;  // chunks per pre-summed group of carries
constexpr int64_t kOffsetsPerBlock = 16384;  // offsets a key-build block validates, at most

// Sentinel for "no key": keys are < 2^31 because sum(M_t) < 2^31.
constexpr uint32_t kNoKey = 0xFFFFFFFFu;

typedef float f4 __attribute__((ext_vector_type(4)));
typedef double d4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

// Table descriptor, passed by value as a kernel argument (kernarg segment).
// For FP32 tables `w[t]` is the table; for split tables `w[t]` is the BF16
// high half and `lo[t]` the low half.
struct TableDesc {
  void* w[kMaxTables];
  void* lo[kMaxTables];
  uint32_t rows[kMaxTables];
  uint32_t rowbase[kMaxTables + 1];
  int32_t num_tables;
  int32_t dim;
};

// The per-table pointers and key bases, copied to LDS by kernels whose
// wavefronts hold several row groups: there the table number differs per
// lane, and a per-lane index into the kernel arguments is a vector load.
struct TableLds {
  void* w[kMaxTables];
  void* lo[kMaxTables];
  uint32_t rowbase[kMaxTables + 1];
};

// Every thread of the block must call it; a barrier must follow.
__device__ __forceinline__ void stage_tables(const TableDesc& d, TableLds& s) {
  const int i = threadIdx.x;
  if (i < d.num_tables) {
    s.w[i] = d.w[i];
    s.lo[i] = d.lo[i];
  }
  if (i <= d.num_tables) s.rowbase[i] = d.rowbase[i];
}

// The LDS copy where the table number is per lane, the kernel arguments
// (scalar loads) where it is uniform over the wavefront.
template <bool kLds>
__device__ __forceinline__ const auto& table_view(const TableDesc& d, const TableLds& s) {
  if constexpr (kLds)
    return s;
  else
    return d;
}

// Element `off` of a table (elements of type S) as a global-memory pointer to
// V.  Table pointers that a kernel staged in LDS come back as generic
// pointers, and a generic (flat) access counts against the LDS wait counter
// as well as the vector-memory one: every later LDS read would wait until the
// row loads and stores in flight had completed.  Tables are always in global
// memory.
template <class V, class S>
__device__ __forceinline__ __attribute__((address_space(1))) V* table_elem(void* p, size_t off) {
  return (__attribute__((address_space(1))) V*)(static_cast<S*>(p) + off);
}

// Lane geometry for a row of E floats: LPR lanes per row (power of two), each
// lane owning CPL groups of 4 consecutive columns, 64/LPR rows per wavefront.
struct RowGeom {
  int lpr;
  int cpl;
};

inline RowGeom row_geom(int dim) {
  const int e4 = dim / 4;
  int lpr = 1;
  while (lpr < e4 && lpr < kWave) lpr *= 2;
  const int cpl = (e4 + lpr - 1) / lpr;
  return {lpr, cpl};
}

// Blocks are handed to the 8 XCDs round-robin (block b runs on XCD b % 8).
// Remap so that each XCD receives one contiguous range of logical blocks:
// neighbouring bags (the same table) then share one XCD's L2.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t n) {
  const uint32_t xcd = b % kNumXcd, idx = b / kNumXcd;
  const uint32_t q = n / kNumXcd, r = n % kNumXcd;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// Order in which a grid walks its logical blocks (bags or chunks in table
// order).  With per-XCD ranges (xcd_remap) each XCD works through its own
// tables: the rows a table reuses stay in that XCD's L2, but about
// kNumXcd + resident / blocks_per_table tables are in flight at once, one or
// more per XCD.  In dispatch order the resident blocks form one window over
// the grid, about 1 + resident / blocks_per_table tables wide, that every XCD
// shares: each L2 then sees more tables, but the MALL, which serves the
// reuse the L2s miss, holds fewer.  Dispatch order is taken when the grid does
// not fit the chip at once and the reused data of the tables that per-XCD
// ranges put in flight (per_table_bytes each) exceeds half of the MALL (the
// rest of it carries the streams that pass through).
inline bool dispatch_order(int64_t blocks, int32_t num_tables, int64_t per_table_bytes) {
  const int64_t resident = int64_t(kNumCu) * kMaxBlocksPerCu;
  if (blocks <= resident || num_tables <= 0) return false;
  const double in_flight = double(kNumXcd) + double(resident) * num_tables / double(blocks);
  return in_flight * double(per_table_bytes) > double(kMallBytes) / 2;
}

// The update's order: a table's reused data there is its dY, B rows of E
// gradients of dy_bytes each.
inline bool apply_in_dispatch_order(int64_t blocks, int32_t T, int32_t B, int32_t E,
                                    int dy_bytes) {
  return dispatch_order(blocks, T, int64_t(B) * E * dy_bytes);
}

__device__ __forceinline__ uint32_t logical_block(bool in_dispatch_order) {
  return in_dispatch_order ? blockIdx.x : xcd_remap(blockIdx.x, gridDim.x);
}

__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x % kWave; }

// Table of bag k = t*B + b, without an integer division: the FP32 estimate
// is off by at most one for any k < 2^31 and T <= 64, and is then corrected.
__device__ __forceinline__ int table_of_bag(uint32_t k, int B, float inv_b) {
  int t = int(float(k) * inv_b);
  t -= int(uint32_t(t) * uint32_t(B) > k);
  t += int(uint32_t(t + 1) * uint32_t(B) <= k);
  return t;
}

__device__ __forceinline__ uint32_t key_of(uint64_t p) { return uint32_t(p >> 32); }
__device__ __forceinline__ uint32_t bag_of(uint64_t p) { return uint32_t(p); }

// Pooling of a bag (Section II's L = A^T W): plain sum (Algorithm 1), sum
// weighted by one weight per look-up, or mean (sum / number of look-ups).
enum PoolMode : int { kPoolPlain = 0, kPoolWeighted = 1, kPoolMean = 2 };

struct PoolArgs {
  int mode = kPoolPlain;
  const float* weights = nullptr;   // kPoolWeighted: [num_indices]
  const int32_t* offsets = nullptr; // kPoolMean: bag sizes for the backward
};

// ---- launchers (host) ------------------------------------------------------
struct BwdLayout {
  int64_t ns;
  int ipt;             // keys per thread of a radix tile (4, 8 or 16)
  int64_t ntiles;      // radix tiles of kBlock * ipt keys
  int64_t nkeyblocks;  // blocks of the key-build kernel
  int64_t chunk;       // sorted look-ups per segment-reduce chunk
  int64_t nchunks;
  int passes;          // radix passes
  int bits;            // digit width of every pass
  int64_t ngroups;     // groups of kCarryGroup chunks
  size_t off_a, off_b, off_hist, off_tot, off_parts, off_flags, off_carry, off_uniq, off_va,
      off_vb, off_gsum, off_gflag,
      total;
};

BwdLayout backward_layout(int32_t T, int32_t B, int64_t NS, int32_t E, uint32_t total_rows,
                          bool for_dedup);

// Stamp the sort phase leaves in the workspace for the apply phase: a hash of
// the sizes the sorted look-ups and the workspace layout belong to and of
// their payload (never 0).
uint32_t phase_token(int32_t T, int32_t B, int64_t NS, int32_t E, uint32_t total_rows,
                     int mode);

// The buffer that holds the sorted look-ups after the sort phase.
inline uint64_t* sorted_buffer(const BwdLayout& L, char* ws) {
  const int passes = L.ns > 0 ? L.passes : 0;
  return reinterpret_cast<uint64_t*>(ws + (passes % 2 == 0 ? L.off_a : L.off_b));
}

// The per-look-up weights in sorted order (weighted bags), beside it.
inline float* sorted_values(const BwdLayout& L, char* ws) {
  const int passes = L.ns > 0 ? L.passes : 0;
  return reinterpret_cast<float*>(ws + (passes % 2 == 0 ? L.off_va : L.off_vb));
}

// Y is FP32 [T*B][E], or (y_bf16, split tables only) BF16 bit patterns.
hipError_t launch_forward(const TableDesc& d, bool split, int32_t B, const int32_t* I,
                          const int32_t* O, int64_t NS, void* Y, bool y_bf16, int32_t* status,
                          const PoolArgs& pool, hipStream_t st);

// Builds keys, validates, sorts into sorted_buffer(L, ws); stamps `token`.
// The payload of a sorted word is the bag; with per-look-up weights A, the
// weights are sorted along into sorted_values(L, ws).
hipError_t launch_sort(const TableDesc& d, int32_t B, const int32_t* I, const int32_t* O,
                       int64_t NS, const BwdLayout& L, char* ws, int32_t* d_status,
                       uint32_t token, const float* A, hipStream_t st);

// dY is FP32 [T*B][E], or (dy_bf16, split tables only) BF16 bit patterns.
hipError_t launch_segment_sgd(const TableDesc& d, bool split, int32_t B, const void* dY,
                              bool dy_bf16, float lr, const BwdLayout& L, char* ws,
                              uint32_t token, const PoolArgs& pool, hipStream_t st);

hipError_t launch_unique(const uint64_t* sorted, const BwdLayout& L, char* ws,
                         uint32_t* sorted_keys, uint32_t* sorted_bags, uint32_t* unique_keys,
                         int32_t* seg_off, int32_t* d_num_unique, hipStream_t st);

// Baselines: the paper's unfused designs (Algorithms 2, 3, 4) on the GPU.
hipError_t launch_materialize(const float* dY, const int32_t* O, int64_t NS, int32_t T, int32_t B,
                              int32_t E, float* dW, int32_t* status, hipStream_t st);
hipError_t launch_atomic_update(const TableDesc& d, const float* src, bool fused,
                                const int32_t* I, const int32_t* O, int64_t NS, int32_t B,
                                float lr, int32_t* status, hipStream_t st);
hipError_t launch_owner_update(const TableDesc& d, const float* dW, const int32_t* I,
                               const int32_t* O, int64_t NS, int32_t B, int32_t owners, float lr,
                               hipStream_t st);

// Floor of the update: reads and writes back (unchanged) every row that the
// sorted look-ups of a prepared workspace touch, once (split rows: both halves).
hipError_t launch_touch_rows(const TableDesc& d, bool split, int32_t B, const BwdLayout& L,
                             char* ws, uint32_t token, hipStream_t st);

hipError_t launch_split(const float* w, uint16_t* hi, uint16_t* lo, int64_t n, hipStream_t st);
hipError_t launch_combine(const uint16_t* hi, const uint16_t* lo, float* w, int64_t n,
                          hipStream_t st);

}  // namespace embbag
