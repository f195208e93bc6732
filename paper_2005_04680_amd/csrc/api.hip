// C ABI of the EmbeddingBag library: argument checks, workspace layout and
// the launch sequence of each entry point on the caller's stream.
#include <cstring>

#include "common.hpp"

using namespace embbag;

namespace {

constexpr int64_t kInt32Max = 2147483647;
// Look-ups per call: indices and offsets are int32 (Algorithm 1's I[NS] and
// O[N+1]), so at most 2^31 - 1.  The kernels hold look-up positions in
// unsigned 32-bit arithmetic, where stepping a tile or a chunk past the last
// look-up still stays below 2^32.
constexpr int64_t kMaxIndices = kInt32Max;
constexpr size_t kWsAlign = 256;

bool aligned(const void* p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Table shapes (and, when `w` is given, the per-table device pointers).
int make_desc(int32_t T, int32_t E, const int64_t* rows, void* const* w, void* const* lo,
              size_t align, TableDesc* d) {
  if (T < 1 || T > kMaxTables) return EMBBAG_ERR_INVALID_ARG;
  if (E < 4 || E > 1024 || E % 4 != 0) return EMBBAG_ERR_INVALID_ARG;
  if (rows == nullptr) return EMBBAG_ERR_INVALID_ARG;
  std::memset(d, 0, sizeof(*d));
  int64_t total = 0;
  for (int t = 0; t < T; ++t) {
    if (rows[t] < 1 || rows[t] > kInt32Max) return EMBBAG_ERR_INVALID_ARG;
    if (align != 0) {
      if (w == nullptr || w[t] == nullptr || !aligned(w[t], align)) return EMBBAG_ERR_INVALID_ARG;
      d->w[t] = w[t];
      if (lo != nullptr) {
        if (lo[t] == nullptr || !aligned(lo[t], align)) return EMBBAG_ERR_INVALID_ARG;
        d->lo[t] = lo[t];
      }
    }
    d->rows[t] = uint32_t(rows[t]);
    d->rowbase[t] = uint32_t(total);
    total += rows[t];
  }
  if (total > kInt32Max) return EMBBAG_ERR_INVALID_ARG;
  d->rowbase[T] = uint32_t(total);
  d->num_tables = T;
  d->dim = E;
  return EMBBAG_OK;
}

int check_bags(int32_t T, int32_t B, const int32_t* I, const int32_t* O, int64_t NS) {
  if (B < 0 || NS < 0 || NS > kMaxIndices) return EMBBAG_ERR_INVALID_ARG;
  if (int64_t(T) * B + 1 > kInt32Max) return EMBBAG_ERR_INVALID_ARG;
  if (O == nullptr || (NS > 0 && I == nullptr)) return EMBBAG_ERR_INVALID_ARG;
  // offsets[0] must be both 0 and num_indices: the sizes alone contradict.
  if (int64_t(T) * B == 0 && NS > 0) return EMBBAG_ERR_OFFSETS;
  return EMBBAG_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? EMBBAG_OK : EMBBAG_ERR_HIP; }

// Pooling from the public (weights, pooling) pair; -1 if the pair is invalid
// (weights are defined for sum pooling only).
int pool_mode(const float* weights, int32_t pooling) {
  if (pooling == EMBBAG_POOL_SUM) return weights ? kPoolWeighted : kPoolPlain;
  if (pooling == EMBBAG_POOL_MEAN && weights == nullptr) return kPoolMean;
  return -1;
}

// Pooled outputs and their gradients: FP32 (16-B aligned rows of float4) or
// BF16 bit patterns (8-B aligned).
int forward_common(const TableDesc& d, bool split, int32_t B, const int32_t* I, const int32_t* O,
                   int64_t NS, void* Y, bool y_bf16, int32_t* d_status, const PoolArgs& pool,
                   hipStream_t st) {
  int rc = check_bags(d.num_tables, B, I, O, NS);
  if (rc) return rc;
  if (int64_t(d.num_tables) * B > 0 && (Y == nullptr || !aligned(Y, y_bf16 ? 8 : 16)))
    return EMBBAG_ERR_INVALID_ARG;
  return hip_status(launch_forward(d, split, B, I, O, NS, Y, y_bf16, d_status, pool, st));
}

// `weights` (weighted bags only) are sorted along with the look-ups.
int prepare_common(const TableDesc& d, int32_t B, const int32_t* I, const int32_t* O, int64_t NS,
                   void* ws, size_t ws_bytes, int32_t* d_status, int mode, const float* weights,
                   hipStream_t st) {
  int rc = check_bags(d.num_tables, B, I, O, NS);
  if (rc) return rc;
  if (mode == kPoolWeighted && NS > 0 && weights == nullptr) return EMBBAG_ERR_INVALID_ARG;
  const uint32_t total = d.rowbase[d.num_tables];
  const BwdLayout L = backward_layout(d.num_tables, B, NS, d.dim, total, false);
  if (ws == nullptr || !aligned(ws, kWsAlign) || ws_bytes < L.total) return EMBBAG_ERR_WORKSPACE;
  return hip_status(launch_sort(d, B, I, O, NS, L, static_cast<char*>(ws), d_status,
                                phase_token(d.num_tables, B, NS, d.dim, total, mode),
                                mode == kPoolWeighted ? weights : nullptr, st));
}

int apply_common(const TableDesc& d, bool split, const void* dY, bool dy_bf16, int32_t B,
                 int64_t NS, float lr, void* ws, size_t ws_bytes, const PoolArgs& pool,
                 hipStream_t st) {
  if (B < 0 || NS < 0 || NS > kMaxIndices || int64_t(d.num_tables) * B + 1 > kInt32Max)
    return EMBBAG_ERR_INVALID_ARG;
  if (int64_t(d.num_tables) * B == 0 && NS > 0) return EMBBAG_ERR_OFFSETS;
  if (NS > 0 && (dY == nullptr || !aligned(dY, dy_bf16 ? 8 : 16))) return EMBBAG_ERR_INVALID_ARG;
  const uint32_t total = d.rowbase[d.num_tables];
  const BwdLayout L = backward_layout(d.num_tables, B, NS, d.dim, total, false);
  if (ws == nullptr || !aligned(ws, kWsAlign) || ws_bytes < L.total) return EMBBAG_ERR_WORKSPACE;
  return hip_status(launch_segment_sgd(d, split, B, dY, dy_bf16, lr, L, static_cast<char*>(ws),
                                       phase_token(d.num_tables, B, NS, d.dim, total, pool.mode),
                                       pool, st));
}

int backward_common(const TableDesc& d, bool split, const void* dY, bool dy_bf16, int32_t B,
                    const int32_t* I, const int32_t* O, int64_t NS, float lr, void* ws,
                    size_t ws_bytes, int32_t* d_status, const PoolArgs& pool, hipStream_t st) {
  int rc = check_bags(d.num_tables, B, I, O, NS);
  if (rc) return rc;
  if (NS > 0 && (dY == nullptr || !aligned(dY, dy_bf16 ? 8 : 16))) return EMBBAG_ERR_INVALID_ARG;
  if (pool.mode == kPoolWeighted && NS > 0 && pool.weights == nullptr) return EMBBAG_ERR_INVALID_ARG;
  rc = prepare_common(d, B, I, O, NS, ws, ws_bytes, d_status, pool.mode, pool.weights, st);
  if (rc) return rc;
  return apply_common(d, split, dY, dy_bf16, B, NS, lr, ws, ws_bytes, pool, st);
}

// Split tables (hi halves, and lo halves when `need_lo`): 8-B aligned.
int split_desc(const embbag_split_tables_t* tables, bool need_lo, TableDesc* d) {
  if (tables == nullptr || (need_lo && tables->lo == nullptr)) return EMBBAG_ERR_INVALID_ARG;
  return make_desc(tables->num_tables, tables->dim, tables->rows,
                   reinterpret_cast<void* const*>(tables->hi),
                   need_lo ? reinterpret_cast<void* const*>(tables->lo) : nullptr, 8, d);
}

}  // namespace

namespace embbag {

uint32_t phase_token(int32_t T, int32_t B, int64_t NS, int32_t E, uint32_t total_rows,
                     int mode) {
  // A weighted prepare also sorts the weights along; the others do not.  E
  // sizes the carry regions, which the sorted weights follow.
  const uint64_t payload = mode == kPoolWeighted ? 1u : 0u;
  uint64_t h = 0x243F6A8885A308D3ull;
  for (uint64_t v : {uint64_t(uint32_t(T)), uint64_t(uint32_t(B)), uint64_t(NS),
                     uint64_t(uint32_t(E)), uint64_t(total_rows), payload}) {
    h ^= v + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
    h *= 0xBF58476D1CE4E5B9ull;
  }
  const uint32_t t = uint32_t(h ^ (h >> 32));
  return t == 0 ? 1u : t;
}

BwdLayout backward_layout(int32_t T, int32_t B, int64_t NS, int32_t E, uint32_t total_rows,
                          bool for_dedup) {
  BwdLayout L{};
  L.ns = NS;
  // As few passes as digits of at most 10 bits allow, the bits spread evenly
  // over them (27-bit keys: 3 passes of 9 bits).
  int nbits = 0;
  if (total_rows > 1) nbits = 32 - __builtin_clz(total_rows - 1u);
  L.passes = (nbits + kMaxRadixBits - 1) / kMaxRadixBits;
  L.bits = L.passes > 0 ? (nbits + L.passes - 1) / L.passes : 6;
  if (L.bits < 6) L.bits = 6;
  // Radix tiles: the largest of 4096, 2048 or 1024 keys that still gives at
  // least 512 tiles (two per compute unit), but at least 2 keys per digit
  // value (a tile's scatter then writes runs, not single words; 1.7M keys of
  // 10-bit digits: 832 tiles of 2048 sort faster than 416 of 4096).  Sizes
  // only shrink as the key width grows, so the workspace computed without
  // the table sizes (6-bit digits) covers every call.
  const int ipt_min = (1 << L.bits) / 128 > 4 ? (1 << L.bits) / 128 : 4;
  L.ipt = kMaxItemsPerThread;
  while (L.ipt > ipt_min &&
         (NS + int64_t(kBlock) * L.ipt - 1) / (int64_t(kBlock) * L.ipt) < 512)
    L.ipt /= 2;
  L.ntiles = (NS + int64_t(kBlock) * L.ipt - 1) / (int64_t(kBlock) * L.ipt);
  // Key-build blocks: one per tile, and at least one per kOffsetsPerBlock
  // offsets, which they validate (with few look-ups in many bags, one block
  // per tile would leave all the offsets to a handful of blocks).
  const int64_t vblocks = (int64_t(T) * B + 1 + kOffsetsPerBlock - 1) / kOffsetsPerBlock;
  L.nkeyblocks = L.ntiles > vblocks ? L.ntiles : vblocks;
  if (L.nkeyblocks < 1) L.nkeyblocks = 1;
  // Chunk of the segmented reduce: at least 128 look-ups per wavefront (a
  // wavefront walks one chunk per row group), growing to at most 1024 while
  // at least ~32K wavefronts remain (Large: 256 look-ups, 51K wavefronts;
  // measured 2% faster than 512).
  const int64_t rgw = kWave / row_geom(E).lpr;
  int64_t c = 128 / rgw > 8 ? 128 / rgw : 8;
  while (c < 1024 && c * 2 * 32768 * rgw <= NS) c *= 2;
  L.chunk = c;
  L.nchunks = (NS + c - 1) / c;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = round_up(off + bytes, kWsAlign);
    return o;
  };
  L.off_a = take(size_t(NS) * 8);
  L.off_b = take(size_t(NS) * 8);
  L.off_hist = take(size_t(kMaxRadix) * size_t(L.ntiles) * 4);
  L.off_tot = take(size_t(kMaxRadix) * 4);
  L.off_parts = take(size_t(L.nkeyblocks) * 4);
  L.off_flags = take(64);
  L.off_carry = take(for_dedup ? 0 : size_t(2) * size_t(L.nchunks) * size_t(E) * 8);
  L.off_uniq = take(for_dedup ? size_t(L.ntiles) * 4 : 0);
  L.off_va = take(for_dedup ? 0 : size_t(NS) * 4);
  L.off_vb = take(for_dedup ? 0 : size_t(NS) * 4);
  L.ngroups = (L.nchunks + kCarryGroup - 1) / kCarryGroup;
  L.off_gsum = take(for_dedup ? 0 : size_t(L.ngroups) * size_t(E) * 8);
  L.off_gflag = take(for_dedup ? 0 : size_t(L.ngroups) * 4);
  L.total = off;
  return L;
}

}  // namespace embbag

extern "C" {

const char* embbag_status_string(int code) {
  switch (code) {
    case EMBBAG_OK: return "ok";
    case EMBBAG_ERR_INVALID_ARG: return "invalid argument";
    case EMBBAG_ERR_WORKSPACE: return "workspace too small or misaligned";
    case EMBBAG_ERR_INDEX_RANGE: return "index out of its table's range";
    case EMBBAG_ERR_OFFSETS: return "invalid offsets";
    case EMBBAG_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

int embbag_forward(const embbag_tables_t* tables, int32_t batch, const int32_t* indices,
                   const int32_t* offsets, int64_t num_indices, float* pooled_out,
                   int32_t* d_status, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  return forward_common(d, false, batch, indices, offsets, num_indices, pooled_out, false,
                        d_status, PoolArgs{}, stream);
}

int embbag_forward_pooled(const embbag_tables_t* tables, int32_t batch, const int32_t* indices,
                          const int32_t* offsets, int64_t num_indices,
                          const float* per_sample_weights, int32_t pooling, float* pooled_out,
                          int32_t* d_status, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  const int mode = pool_mode(per_sample_weights, pooling);
  if (mode < 0) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  PoolArgs pool;
  pool.mode = mode;
  pool.weights = per_sample_weights;
  pool.offsets = offsets;
  return forward_common(d, false, batch, indices, offsets, num_indices, pooled_out, false,
                        d_status, pool, stream);
}

int embbag_forward_split_bf16(const embbag_split_tables_t* tables, int32_t batch,
                              const int32_t* indices, const int32_t* offsets,
                              int64_t num_indices, float* pooled_out, int32_t* d_status,
                              hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->hi), nullptr, 8, &d);
  if (rc) return rc;
  return forward_common(d, true, batch, indices, offsets, num_indices, pooled_out, false,
                        d_status, PoolArgs{}, stream);
}

size_t embbag_backward_workspace_bytes(int32_t num_tables, int32_t batch, int64_t num_indices,
                                       int32_t dim) {
  if (num_tables < 1 || num_tables > kMaxTables || dim < 4 || dim > 1024 || dim % 4 != 0)
    return 0;
  if (batch < 0 || num_indices < 0 || num_indices > kMaxIndices) return 0;
  if (int64_t(num_tables) * batch + 1 > kInt32Max) return 0;
  return backward_layout(num_tables, batch, num_indices, dim, 0, false).total;
}

int embbag_backward_sgd(const float* grad_pooled, int32_t batch, const int32_t* indices,
                        const int32_t* offsets, int64_t num_indices, float lr,
                        const embbag_tables_t* tables, void* workspace, size_t workspace_bytes,
                        int32_t* d_status, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  return backward_common(d, false, grad_pooled, false, batch, indices, offsets, num_indices, lr,
                         workspace, workspace_bytes, d_status, PoolArgs{}, stream);
}

int embbag_backward_sgd_pooled(const float* grad_pooled, int32_t batch, const int32_t* indices,
                               const int32_t* offsets, int64_t num_indices,
                               const float* per_sample_weights, int32_t pooling, float lr,
                               const embbag_tables_t* tables, void* workspace,
                               size_t workspace_bytes, int32_t* d_status, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  const int mode = pool_mode(per_sample_weights, pooling);
  if (mode < 0) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  PoolArgs pool;
  pool.mode = mode;
  pool.weights = per_sample_weights;
  pool.offsets = offsets;
  return backward_common(d, false, grad_pooled, false, batch, indices, offsets, num_indices, lr,
                         workspace, workspace_bytes, d_status, pool, stream);
}

int embbag_backward_prepare_pooled(int32_t num_tables, const int64_t* rows, int32_t dim,
                                   int32_t batch, const int32_t* indices, const int32_t* offsets,
                                   int64_t num_indices, const float* per_sample_weights,
                                   int32_t pooling, void* workspace, size_t workspace_bytes,
                                   int32_t* d_status, hipStream_t stream) {
  const int mode = pool_mode(per_sample_weights, pooling);
  if (mode < 0) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(num_tables, dim, rows, nullptr, nullptr, 0, &d);
  if (rc) return rc;
  return prepare_common(d, batch, indices, offsets, num_indices, workspace, workspace_bytes,
                        d_status, mode, per_sample_weights, stream);
}

int embbag_backward_apply_sgd_pooled(const float* grad_pooled, int32_t batch,
                                     const int32_t* offsets, int64_t num_indices,
                                     const float* per_sample_weights, int32_t pooling, float lr,
                                     const embbag_tables_t* tables, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  const int mode = pool_mode(per_sample_weights, pooling);
  if (mode < 0) return EMBBAG_ERR_INVALID_ARG;
  if (mode == kPoolMean && num_indices > 0 && offsets == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  PoolArgs pool;
  pool.mode = mode;
  pool.weights = per_sample_weights;
  pool.offsets = offsets;
  return apply_common(d, false, grad_pooled, false, batch, num_indices, lr, workspace,
                      workspace_bytes, pool, stream);
}

int embbag_backward_sgd_split_bf16(const float* grad_pooled, int32_t batch,
                                   const int32_t* indices, const int32_t* offsets,
                                   int64_t num_indices, float lr,
                                   const embbag_split_tables_t* tables, void* workspace,
                                   size_t workspace_bytes, int32_t* d_status,
                                   hipStream_t stream) {
  if (tables == nullptr || tables->lo == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->hi),
                     reinterpret_cast<void* const*>(tables->lo), 8, &d);
  if (rc) return rc;
  return backward_common(d, true, grad_pooled, false, batch, indices, offsets, num_indices, lr,
                         workspace, workspace_bytes, d_status, PoolArgs{}, stream);
}

int embbag_backward_prepare(int32_t num_tables, const int64_t* rows, int32_t dim, int32_t batch,
                            const int32_t* indices, const int32_t* offsets, int64_t num_indices,
                            void* workspace, size_t workspace_bytes, int32_t* d_status,
                            hipStream_t stream) {
  TableDesc d;
  int rc = make_desc(num_tables, dim, rows, nullptr, nullptr, 0, &d);
  if (rc) return rc;
  return prepare_common(d, batch, indices, offsets, num_indices, workspace, workspace_bytes,
                        d_status, kPoolPlain, nullptr, stream);
}

int embbag_backward_apply_sgd(const float* grad_pooled, int32_t batch, int64_t num_indices,
                              float lr, const embbag_tables_t* tables, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  return apply_common(d, false, grad_pooled, false, batch, num_indices, lr, workspace,
                      workspace_bytes, PoolArgs{}, stream);
}

int embbag_backward_apply_sgd_split_bf16(const float* grad_pooled, int32_t batch,
                                         int64_t num_indices, float lr,
                                         const embbag_split_tables_t* tables, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
  if (tables == nullptr || tables->lo == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->hi),
                     reinterpret_cast<void* const*>(tables->lo), 8, &d);
  if (rc) return rc;
  return apply_common(d, true, grad_pooled, false, batch, num_indices, lr, workspace,
                      workspace_bytes, PoolArgs{}, stream);
}

int embbag_forward_split_bf16_act(const embbag_split_tables_t* tables, int32_t batch,
                                  const int32_t* indices, const int32_t* offsets,
                                  int64_t num_indices, uint16_t* pooled_out, int32_t* d_status,
                                  hipStream_t stream) {
  TableDesc d;
  int rc = split_desc(tables, false, &d);
  if (rc) return rc;
  return forward_common(d, true, batch, indices, offsets, num_indices, pooled_out, true, d_status,
                        PoolArgs{}, stream);
}

int embbag_backward_sgd_split_bf16_act(const uint16_t* grad_pooled, int32_t batch,
                                       const int32_t* indices, const int32_t* offsets,
                                       int64_t num_indices, float lr,
                                       const embbag_split_tables_t* tables, void* workspace,
                                       size_t workspace_bytes, int32_t* d_status,
                                       hipStream_t stream) {
  TableDesc d;
  int rc = split_desc(tables, true, &d);
  if (rc) return rc;
  return backward_common(d, true, grad_pooled, true, batch, indices, offsets, num_indices, lr,
                         workspace, workspace_bytes, d_status, PoolArgs{}, stream);
}

int embbag_backward_apply_sgd_split_bf16_act(const uint16_t* grad_pooled, int32_t batch,
                                             int64_t num_indices, float lr,
                                             const embbag_split_tables_t* tables,
                                             void* workspace, size_t workspace_bytes,
                                             hipStream_t stream) {
  TableDesc d;
  int rc = split_desc(tables, true, &d);
  if (rc) return rc;
  return apply_common(d, true, grad_pooled, true, batch, num_indices, lr, workspace,
                      workspace_bytes, PoolArgs{}, stream);
}

int embbag_split_fp32(const float* w, uint16_t* hi, uint16_t* lo, int64_t n, hipStream_t stream) {
  if (n < 0 || (n > 0 && (w == nullptr || hi == nullptr || lo == nullptr)))
    return EMBBAG_ERR_INVALID_ARG;
  return hip_status(launch_split(w, hi, lo, n, stream));
}

int embbag_combine_fp32(const uint16_t* hi, const uint16_t* lo, float* w, int64_t n,
                        hipStream_t stream) {
  if (n < 0 || (n > 0 && (w == nullptr || hi == nullptr || lo == nullptr)))
    return EMBBAG_ERR_INVALID_ARG;
  return hip_status(launch_combine(hi, lo, w, n, stream));
}

size_t embbag_dedup_workspace_bytes(int32_t num_tables, int32_t batch, int64_t num_indices) {
  if (num_tables < 1 || num_tables > kMaxTables) return 0;
  if (batch < 0 || num_indices < 0 || num_indices > kMaxIndices) return 0;
  if (int64_t(num_tables) * batch + 1 > kInt32Max) return 0;
  return backward_layout(num_tables, batch, num_indices, 4, 0, true).total;
}

int embbag_dedup(int32_t num_tables, const int64_t* rows, int32_t batch, const int32_t* indices,
                 const int32_t* offsets, int64_t num_indices, uint32_t* sorted_keys,
                 uint32_t* sorted_bags, uint32_t* unique_keys, int32_t* seg_off,
                 int32_t* d_num_unique, void* workspace, size_t workspace_bytes,
                 int32_t* d_status, hipStream_t stream) {
  TableDesc d;
  int rc = make_desc(num_tables, 4, rows, nullptr, nullptr, 0, &d);
  if (rc) return rc;
  rc = check_bags(num_tables, batch, indices, offsets, num_indices);
  if (rc) return rc;
  if (seg_off == nullptr || d_num_unique == nullptr) return EMBBAG_ERR_INVALID_ARG;
  if (num_indices > 0 && (sorted_keys == nullptr || sorted_bags == nullptr || unique_keys == nullptr))
    return EMBBAG_ERR_INVALID_ARG;
  const BwdLayout L = backward_layout(num_tables, batch, num_indices, 4, d.rowbase[num_tables], true);
  if (workspace == nullptr || !aligned(workspace, kWsAlign) || workspace_bytes < L.total)
    return EMBBAG_ERR_WORKSPACE;
  char* w = static_cast<char*>(workspace);
  if (launch_sort(d, batch, indices, offsets, num_indices, L, w, d_status,
                  phase_token(num_tables, batch, num_indices, 4, d.rowbase[num_tables],
                              kPoolPlain),
                  nullptr, stream) != hipSuccess)
    return EMBBAG_ERR_HIP;
  return hip_status(launch_unique(sorted_buffer(L, w), L, w, sorted_keys, sorted_bags,
                                  unique_keys, seg_off, d_num_unique, stream));
}

int embbag_baseline_materialize(const float* grad_pooled, int32_t num_tables, int32_t batch,
                                int32_t dim, const int32_t* offsets, int64_t num_indices,
                                float* dW, int32_t* d_status, hipStream_t stream) {
  if (num_tables < 1 || num_tables > kMaxTables || dim < 4 || dim > 1024 || dim % 4 != 0)
    return EMBBAG_ERR_INVALID_ARG;
  int rc = check_bags(num_tables, batch, nullptr, offsets, 0);
  if (rc) return rc;
  if (num_indices < 0 || num_indices > kMaxIndices) return EMBBAG_ERR_INVALID_ARG;
  if (int64_t(num_tables) * batch > 0 && (grad_pooled == nullptr || !aligned(grad_pooled, 16)))
    return EMBBAG_ERR_INVALID_ARG;
  if (num_indices > 0 && (dW == nullptr || !aligned(dW, 16))) return EMBBAG_ERR_INVALID_ARG;
  return hip_status(
      launch_materialize(grad_pooled, offsets, num_indices, num_tables, batch, dim, dW, d_status,
                         stream));
}

static int baseline_update(const float* src, bool fused, int32_t batch, const int32_t* indices,
                           const int32_t* offsets, int64_t num_indices, float lr,
                           const embbag_tables_t* tables, int32_t* d_status, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  rc = check_bags(d.num_tables, batch, indices, offsets, num_indices);
  if (rc) return rc;
  if (num_indices > 0 && (src == nullptr || !aligned(src, 16))) return EMBBAG_ERR_INVALID_ARG;
  return hip_status(launch_atomic_update(d, src, fused, indices, offsets, num_indices, batch, lr,
                                         d_status, stream));
}

int embbag_baseline_update_atomic(const float* dW, int32_t batch, const int32_t* indices,
                                  const int32_t* offsets, int64_t num_indices, float lr,
                                  const embbag_tables_t* tables, int32_t* d_status,
                                  hipStream_t stream) {
  return baseline_update(dW, false, batch, indices, offsets, num_indices, lr, tables, d_status,
                         stream);
}

int embbag_baseline_backward_sgd_atomic(const float* grad_pooled, int32_t batch,
                                        const int32_t* indices, const int32_t* offsets,
                                        int64_t num_indices, float lr,
                                        const embbag_tables_t* tables, int32_t* d_status,
                                        hipStream_t stream) {
  return baseline_update(grad_pooled, true, batch, indices, offsets, num_indices, lr, tables,
                         d_status, stream);
}

int embbag_baseline_update_owner(const float* dW, int32_t batch, const int32_t* indices,
                                 const int32_t* offsets, int64_t num_indices, float lr,
                                 const embbag_tables_t* tables, int32_t owners,
                                 hipStream_t stream) {
  if (tables == nullptr || owners < 1 || owners > 65536) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  rc = check_bags(d.num_tables, batch, indices, offsets, num_indices);
  if (rc) return rc;
  if (num_indices > 0 && (dW == nullptr || !aligned(dW, 16))) return EMBBAG_ERR_INVALID_ARG;
  return hip_status(
      launch_owner_update(d, dW, indices, offsets, num_indices, batch, owners, lr, stream));
}

static int touch_common(const TableDesc& d, bool split, int32_t batch, int64_t num_indices,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (batch < 0 || num_indices < 0 || num_indices > kMaxIndices ||
      int64_t(d.num_tables) * batch + 1 > kInt32Max)
    return EMBBAG_ERR_INVALID_ARG;
  if (int64_t(d.num_tables) * batch == 0 && num_indices > 0) return EMBBAG_ERR_OFFSETS;
  const uint32_t total = d.rowbase[d.num_tables];
  const BwdLayout L = backward_layout(d.num_tables, batch, num_indices, d.dim, total, false);
  if (workspace == nullptr || !aligned(workspace, kWsAlign) || workspace_bytes < L.total)
    return EMBBAG_ERR_WORKSPACE;
  return hip_status(launch_touch_rows(d, split, batch, L, static_cast<char*>(workspace),
                                      phase_token(d.num_tables, batch, num_indices, d.dim,
                                                  total, kPoolPlain),
                                      stream));
}

int embbag_baseline_touch_rows(int32_t batch, int64_t num_indices, const embbag_tables_t* tables,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (tables == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->weights), nullptr, 16, &d);
  if (rc) return rc;
  return touch_common(d, false, batch, num_indices, workspace, workspace_bytes, stream);
}

int embbag_baseline_touch_rows_split(int32_t batch, int64_t num_indices,
                                     const embbag_split_tables_t* tables, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
  if (tables == nullptr || tables->lo == nullptr) return EMBBAG_ERR_INVALID_ARG;
  TableDesc d;
  int rc = make_desc(tables->num_tables, tables->dim, tables->rows,
                     reinterpret_cast<void* const*>(tables->hi),
                     reinterpret_cast<void* const*>(tables->lo), 8, &d);
  if (rc) return rc;
  return touch_common(d, true, batch, num_indices, workspace, workspace_bytes, stream);
}

int embbag_status_read(const int32_t* d_status, hipStream_t stream) {
  if (d_status == nullptr) return EMBBAG_ERR_INVALID_ARG;
  if (hipStreamSynchronize(stream) != hipSuccess) return EMBBAG_ERR_HIP;
  int32_t v = 0;
  if (hipMemcpy(&v, d_status, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess)
    return EMBBAG_ERR_HIP;
  return v;
}

}  // extern "C"
