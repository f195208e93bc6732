/*
 * embbag.h — C ABI of the MI355X (gfx950) EmbeddingBag training step.
 *
 * Operators (Kalamkar et al., "Optimizing Deep Learning Recommender Systems'
 * Training on CPU Cluster Architectures", arXiv 2005.04680):
 *   - forward: sum-pooled gather over many tables (Section III-A,
 *     Algorithm 1; Section II's L = A^T W over the bags of a minibatch);
 *   - backward fused with the sparse SGD update of only the touched rows
 *     (Algorithms 2 and 3, whose fusion the end of Section III-A describes;
 *     every row receives the sum of all its look-ups' gradients exactly once,
 *     the single-writer property of Algorithm 4, here without float atomics);
 *   - the Split-SGD-BF16 variants of both (Section VII).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tables.  T tables (1 <= T <= 64) of M_t rows (1 <= M_t, sum of M_t <=
 *   2^31 - 1) and dimension E (4 <= E <= 1024, E % 4 == 0).  An FP32 table is a
 *   row-major [M_t][E] device array, 16-byte aligned.  A split table is two
 *   row-major [M_t][E] uint16 device arrays, 8-byte aligned: `hi` holds the 16
 *   most significant bits of each FP32 weight (a BF16 number, by truncation)
 *   and `lo` the 16 least significant bits (Section VII stores them as two
 *   separate tensors).
 * Bags.  `batch` = B bags per table.  Bag k = t*B + b reads
 *   indices[offsets[k] .. offsets[k+1]) (half-open), rows of table t.
 *   `indices`: device int32 [num_indices], table-local rows; num_indices <=
 *   2^31 - 1 (indices and offsets are int32).
 *   `offsets`: device int32 [T*B + 1], offsets[0] == 0, non-decreasing,
 *   offsets[T*B] == num_indices.  (Algorithm 1's header swaps the two sizes;
 *   its loops read O[n] and O[n+1].)  A row may repeat within and across
 *   bags; repeats count with multiplicity.  An empty bag pools to +0.0.
 * Pooled data.  `pooled_out` and `grad_pooled`: device FP32 [T][B][E],
 *   contiguous, 16-byte aligned.
 * Streams.  Every call only enqueues work on `stream` (0 = the null stream)
 *   and returns; the caller keeps all buffers alive until that work is done.
 *   The only call that waits is embbag_status_read.
 * Ownership.  The caller owns every buffer.  Apart from the fixed device
 *   array of embbag_backward_sgd_noalloc (declared below), the library
 *   allocates no device memory, keeps no pointer after returning and holds no
 *   global state, so calls on distinct workspaces are thread-safe.  Tables are
 *   updated in place; `pooled_out` must not alias a table.
 * Errors.  Argument errors (null pointers, sizes out of range, a workspace
 *   that is too small or misaligned) are found on the host: the call returns
 *   the code and enqueues nothing.  Data errors (bad offsets, an index out of
 *   its table's range) are found on the device: the call returns EMBBAG_OK,
 *   and the device lowers `*d_status` to min(*d_status, code) (the caller
 *   zeroes it; EMBBAG_ERR_OFFSETS wins over EMBBAG_ERR_INDEX_RANGE).  After a
 *   data error the forward's output is unspecified and the backward writes no
 *   table row at all.  Launch failures return EMBBAG_ERR_HIP.
 */
#ifndef EMBBAG_H_
#define EMBBAG_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define EMBBAG_OK 0
#define EMBBAG_ERR_INVALID_ARG (-1) /* null pointer, T/E/B/sizes out of range */
#define EMBBAG_ERR_WORKSPACE (-2)   /* workspace smaller than required, or not 256-B aligned */
#define EMBBAG_ERR_INDEX_RANGE (-3) /* an index outside [0, M_t) (device-detected) */
#define EMBBAG_ERR_OFFSETS (-4)     /* offsets[0] != 0, decreasing, or offsets[T*B] != num_indices */
#define EMBBAG_ERR_HIP (-5)         /* a HIP launch or runtime call failed */

/* Static string naming a status code ("unknown status" otherwise). */
const char* embbag_status_string(int code);

/* FP32 tables.  `rows` and `weights` are HOST arrays of num_tables entries;
 * weights[t] is a device pointer to rows[t] x dim floats. */
typedef struct {
  int32_t num_tables;
  int32_t dim;
  const int64_t* rows;
  float* const* weights;
} embbag_tables_t;

/* Split-SGD-BF16 tables (Section VII): hi[t], lo[t] are device pointers to
 * rows[t] x dim uint16 each. */
typedef struct {
  int32_t num_tables;
  int32_t dim;
  const int64_t* rows;
  uint16_t* const* hi;
  uint16_t* const* lo;
} embbag_split_tables_t;

/* Forward, Algorithm 1 (sum pooling): for every bag k = t*B + b,
 *   pooled_out[t][b][:] = sum over s in [offsets[k], offsets[k+1]) of
 *                         weights[t][indices[s]][:]        (+0.0 if empty).
 * Each bag is summed in FP64 in look-up order and rounded once to FP32.
 * `d_status` (device int32, nullable) receives data errors as described in
 * the header comment. */
int embbag_forward(const embbag_tables_t* tables, int32_t batch, const int32_t* indices,
                   const int32_t* offsets, int64_t num_indices, float* pooled_out,
                   int32_t* d_status, hipStream_t stream);

/* Bytes of device workspace the backward (FP32 or split) needs for these
 * sizes; 0 for invalid sizes.  The workspace must be 256-byte aligned. */
size_t embbag_backward_workspace_bytes(int32_t num_tables, int32_t batch, int64_t num_indices,
                                       int32_t dim);

/* Fused backward + sparse SGD, Algorithms 2-3 with alpha = -lr:
 * for every (table t, row r) named by at least one look-up,
 *   weights[t][r][:] -= lr * sum over look-ups s with indices[s] == r in a
 *                       bag k of table t of grad_pooled[k][:],
 * each touched row read and written exactly once (no float atomics; the
 * gradient sum is accumulated in FP64 and rounded once).  Rows no look-up
 * names are not written.  `workspace` (device, >= embbag_backward_workspace_bytes)
 * is scratch owned by the caller.  `d_status` is nullable. */
int embbag_backward_sgd(const float* grad_pooled, int32_t batch, const int32_t* indices,
                        const int32_t* offsets, int64_t num_indices, float lr,
                        const embbag_tables_t* tables, void* workspace, size_t workspace_bytes,
                        int32_t* d_status, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation as embbag_backward_sgd, with the same arguments but no workspace,
 * and the same kernels.  Its workspace is a fixed device array of
 * EMBBAG_NOALLOC_SCRATCH_BYTES (64 MiB) inside the library, which each GPU it
 * runs on holds from its first call until the process ends; the call itself
 * allocates nothing.  A step whose workspace (embbag_backward_workspace_bytes)
 * exceeds the array is refused with EMBBAG_ERR_WORKSPACE and enqueues nothing
 * (64 MiB holds 8 tables x 2048 bags x 32 look-ups at E = 64, 30.5 MiB, or
 * 819,200 look-ups at E = 64, 47.7 MiB).  Argument errors are those of
 * embbag_backward_sgd.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (other streams, other threads) race; calls ordered
 * on one stream are safe.  EMBBAG_ERR_HIP if the array's device address
 * cannot be obtained. */
#define EMBBAG_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int embbag_backward_sgd_noalloc(const float* grad_pooled, int32_t batch, const int32_t* indices,
                                const int32_t* offsets, int64_t num_indices, float lr,
                                const embbag_tables_t* tables, int32_t* d_status,
                                hipStream_t stream);

/* Pooling modes of the *_pooled entry points (Section II: L = A^T W, where
 * column n of A holds a weight a_p for every row bag n reads). */
#define EMBBAG_POOL_SUM 0  /* Y[k] = sum over s of a_s * W[I[s]] (a_s = 1 without weights) */
#define EMBBAG_POOL_MEAN 1 /* Y[k] = (sum over s of W[I[s]]) / |bag k|; empty bag -> +0.0 */

/* Forward with per-look-up weights or mean pooling.  `per_sample_weights` is
 * a device FP32 array [num_indices] (one weight per look-up, nullable; only
 * with EMBBAG_POOL_SUM).  With null weights and EMBBAG_POOL_SUM this is
 * embbag_forward.  An invalid (weights, pooling) pair is EMBBAG_ERR_INVALID_ARG. */
int embbag_forward_pooled(const embbag_tables_t* tables, int32_t batch, const int32_t* indices,
                          const int32_t* offsets, int64_t num_indices,
                          const float* per_sample_weights, int32_t pooling, float* pooled_out,
                          int32_t* d_status, hipStream_t stream);

/* The matching fused backward + SGD: every touched row r of table t gets
 *   W[r] -= lr * sum over its look-ups s of c_s * grad_pooled[bag(s)],
 * c_s = a_s (weighted sum), 1 (sum) or 1/|bag(s)| (mean), once per row, the
 * sum in FP64.  Same workspace as embbag_backward_sgd. */
int embbag_backward_sgd_pooled(const float* grad_pooled, int32_t batch, const int32_t* indices,
                               const int32_t* offsets, int64_t num_indices,
                               const float* per_sample_weights, int32_t pooling, float lr,
                               const embbag_tables_t* tables, void* workspace,
                               size_t workspace_bytes, int32_t* d_status, hipStream_t stream);

/* The same in two phases, like embbag_backward_prepare / _apply_sgd.  Phase 1
 * sorts the weights, if given, along with the look-ups into the workspace
 * (mean pooling needs nothing more than a plain phase 1); phase 2 must get the
 * same (weights, pooling) pair, the same offsets (mean pooling reads the bag
 * sizes from them) and the same sizes.  A workspace prepared with weights and
 * applied without (or the reverse), or prepared for other sizes, makes the
 * apply write nothing. */
int embbag_backward_prepare_pooled(int32_t num_tables, const int64_t* rows, int32_t dim,
                                   int32_t batch, const int32_t* indices, const int32_t* offsets,
                                   int64_t num_indices, const float* per_sample_weights,
                                   int32_t pooling, void* workspace, size_t workspace_bytes,
                                   int32_t* d_status, hipStream_t stream);
int embbag_backward_apply_sgd_pooled(const float* grad_pooled, int32_t batch,
                                     const int32_t* offsets, int64_t num_indices,
                                     const float* per_sample_weights, int32_t pooling, float lr,
                                     const embbag_tables_t* tables, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/* The fused backward in two phases, for callers that overlap its integer
 * work with other parts of a training step.  embbag_backward_sgd(...) is
 * exactly embbag_backward_prepare(...) followed by embbag_backward_apply_sgd(...).
 *
 * Phase 1 (Algorithms 2-4's index work): builds the row key of every look-up,
 * validates offsets and indices, and stably sorts the look-ups by key into
 * `workspace`.  It reads no gradient, so it may be enqueued as soon as the
 * batch's indices and offsets exist.  `rows` is a HOST array of num_tables
 * row counts; `dim` sizes the workspace (embbag_backward_workspace_bytes).
 * `d_status` (nullable) receives data errors as in the header comment. */
int embbag_backward_prepare(int32_t num_tables, const int64_t* rows, int32_t dim, int32_t batch,
                            const int32_t* indices, const int32_t* offsets, int64_t num_indices,
                            void* workspace, size_t workspace_bytes, int32_t* d_status,
                            hipStream_t stream);

/* Phase 2: gathers grad_pooled rows per sorted look-up, sums each row's
 * gradient in FP64 and applies W -= lr * G once per touched row.  The
 * workspace must hold a phase-1 result for the same batch, num_indices and
 * table row counts, ordered before this call (same stream, or an event).  If
 * phase 1 found a data error, or the workspace does not carry a phase-1
 * result for these sizes, no table row is written.  The same phase-1 result
 * may be applied more than once (e.g. to several gradients). */
int embbag_backward_apply_sgd(const float* grad_pooled, int32_t batch, int64_t num_indices,
                              float lr, const embbag_tables_t* tables, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Phase 2 for split tables (Section VII update, as embbag_backward_sgd_split_bf16). */
int embbag_backward_apply_sgd_split_bf16(const float* grad_pooled, int32_t batch,
                                         int64_t num_indices, float lr,
                                         const embbag_split_tables_t* tables, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream);

/* Forward of Section VII: Algorithm 1 reading only the BF16 high halves
 * (each value is hi << 16 as FP32); the low halves are not read. */
int embbag_forward_split_bf16(const embbag_split_tables_t* tables, int32_t batch,
                              const int32_t* indices, const int32_t* offsets,
                              int64_t num_indices, float* pooled_out, int32_t* d_status,
                              hipStream_t stream);

/* Update of Section VII: for every touched row, recombine hi/lo into the FP32
 * weight, apply the same update as embbag_backward_sgd in FP32, and split the
 * result back into hi/lo.  Untouched rows keep both halves. */
int embbag_backward_sgd_split_bf16(const float* grad_pooled, int32_t batch,
                                   const int32_t* indices, const int32_t* offsets,
                                   int64_t num_indices, float lr,
                                   const embbag_split_tables_t* tables, void* workspace,
                                   size_t workspace_bytes, int32_t* d_status,
                                   hipStream_t stream);

/* BF16 activations (Section VII trains with BF16 activations and gradients
 * and keeps the FP32 weight only for the update).  Same operations as the
 * split entry points above, with the pooled output and its gradient stored as
 * BF16 bit patterns, [T][B][E] uint16, 8-byte aligned:
 *   - forward: each pooled value is the FP32 sum of the bag's high halves
 *     (as embbag_forward_split_bf16), rounded to the nearest BF16, ties to
 *     even; an empty bag gives +0;
 *   - backward: each gradient value is widened exactly (g << 16 as FP32) and
 *     the update is that of embbag_backward_sgd_split_bf16.
 * Errors, workspace and phases as for the FP32-activation entry points. */
int embbag_forward_split_bf16_act(const embbag_split_tables_t* tables, int32_t batch,
                                  const int32_t* indices, const int32_t* offsets,
                                  int64_t num_indices, uint16_t* pooled_out, int32_t* d_status,
                                  hipStream_t stream);
int embbag_backward_sgd_split_bf16_act(const uint16_t* grad_pooled, int32_t batch,
                                       const int32_t* indices, const int32_t* offsets,
                                       int64_t num_indices, float lr,
                                       const embbag_split_tables_t* tables, void* workspace,
                                       size_t workspace_bytes, int32_t* d_status,
                                       hipStream_t stream);
int embbag_backward_apply_sgd_split_bf16_act(const uint16_t* grad_pooled, int32_t batch,
                                             int64_t num_indices, float lr,
                                             const embbag_split_tables_t* tables,
                                             void* workspace, size_t workspace_bytes,
                                             hipStream_t stream);

/* Section VII storage helpers (device, elementwise over n values):
 * hi[i] = bits(w[i]) >> 16, lo[i] = bits(w[i]) & 0xFFFF, and the inverse
 * w[i] = from_bits(hi[i] << 16 | lo[i]).  Lossless in both directions. */
int embbag_split_fp32(const float* w, uint16_t* hi, uint16_t* lo, int64_t n, hipStream_t stream);
int embbag_combine_fp32(const uint16_t* hi, const uint16_t* lo, float* w, int64_t n,
                        hipStream_t stream);

/* Bytes of device workspace embbag_dedup needs (256-byte aligned). */
size_t embbag_dedup_workspace_bytes(int32_t num_tables, int32_t batch, int64_t num_indices);

/* Integer work of the backward, exposed for bit-exact checking.  Algorithm 2's
 * loop over bags n and look-ups s gives every look-up its bag; the look-ups
 * grouped by row are what Algorithm 3 needs to add all of a row's gradients
 * and Algorithm 4 to give each row a single writer (Section III-A):
 *   key[s] = rowbase[t] + indices[s] (rowbase = exclusive prefix sum of rows),
 *   bag[s] = k for offsets[k] <= s < offsets[k+1];
 *   (sorted_keys, sorted_bags)[NS] = (key, bag) stably sorted by key (ties in
 *     increasing s);
 *   unique_keys[U] = the distinct keys, increasing; seg_off[U+1] = first sorted
 *     position of each, seg_off[U] = NS; *d_num_unique = U.
 * All outputs are device arrays sized for the worst case (U = NS):
 * sorted_keys, sorted_bags, unique_keys [NS] uint32, seg_off [NS+1] int32,
 * d_num_unique one int32.  `rows` is a HOST array of num_tables entries. */
int embbag_dedup(int32_t num_tables, const int64_t* rows, int32_t batch, const int32_t* indices,
                 const int32_t* offsets, int64_t num_indices, uint32_t* sorted_keys,
                 uint32_t* sorted_bags, uint32_t* unique_keys, int32_t* seg_off,
                 int32_t* d_num_unique, void* workspace, size_t workspace_bytes,
                 int32_t* d_status, hipStream_t stream);

/* ---- Baselines: the paper's unfused update designs on the GPU -------------
 * For measurement against the fused backward; not needed to train.  The
 * atomic variants add in a scheduling-dependent FP32 order (results vary in
 * the last bits between runs); the owner variant is deterministic.  Indices
 * out of range are skipped (and reported through the nullable d_status);
 * offsets must be valid. */

/* Algorithm 2: dW[s][:] = grad_pooled[bag(s)][:], dW a device FP32 array
 * [num_indices][dim] (NS x E: 13.4 GB at 13.1M look-ups of E = 256). */
int embbag_baseline_materialize(const float* grad_pooled, int32_t num_tables, int32_t batch,
                                int32_t dim, const int32_t* offsets, int64_t num_indices,
                                float* dW, int32_t* d_status, hipStream_t stream);

/* Algorithm 3 with hardware FP32 atomics: W_t[I[s]][:] += (-lr) * dW[s][:]. */
int embbag_baseline_update_atomic(const float* dW, int32_t batch, const int32_t* indices,
                                  const int32_t* offsets, int64_t num_indices, float lr,
                                  const embbag_tables_t* tables, int32_t* d_status,
                                  hipStream_t stream);

/* Algorithms 2+3 fused with atomics: W_t[I[s]][:] += (-lr) * grad_pooled[bag(s)][:]. */
int embbag_baseline_backward_sgd_atomic(const float* grad_pooled, int32_t batch,
                                        const int32_t* indices, const int32_t* offsets,
                                        int64_t num_indices, float lr,
                                        const embbag_tables_t* tables, int32_t* d_status,
                                        hipStream_t stream);

/* Algorithm 4, race-free by row ownership: `owners` wavefronts each own an
 * equal range of the global row space (tables concatenated), scan all
 * look-ups and apply W[row] += (-lr) * dW[s] for their own rows in increasing
 * s, in FP32 (the order and precision of a sequential loop over s). */
int embbag_baseline_update_owner(const float* dW, int32_t batch, const int32_t* indices,
                                 const int32_t* offsets, int64_t num_indices, float lr,
                                 const embbag_tables_t* tables, int32_t owners,
                                 hipStream_t stream);

/* The floor of the update, for measurement: every row that the workspace
 * prepared by embbag_backward_prepare (same batch, num_indices and tables,
 * no weights) touches is read and written back unchanged, once: the memory
 * traffic of the single-writer update of Algorithm 4 with nothing summed.
 * Its time bounds embbag_backward_apply_sgd on the same rows from below.
 * Tables are left bit-identical.  A workspace that holds no sort result for
 * these sizes (or a data error) makes it write nothing.  Argument errors as
 * embbag_backward_apply_sgd. */
int embbag_baseline_touch_rows(int32_t batch, int64_t num_indices, const embbag_tables_t* tables,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The same floor for split tables (Section VII storage): each touched row's
 * BF16 high half and 16-bit low half are read and written back unchanged,
 * once, as embbag_backward_apply_sgd_split_bf16 moves them.  `tables->lo`
 * must be given; halves 8-byte aligned.  Workspace, errors and the
 * bit-identical result as embbag_baseline_touch_rows. */
int embbag_baseline_touch_rows_split(int32_t batch, int64_t num_indices,
                                     const embbag_split_tables_t* tables, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/* Waits for `stream` and returns the device status word (*d_status), or
 * EMBBAG_ERR_HIP if the wait or copy fails. */
int embbag_status_read(const int32_t* d_status, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* EMBBAG_H_ */
