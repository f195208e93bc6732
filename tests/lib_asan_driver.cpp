// Drives the host side of libembbag (its C ABI's argument checks and the
// workspace layout arithmetic) with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code.  Every call below fails an
// argument check, so nothing is enqueued and no pointer is dereferenced: the
// device pointers are dummies.  The workspace sizes are computed over a grid
// of sizes up to the library's limits (2^31 - 1 look-ups, 64 tables,
// E = 1024), where an overflow in the layout arithmetic would be undefined
// behaviour.  Exits 0 unless a sanitizer stops it or a call returns another
// status than its arguments call for.
//
// Built with the library sources by tests/test_lib_sanitizers.py, which runs
// it only where no GPU is visible.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "embbag.h"

namespace {

int failures = 0;

void expect(int got, int want, const char* what) {
  if (got != want) {
    std::fprintf(stderr, "%s: status %d, expected %d\n", what, got, want);
    ++failures;
  }
}

// Dummy device addresses: 256-byte aligned (or deliberately not), never read.
template <class T>
T* dev(uintptr_t k, uintptr_t misalign = 0) {
  return reinterpret_cast<T*>((uintptr_t(1) << 32) + k * 4096 + misalign);
}

}  // namespace

int main() {
  constexpr int kInv = EMBBAG_ERR_INVALID_ARG, kWs = EMBBAG_ERR_WORKSPACE,
                kOff = EMBBAG_ERR_OFFSETS;
  hipStream_t st = nullptr;

  // Workspace sizes over a grid, including every limit.
  const int32_t Ts[] = {-1, 0, 1, 2, 16, 26, 64, 65};
  const int32_t Bs[] = {-1, 0, 1, 31, 2048, 8192, 65536, 1 << 24, 33554431, 2147483647};
  const int64_t NSs[] = {-1, 0, 1, 4095, 4097, 524288, 13107200, 1703936,
                         int64_t(2147483647) - 65536, int64_t(2147483647) - 1,
                         int64_t(2147483647), int64_t(2147483648), int64_t(1) << 40};
  const int32_t Es[] = {0, 4, 6, 16, 64, 128, 256, 512, 1020, 1024, 1028};
  size_t sink = 0;
  for (int32_t T : Ts)
    for (int32_t B : Bs)
      for (int64_t NS : NSs) {
        const size_t dd = embbag_dedup_workspace_bytes(T, B, NS);
        const bool valid = T >= 1 && T <= 64 && B >= 0 && NS >= 0 &&
                           NS <= int64_t(2147483647) &&
                           int64_t(T) * B + 1 <= 2147483647;
        if (!valid && dd != 0) expect(int(dd != 0), 0, "dedup workspace for invalid sizes");
        if (valid && dd == 0) expect(0, 1, "dedup workspace for valid sizes");
        for (int32_t E : Es) {
          const size_t b = embbag_backward_workspace_bytes(T, B, NS, E);
          const bool ok = valid && E >= 4 && E <= 1024 && E % 4 == 0;
          if (ok != (b != 0)) expect(int(b != 0), int(ok), "backward workspace");
          if (ok && b < size_t(NS) * 16) expect(0, 1, "backward workspace below the key buffers");
          sink += b + dd;
        }
      }
  for (int c = -7; c <= 1; ++c) sink += std::strlen(embbag_status_string(c));

  // Argument errors of every entry point.
  int64_t rows[3] = {100, 200, 300};
  float* w[3] = {dev<float>(1), dev<float>(2), dev<float>(3)};
  float* wmis[3] = {dev<float>(1), dev<float>(2, 4), dev<float>(3)};
  uint16_t* hi[3] = {dev<uint16_t>(4), dev<uint16_t>(5), dev<uint16_t>(6)};
  uint16_t* lo[3] = {dev<uint16_t>(7), dev<uint16_t>(8), dev<uint16_t>(9)};
  embbag_tables_t tb{3, 16, rows, w};
  embbag_split_tables_t sp{3, 16, rows, hi, lo};
  embbag_split_tables_t sp_nolo{3, 16, rows, hi, nullptr};
  const int32_t* I = dev<const int32_t>(10);
  const int32_t* O = dev<const int32_t>(11);
  float* Y = dev<float>(12);
  const float* G = dev<const float>(13);
  void* ws = dev<void>(20);
  const size_t wsb = embbag_backward_workspace_bytes(3, 8, 64, 16);
  int32_t* stt = dev<int32_t>(14);

  expect(embbag_forward(nullptr, 8, I, O, 64, Y, stt, st), kInv, "forward: no tables");
  for (int32_t T : {0, 65}) {
    embbag_tables_t t2{T, 16, rows, w};
    expect(embbag_forward(&t2, 8, I, O, 64, Y, stt, st), kInv, "forward: table count");
  }
  for (int32_t E : {0, 2, 6, 1028}) {
    embbag_tables_t t2{3, E, rows, w};
    expect(embbag_forward(&t2, 8, I, O, 64, Y, stt, st), kInv, "forward: dim");
  }
  {
    embbag_tables_t t2{3, 16, nullptr, w};
    expect(embbag_forward(&t2, 8, I, O, 64, Y, stt, st), kInv, "forward: no rows");
    int64_t r0[3] = {100, 0, 300};
    embbag_tables_t t3{3, 16, r0, w};
    expect(embbag_forward(&t3, 8, I, O, 64, Y, stt, st), kInv, "forward: empty table");
    int64_t rbig[3] = {2000000000, 2000000000, 5};
    embbag_tables_t t4{3, 16, rbig, w};
    expect(embbag_forward(&t4, 8, I, O, 64, Y, stt, st), kInv, "forward: rows over 2^31");
    embbag_tables_t t5{3, 16, rows, wmis};
    expect(embbag_forward(&t5, 8, I, O, 64, Y, stt, st), kInv, "forward: misaligned table");
    embbag_tables_t t6{3, 16, rows, nullptr};
    expect(embbag_forward(&t6, 8, I, O, 64, Y, stt, st), kInv, "forward: no table pointers");
  }
  expect(embbag_forward(&tb, -1, I, O, 64, Y, stt, st), kInv, "forward: batch < 0");
  expect(embbag_forward(&tb, 8, I, O, -1, Y, stt, st), kInv, "forward: NS < 0");
  expect(embbag_forward(&tb, 8, I, O, int64_t(2147483648), Y, stt, st), kInv,
         "forward: NS over the limit");
  expect(embbag_forward(&tb, 715827883, I, O, 64, Y, stt, st), kInv, "forward: T*B+1 over 2^31");
  expect(embbag_forward(&tb, 8, I, nullptr, 64, Y, stt, st), kInv, "forward: no offsets");
  expect(embbag_forward(&tb, 8, nullptr, O, 64, Y, stt, st), kInv, "forward: no indices");
  expect(embbag_forward(&tb, 8, I, O, 64, nullptr, stt, st), kInv, "forward: no output");
  expect(embbag_forward(&tb, 8, I, O, 64, dev<float>(12, 4), stt, st), kInv,
         "forward: misaligned output");
  expect(embbag_forward(&tb, 0, I, O, 64, Y, stt, st), kOff, "forward: look-ups, no bags");
  expect(embbag_forward_pooled(&tb, 8, I, O, 64, G, EMBBAG_POOL_MEAN, Y, stt, st), kInv,
         "forward: mean with weights");
  expect(embbag_forward_pooled(&tb, 8, I, O, 64, nullptr, 7, Y, stt, st), kInv,
         "forward: pooling mode");
  expect(embbag_forward_split_bf16(nullptr, 8, I, O, 64, Y, stt, st), kInv, "split forward");
  expect(embbag_forward_split_bf16_act(&sp, 8, I, O, 64, nullptr, stt, st), kInv,
         "split forward: no BF16 output");

  expect(embbag_backward_sgd(G, 8, I, O, 64, 0.1f, &tb, nullptr, wsb, stt, st), kWs,
         "backward: no workspace");
  expect(embbag_backward_sgd(G, 8, I, O, 64, 0.1f, &tb, dev<void>(20, 64), wsb, stt, st), kWs,
         "backward: misaligned workspace");
  expect(embbag_backward_sgd(G, 8, I, O, 64, 0.1f, &tb, ws, wsb - 1, stt, st), kWs,
         "backward: workspace too small");
  expect(embbag_backward_sgd(nullptr, 8, I, O, 64, 0.1f, &tb, ws, wsb, stt, st), kInv,
         "backward: no gradient");
  expect(embbag_backward_sgd(dev<const float>(13, 4), 8, I, O, 64, 0.1f, &tb, ws, wsb, stt, st),
         kInv, "backward: misaligned gradient");
  expect(embbag_backward_sgd(G, -1, I, O, 64, 0.1f, &tb, ws, wsb, stt, st), kInv,
         "backward: batch < 0");
  expect(embbag_backward_sgd_pooled(G, 8, I, O, 64, nullptr, 9, 0.1f, &tb, ws, wsb, stt, st),
         kInv, "backward: pooling mode");
  // the no-allocation backward reports argument errors before it looks up
  // its scratch array, and refuses a step larger than the array
  expect(embbag_backward_sgd_noalloc(G, 8, I, O, 64, 0.1f, nullptr, stt, st), kInv,
         "no-allocation backward: no tables");
  expect(embbag_backward_sgd_noalloc(nullptr, 8, I, O, 64, 0.1f, &tb, stt, st), kInv,
         "no-allocation backward: no gradient");
  expect(embbag_backward_sgd_noalloc(G, 8, I, O, int64_t(2147483648), 0.1f, &tb, stt, st), kInv,
         "no-allocation backward: NS over the limit");
  expect(embbag_backward_sgd_noalloc(G, 8, I, nullptr, 64, 0.1f, &tb, stt, st), kInv,
         "no-allocation backward: no offsets");
  expect(embbag_backward_sgd_noalloc(G, 8, I, O, int64_t(1) << 30, 0.1f, &tb, stt, st), kWs,
         "no-allocation backward: step past the scratch array");
  expect(embbag_backward_prepare(0, rows, 16, 8, I, O, 64, ws, wsb, stt, st), kInv,
         "prepare: table count");
  expect(embbag_backward_prepare(3, rows, 16, 8, I, nullptr, 64, ws, wsb, stt, st), kInv,
         "prepare: no offsets");
  expect(embbag_backward_prepare(3, rows, 16, 8, I, O, 64, ws, 16, stt, st), kWs,
         "prepare: workspace too small");
  expect(embbag_backward_prepare_pooled(3, rows, 16, 8, I, O, 64, G, EMBBAG_POOL_MEAN, ws, wsb,
                                        stt, st),
         kInv, "prepare: mean with weights");
  expect(embbag_backward_apply_sgd(nullptr, 8, 64, 0.1f, &tb, ws, wsb, st), kInv,
         "apply: no gradient");
  expect(embbag_backward_apply_sgd(G, 8, 64, 0.1f, &tb, ws, 0, st), kWs, "apply: no workspace");
  expect(embbag_backward_apply_sgd_pooled(G, 8, O, 64, nullptr, 5, 0.1f, &tb, ws, wsb, st), kInv,
         "apply: pooling mode");
  expect(embbag_backward_apply_sgd_split_bf16(G, 8, 64, 0.1f, &sp_nolo, ws, wsb, st), kInv,
         "split apply: no lo halves");
  expect(embbag_backward_sgd_split_bf16(G, 8, I, O, 64, 0.1f, &sp_nolo, ws, wsb, stt, st), kInv,
         "split backward: no lo halves");
  expect(embbag_backward_sgd_split_bf16_act(dev<const uint16_t>(13, 2), 8, I, O, 64, 0.1f, &sp,
                                            ws, wsb, stt, st),
         kInv, "split backward: misaligned BF16 gradient");
  expect(embbag_backward_apply_sgd_split_bf16_act(nullptr, 8, 64, 0.1f, &sp, ws, wsb, st), kInv,
         "split apply: no BF16 gradient");
  expect(embbag_split_fp32(nullptr, hi[0], lo[0], 16, st), kInv, "split: no input");
  expect(embbag_split_fp32(G, hi[0], lo[0], -1, st), kInv, "split: n < 0");
  expect(embbag_combine_fp32(hi[0], nullptr, Y, 16, st), kInv, "combine: no lo");
  const size_t dwb = embbag_dedup_workspace_bytes(3, 8, 64);
  expect(embbag_dedup(3, rows, 8, I, O, 64, dev<uint32_t>(30), dev<uint32_t>(31),
                      dev<uint32_t>(32), nullptr, dev<int32_t>(33), ws, dwb, stt, st),
         kInv, "dedup: no segment offsets");
  expect(embbag_dedup(3, rows, 8, I, O, 64, nullptr, dev<uint32_t>(31), dev<uint32_t>(32),
                      dev<int32_t>(34), dev<int32_t>(33), ws, dwb, stt, st),
         kInv, "dedup: no sorted keys");
  expect(embbag_baseline_touch_rows(-1, 64, &tb, ws, wsb, st), kInv, "touch rows: batch < 0");
  expect(embbag_baseline_touch_rows(8, 64, &tb, ws, 8, st), kWs, "touch rows: workspace");
  expect(embbag_baseline_touch_rows_split(8, 64, &sp_nolo, ws, wsb, st), kInv,
         "split touch rows: no lo");
  expect(embbag_baseline_touch_rows_split(-1, 64, &sp, ws, wsb, st), kInv,
         "split touch rows: batch < 0");
  expect(embbag_baseline_touch_rows_split(8, 64, &sp, ws, 8, st), kWs,
         "split touch rows: workspace");
  expect(embbag_baseline_touch_rows_split(8, 64, nullptr, ws, wsb, st), kInv,
         "split touch rows: no tables");
  expect(embbag_baseline_update_owner(G, 8, I, O, 64, 0.1f, &tb, 0, st), kInv,
         "owner update: no owners");
  expect(embbag_baseline_materialize(G, 3, 8, 16, O, 64, nullptr, stt, st), kInv,
         "materialize: no output");
  expect(embbag_status_read(nullptr, st), kInv, "status read: no word");

  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("library host driver: all cases ran clean (%zu)\n", sink);
  return 0;
}
