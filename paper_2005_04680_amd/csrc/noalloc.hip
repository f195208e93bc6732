// The fused backward + SGD without a caller workspace, for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc).
//
// The workspace is a fixed array in device memory, `scratch`, that each GPU
// the library runs on holds until the process ends.  In host code the name
// `scratch` is only a stand-in for the symbol: its device address is looked
// up with hipGetSymbolAddress once per device (with that device current) and
// only that address is ever handed to kernels.  Every call on one GPU uses
// that GPU's one array, so calls that overlap on one GPU (several streams or
// threads) race; calls in one stream order are safe.  Nothing in the array
// has to start at zero: the sort phase writes every word the update reads.
//
// This file holds no kernel, so the array's code object is loaded (and the
// array placed on a GPU) only when this entry point first runs there.
#include <mutex>

#include "common.hpp"

namespace {

constexpr size_t kScratchBytes = EMBBAG_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch`, per device

// Device address of `scratch` on the device that `stream` belongs to.
int scratch_address(hipStream_t stream, void** out) {
  int dev = -1;
  if (stream != nullptr) {
    if (hipStreamGetDevice(stream, &dev) != hipSuccess) return EMBBAG_ERR_HIP;
  } else if (hipGetDevice(&dev) != hipSuccess) {
    return EMBBAG_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return EMBBAG_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return EMBBAG_ERR_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return EMBBAG_ERR_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return EMBBAG_ERR_HIP;
    if (e != hipSuccess || p == nullptr) return EMBBAG_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return EMBBAG_OK;
}

}  // namespace

extern "C" int embbag_backward_sgd_noalloc(const float* grad_pooled, int32_t batch,
                                           const int32_t* indices, const int32_t* offsets,
                                           int64_t num_indices, float lr,
                                           const embbag_tables_t* tables, int32_t* d_status,
                                           hipStream_t stream) {
  // Argument errors first, with the codes embbag_backward_sgd gives: it checks
  // every argument before the workspace and enqueues nothing when a check
  // fails, so without a workspace it fails on the workspace exactly when the
  // arguments are valid.
  int rc = embbag_backward_sgd(grad_pooled, batch, indices, offsets, num_indices, lr, tables,
                               nullptr, 0, d_status, stream);
  if (rc != EMBBAG_ERR_WORKSPACE) return rc;
  // Valid arguments: the step's workspace must fit the array.
  if (embbag_backward_workspace_bytes(tables->num_tables, batch, num_indices, tables->dim) >
      kScratchBytes)
    return EMBBAG_ERR_WORKSPACE;
  void* ws = nullptr;
  rc = scratch_address(stream, &ws);
  if (rc != EMBBAG_OK) return rc;
  return embbag_backward_sgd(grad_pooled, batch, indices, offsets, num_indices, lr, tables, ws,
                             kScratchBytes, d_status, stream);
}
