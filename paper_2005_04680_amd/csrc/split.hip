// Split-SGD-BF16 storage helpers (Section VII): an FP32 array <-> its 16 most
// significant bits (a BF16 number, by truncation) and 16 least significant
// bits, kept as two separate arrays.  Both directions are lossless.
#include "common.hpp"

namespace embbag {
namespace {

__global__ __launch_bounds__(kBlock) void split_kernel(const float* __restrict__ w,
                                                       uint16_t* __restrict__ hi,
                                                       uint16_t* __restrict__ lo, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * kBlock;
  for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride) {
    const uint32_t u = __float_as_uint(w[i]);
    hi[i] = uint16_t(u >> 16);
    lo[i] = uint16_t(u & 0xFFFFu);
  }
}

__global__ __launch_bounds__(kBlock) void combine_kernel(const uint16_t* __restrict__ hi,
                                                         const uint16_t* __restrict__ lo,
                                                         float* __restrict__ w, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * kBlock;
  for (int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride)
    w[i] = __uint_as_float((uint32_t(hi[i]) << 16) | uint32_t(lo[i]));
}

unsigned grid_for(int64_t n) {
  const int64_t b = (n + kBlock - 1) / kBlock;
  return unsigned(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

}  // namespace

hipError_t launch_split(const float* w, uint16_t* hi, uint16_t* lo, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(split_kernel, dim3(grid_for(n)), dim3(kBlock), 0, st, w, hi, lo, n);
  return hipGetLastError();
}

hipError_t launch_combine(const uint16_t* hi, const uint16_t* lo, float* w, int64_t n,
                          hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(grid_for(n)), dim3(kBlock), 0, st, hi, lo, w, n);
  return hipGetLastError();
}

}  // namespace embbag
