// Helpers for ranks above the edge kernels' 256: the layer is linear in each
// rank component (the CP sum over r, Sec. 3.1 eq. cp), so a rank-R problem is
// the sum of problems over disjoint column ranges of the factors and radial
// weights.  These kernels cut a column range out of a row-major [rows, R]
// matrix, put a [rows, n] block back into columns r0 .. r0+n-1, and add one
// float array into another (the chunks' partial results, in chunk order).
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

__global__ __launch_bounds__(256) void k_slice_cols(int rows, int R, int r0, int n, const float* __restrict__ src,
                                                    float* __restrict__ dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * n) return;
  const int row = i / n, j = i - row * n;
  dst[i] = src[size_t(row) * R + r0 + j];
}

__global__ __launch_bounds__(256) void k_scatter_cols(int rows, int R, int r0, int n, const float* __restrict__ src,
                                                      float* __restrict__ dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * n) return;
  const int row = i / n, j = i - row * n;
  dst[size_t(row) * R + r0 + j] = src[i];
}

__global__ __launch_bounds__(256) void k_accumulate(size_t n, const float* __restrict__ src, float* __restrict__ dst) {
  const size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) dst[i] += src[i];
}

}  // namespace

hipError_t launch_slice_cols(int rows, int R, int r0, int n, const float* src, float* dst, hipStream_t s) {
  if (rows < 0 || n < 0 || r0 < 0 || r0 + n > R) return hipErrorInvalidValue;
  const int total = rows * n;
  if (total == 0) return hipSuccess;
  k_slice_cols<<<dim3((total + 255) / 256), dim3(256), 0, s>>>(rows, R, r0, n, src, dst);
  return hipGetLastError();
}

hipError_t launch_scatter_cols(int rows, int R, int r0, int n, const float* src, float* dst, hipStream_t s) {
  if (rows < 0 || n < 0 || r0 < 0 || r0 + n > R) return hipErrorInvalidValue;
  const int total = rows * n;
  if (total == 0) return hipSuccess;
  k_scatter_cols<<<dim3((total + 255) / 256), dim3(256), 0, s>>>(rows, R, r0, n, src, dst);
  return hipGetLastError();
}

hipError_t launch_accumulate(size_t n, const float* src, float* dst, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t blocks = (n + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  k_accumulate<<<dim3(unsigned(blocks)), dim3(256), 0, s>>>(n, src, dst);
  return hipGetLastError();
}

}  // namespace tdn
