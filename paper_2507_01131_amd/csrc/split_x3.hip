// Features for the fp32 edge pass: x [N, d, C] (fp32) becomes
// xs [N, C, 3, DP] bfloat16, the exact three-way split hi/mid/lo of every
// value with the degree index k fastest and padded with zeros to DP = 32
// (d <= 32) or 64.  A lane of the 32x32x16 bf16 MFMA then reads the eight
// consecutive k it needs for one split with a single 16-byte load.  One
// block per node: the node's [d, C] rows are staged in LDS, then each
// thread writes groups of eight k for one channel and all three parts.
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int DP>
__global__ __launch_bounds__(256) void k_split_x3(int d, int C, const float* __restrict__ x,
                                                  uint16_t* __restrict__ xs) {
  extern __shared__ float tile[];  // [d][C]
  const int n = blockIdx.x;
  const float* src = x + size_t(n) * d * C;
  for (int i = threadIdx.x; i < d * C; i += blockDim.x) tile[i] = src[i];
  __syncthreads();
  uint16_t* dst = xs + size_t(n) * C * 3 * DP;
  for (int i = threadIdx.x; i < C * (DP / 8); i += blockDim.x) {
    const int c = i / (DP / 8), g = i - c * (DP / 8);
    uint32_t w[3][4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint16_t part[3][2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int k = 8 * g + 2 * p + q;
        split_bf16x3(k < d ? tile[k * C + c] : 0.f, part[0][q], part[1][q], part[2][q]);
      }
#pragma unroll
      for (int s = 0; s < 3; ++s) w[s][p] = uint32_t(part[s][0]) | (uint32_t(part[s][1]) << 16);
    }
#pragma unroll
    for (int s = 0; s < 3; ++s)
      *reinterpret_cast<u32x4*>(dst + (size_t(c) * 3 + s) * DP + 8 * g) = u32x4{w[s][0], w[s][1], w[s][2], w[s][3]};
  }
}

template <int DP>
hipError_t launch_dp(int N, int d, int C, const float* x, uint16_t* xs, hipStream_t s) {
  const size_t lds = size_t(d) * C * 4;
  auto k = k_split_x3<DP>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(N), dim3(256), lds, s>>>(d, C, x, xs);
  return hipGetLastError();
}

}  // namespace

int x3_kpad(int d) { return d <= 32 ? 32 : 64; }

hipError_t launch_split_x3(int N, int d, int C, const float* x, void* xs, hipStream_t s) {
  if (N == 0) return hipSuccess;
  uint16_t* o = static_cast<uint16_t*>(xs);
  return x3_kpad(d) == 32 ? launch_dp<32>(N, d, C, x, o, s) : launch_dp<64>(N, d, C, x, o, s);
}

}  // namespace tdn
