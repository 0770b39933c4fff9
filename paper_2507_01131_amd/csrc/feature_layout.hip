// Feature layout for the edge pass: x [N, d, C] becomes 16-bit operand
// blocks of the 32x32x16 MFMA, xs [N, Cq/32, P, DP/16, 2, 32, 8]: element
// [n][ct][s][b][h][c][i] is part s of x[n][16 b + 8 h + i][32 ct + c], zero
// for k >= d (DP = 32 for d <= 32, else 64) and for channels from C (Cq is C
// rounded up to 32).  Lane (h, c) of a wave reads its eight k with one
// 16-byte load, and the 64 lanes read one contiguous kilobyte.
//   P = 2 (fp32 problems): fp16 parts hi, lo of x[n] 2^-e_n, the power of
//         two that puts the node's largest |x| in [2^13, 2^14); the factor
//         2^e_n goes to row_scale[n];
//   P = 1 (bf16 problems): x itself (bf16 input), or an fp32 input (the
//         backward's Gz) rounded to bf16.
// One block per node: the node's [d, C] rows are staged in LDS (with their
// largest magnitude), then each thread writes a group of eight k of one
// channel in all P parts.
// The backward's destination kernel contracts over channels instead and reads
// x in bf16 MFMA operand blocks over channels (launch_channel_layout).
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }

template <int DP, int P, typename TI>
__global__ __launch_bounds__(256) void k_feature_layout(int d, int C, const TI* __restrict__ x,
                                                        uint16_t* __restrict__ xs, float* __restrict__ row_scale) {
  extern __shared__ float tile[];  // [d][C], then four floats for the row maximum
  float* red = tile + d * C;
  const int n = blockIdx.x;
  const TI* src = x + size_t(n) * d * C;
  float mx = 0.f;
  for (int i = threadIdx.x; i < d * C; i += blockDim.x) {
    const float v = to_f32(src[i]);
    tile[i] = v;
    mx = fmaxf(mx, fabsf(v));
  }
  float sc = 1.f;  // 2^-e_n: the row's largest |x| to [2^13, 2^14) (fp16 parts)
  if constexpr (P == 2) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  }
  __syncthreads();
  if constexpr (P == 2) {
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const int e = f16_split_exponent(mx);
    sc = ldexpf(1.f, -e);
    if (threadIdx.x == 0) row_scale[n] = ldexpf(1.f, e);
  }
  constexpr int KB = DP / 16;
  const int Cq = (C + 31) / 32 * 32;
  uint16_t* dst = xs + size_t(n) * Cq * P * DP;
  // thread (g, c), c fastest: the eight k = 8 g .. 8 g + 7 of channel c
  for (int i = threadIdx.x; i < Cq * (DP / 8); i += blockDim.x) {
    const int g = i / Cq, c = i - g * Cq;
    uint32_t w[P][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = 8 * g + 2 * q;
      const float v0 = (k < d && c < C) ? tile[k * C + c] : 0.f;
      const float v1 = (k + 1 < d && c < C) ? tile[(k + 1) * C + c] : 0.f;
      if constexpr (P == 2)
        split_f16x2_pair(v0 * sc, v1 * sc, w[0][q], w[1][q]);
      else
        w[0][q] = pack_bf16x2_rne(v0, v1);  // exact for bf16 input
    }
    const int ct = c / 32, c32 = c % 32, b = g / 2, h = g % 2;
#pragma unroll
    for (int s = 0; s < P; ++s)
      *reinterpret_cast<u32x4*>(dst + (((((ct * P + s) * KB + b) * 2 + h) * 32 + c32) * 8)) =
          u32x4{w[s][0], w[s][1], w[s][2], w[s][3]};
  }
}

template <int DP, int P, typename TI>
hipError_t launch_dp(int N, int d, int C, const TI* x, uint16_t* xs, float* row_scale, hipStream_t s) {
  const size_t lds = (size_t(d) * C + 4) * 4;
  auto k = k_feature_layout<DP, P, TI>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(N), dim3(256), lds, s>>>(d, C, x, xs, row_scale);
  return hipGetLastError();
}

template <int P, typename TI>
hipError_t launch_p(int N, int d, int C, const TI* x, void* xs, float* row_scale, hipStream_t s) {
  uint16_t* o = static_cast<uint16_t*>(xs);
  return edge_kpad(d) == 32 ? launch_dp<32, P>(N, d, C, x, o, row_scale, s)
                            : launch_dp<64, P>(N, d, C, x, o, row_scale, s);
}

// xc[n][p][s][h][k][i] = part p of x[n][k][16 s + 8 h + i] (zero from
// channel C): for every node, part and K-step s of 16 channels, the operand
// block of a 32x32x16 MFMA with the rows k < d, so that the 64 lanes of a
// wave read one contiguous block.  One thread per (node, s, h, k), k fastest.
template <int P, typename TI>
__global__ __launch_bounds__(256) void k_channel_layout(int N, int d, int C, int Cp, const TI* __restrict__ x,
                                                        uint16_t* __restrict__ xc) {
  const int nks = Cp / 16;
  const size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= size_t(N) * nks * 2 * d) return;
  const int k = int(i % d);
  size_t rest = i / d;
  const int h = int(rest % 2);
  rest /= 2;
  const int st = int(rest % nks);
  const size_t n = rest / nks;
  const int c0 = 16 * st + 8 * h;
  const TI* src = x + (n * d + k) * C;
  uint32_t w[P][4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = c0 + 2 * q;
    const float v0 = c < C ? to_f32(src[c]) : 0.f;
    const float v1 = c + 1 < C ? to_f32(src[c + 1]) : 0.f;
    if constexpr (P == 3)
      split_bf16x3_pair(v0, v1, w[0][q], w[1][q], w[2][q]);
    else
      w[0][q] = pack_bf16x2_rne(v0, v1);
  }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    uint16_t* dst = xc + ((((n * P + p) * nks + st) * 2 + h) * d + k) * 8;
    *reinterpret_cast<u32x4*>(dst) = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
  }
}

template <int P, typename TI>
hipError_t launch_channel_p(int N, int d, int C, int Cp, const TI* x, void* xc, hipStream_t s) {
  const size_t items = size_t(N) * (Cp / 16) * 2 * d;
  k_channel_layout<P, TI><<<dim3(unsigned((items + 255) / 256)), dim3(256), 0, s>>>(N, d, C, Cp, x,
                                                                                    static_cast<uint16_t*>(xc));
  return hipGetLastError();
}

// xd[n][p][s][h][k][i] = part p of x[n][k][16 s + 8 (i/4) + 4 h + i%4] (zero
// from channel C): the operand blocks of a 32x32x16 MFMA contracting
// channels in the order in which the backward's direct kernel holds
// Gh^T in accumulator registers.  P = 2: fp16 hi and lo of x[n] 2^-e_n with
// 2^e_n (the row's largest |x| to [2^13, 2^14)) in row_scale[n]; P = 1:
// bf16.  One block per node: its [d, C] rows staged in LDS with their
// maximum, then one thread per (s, h, k) run of eight channels.
template <int P, typename TI>
__global__ __launch_bounds__(256) void k_direct_layout(int d, int C, int Cp, const TI* __restrict__ x,
                                                       uint16_t* __restrict__ xd, float* __restrict__ row_scale) {
  extern __shared__ float tile[];  // [d][C], then four floats for the row maximum
  float* red = tile + d * C;
  const int n = blockIdx.x;
  const TI* src = x + size_t(n) * d * C;
  float mx = 0.f;
  for (int i = threadIdx.x; i < d * C; i += blockDim.x) {
    const float v = to_f32(src[i]);
    tile[i] = v;
    mx = fmaxf(mx, fabsf(v));
  }
  float sc = 1.f;
  if constexpr (P == 2) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  }
  __syncthreads();
  if constexpr (P == 2) {
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const int e = f16_split_exponent(mx);
    sc = ldexpf(1.f, -e);
    if (threadIdx.x == 0) row_scale[n] = ldexpf(1.f, e);
  }
  const int ns = Cp / 16;
  uint16_t* dst = xd + size_t(n) * P * ns * 2 * d * 8;
  // thread (s, h, k), k fastest: consecutive threads write consecutive 16 bytes
  for (int i = threadIdx.x; i < ns * 2 * d; i += blockDim.x) {
    const int k = i % d, sh = i / d, h = sh & 1, st = sh >> 1;
    uint32_t w[P][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i0 = 2 * q;  // elements i0, i0 + 1 of the run
      const int c0 = 16 * st + 8 * (i0 / 4) + 4 * h + i0 % 4;
      const float v0 = c0 < C ? tile[k * C + c0] : 0.f;
      const float v1 = c0 + 1 < C ? tile[k * C + c0 + 1] : 0.f;
      if constexpr (P == 2)
        split_f16x2_pair(v0 * sc, v1 * sc, w[0][q], w[1][q]);
      else
        w[0][q] = pack_bf16x2_rne(v0, v1);
    }
#pragma unroll
    for (int p = 0; p < P; ++p)
      *reinterpret_cast<u32x4*>(dst + ((size_t(p) * ns * 2 + sh) * d + k) * 8) =
          u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
  }
}

template <int P, typename TI>
hipError_t launch_direct_p(int N, int d, int C, int Cp, const TI* x, void* xd, float* row_scale, hipStream_t s) {
  const size_t lds = (size_t(d) * C + 4) * 4;
  auto k = k_direct_layout<P, TI>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(N), dim3(256), lds, s>>>(d, C, Cp, x, static_cast<uint16_t*>(xd), row_scale);
  return hipGetLastError();
}

}  // namespace

int edge_kpad(int d) { return d <= 32 ? 32 : 64; }

hipError_t launch_channel_layout(int N, int d, int C, int Cp, const void* x, bool x_is_f32, int parts, void* xc,
                                 hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (Cp < C || Cp % 16) return hipErrorInvalidValue;
  if (parts == 3) {
    if (!x_is_f32) return hipErrorInvalidValue;
    return launch_channel_p<3>(N, d, C, Cp, static_cast<const float*>(x), xc, s);
  }
  if (parts != 1) return hipErrorInvalidValue;
  return x_is_f32 ? launch_channel_p<1>(N, d, C, Cp, static_cast<const float*>(x), xc, s)
                  : launch_channel_p<1>(N, d, C, Cp, static_cast<const uint16_t*>(x), xc, s);
}

hipError_t launch_direct_layout(int N, int d, int C, int Cp, const void* x, bool x_is_f32, int parts, void* xd,
                                float* row_scale, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (Cp < C || Cp % 16 || size_t(d) * C * 4 + 16 > 160 * 1024) return hipErrorInvalidValue;
  if (parts == 2) {
    if (!x_is_f32 || !row_scale) return hipErrorInvalidValue;
    return launch_direct_p<2>(N, d, C, Cp, static_cast<const float*>(x), xd, row_scale, s);
  }
  if (parts != 1) return hipErrorInvalidValue;
  return x_is_f32 ? launch_direct_p<1>(N, d, C, Cp, static_cast<const float*>(x), xd, nullptr, s)
                  : launch_direct_p<1>(N, d, C, Cp, static_cast<const uint16_t*>(x), xd, nullptr, s);
}

hipError_t launch_feature_layout(int N, int d, int C, const void* x, bool x_is_f32, int parts, void* xs,
                                 float* row_scale, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (parts == 2) {
    if (!x_is_f32 || !row_scale) return hipErrorInvalidValue;
    return launch_p<2>(N, d, C, static_cast<const float*>(x), xs, row_scale, s);
  }
  if (parts != 1) return hipErrorInvalidValue;
  return x_is_f32 ? launch_p<1>(N, d, C, static_cast<const float*>(x), xs, nullptr, s)
                  : launch_p<1>(N, d, C, static_cast<const uint16_t*>(x), xs, nullptr, s);
}

}  // namespace tdn
