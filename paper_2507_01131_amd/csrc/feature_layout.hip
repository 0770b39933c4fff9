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
// The backward's destination kernels contract over channels instead and read
// x in MFMA operand blocks over channels (launch_direct_layout).
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }

// x[node] ([d, C] values, dC = d C a multiple of 16) into LDS as fp32, rows
// contiguous, or C + 1 floats apart when C > 0 is given; returns this
// thread's largest |x|.  Sixteen-byte loads, four per thread
// issued before their LDS stores, when the rows are 16-byte aligned; single
// values otherwise.
template <typename TI>
__device__ inline float stage_node(const TI* __restrict__ src, int dC, float* __restrict__ tile, int C = 0) {
  float mx = 0.f;
  if ((reinterpret_cast<uintptr_t>(src) & 15) != 0) {
    for (int i = threadIdx.x; i < dC; i += blockDim.x) {
      const float v = to_f32(src[i]);
      tile[C > 0 ? i + i / C : i] = v;
      mx = fmaxf(mx, fabsf(v));
    }
    return mx;
  }
  constexpr int V = 16 / sizeof(TI);  // values per load
  const int nv = dC / V;
  const u32x4* s4 = reinterpret_cast<const u32x4*>(src);
  for (int i0 = threadIdx.x; i0 < nv; i0 += 4 * blockDim.x) {
    u32x4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * blockDim.x;
      r[u] = i < nv ? s4[i] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * blockDim.x;
      if (i >= nv) continue;
      float v[V];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (V == 4) {
          v[j] = __uint_as_float(r[u][j]);
        } else {
          v[2 * j] = bf16_to_f32(uint16_t(r[u][j] & 0xffffu));
          v[2 * j + 1] = bf16_to_f32(uint16_t(r[u][j] >> 16));
        }
      }
#pragma unroll
      for (int j = 0; j < V; j += 4) {
        if (C > 0) {
          // rows C + 1 floats apart (C a multiple of 16: the run lies in one row)
          float* o = tile + i * V + j + (i * V) / C;
#pragma unroll
          for (int u2 = 0; u2 < 4; ++u2) o[u2] = v[j + u2];
        } else {
          *reinterpret_cast<float4*>(tile + i * V + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
        }
        mx = fmaxf(mx, fmaxf(fmaxf(fabsf(v[j]), fabsf(v[j + 1])), fmaxf(fabsf(v[j + 2]), fabsf(v[j + 3]))));
      }
    }
  }
  return mx;
}

template <int DP, int P, typename TI>
__global__ __launch_bounds__(256) void k_feature_layout(int d, int C, const TI* __restrict__ x,
                                                        uint16_t* __restrict__ xs, float* __restrict__ row_scale) {
  extern __shared__ __align__(16) float tile[];  // [d][C], then four floats for the row maximum
  float* red = tile + d * C;
  const int n = blockIdx.x;
  const TI* src = x + size_t(n) * d * C;
  float mx = stage_node(src, d * C, tile);
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

// Packed split operands of the edge pass (fp32 features; see
// launch_feature_layout_packed): per node and 32-channel tile, lane
// (h, c) = (lane / 32, lane % 32) holds n = pk_rows(d) 32-bit words, word j
// packing the fp16 values 2j (low half) and 2j + 1, value p being the hi
// part of x'[h n + p][c] for p < n and the lo part of x'[h n + p - n][c]
// otherwise (x' = x[node] 2^-e_node, zero past d and C).  The words sit as
// [n / 4 quads][64 lanes][4 words] and then [64 lanes][n % 4 words], so the
// 64 lanes of each load read one contiguous run.
// One block of four waves per node, no LDS staging: thread (wave, lane)
// loads the n values that its words need (rows h n .. h n + n - 1 of
// channel c in tiles wave, wave + 4; one row's 32 channels are a 128-byte
// run per half-wave), the block takes the node's largest magnitude, and
// each thread forms and stores its words.  Against a block that staged the
// node's rows in LDS first: 0.025 -> 0.017 ms at the 3200-node, L = 4,
// C = 128 size (the LDS copy capped the blocks per CU), same words.
template <int PN, int MT>
__global__ __launch_bounds__(256) void k_feature_layout_packed(int d, int C, const float* __restrict__ x,
                                                               uint32_t* __restrict__ xp,
                                                               float* __restrict__ row_scale) {
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int n_ct = (C + 31) / 32;
  const int node = blockIdx.x;
  float v[MT][PN];
  float mx = 0.f;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int c = (wave + 4 * m) * 32 + l32;
    const float* src = x + size_t(node) * d * C + c;
#pragma unroll
    for (int r = 0; r < PN; ++r) {
      const int row = h * PN + r;
      v[m][r] = (c < C && row < d) ? src[size_t(row) * C] : 0.f;
    }
  }
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int r = 0; r < PN; ++r) mx = fmaxf(mx, fabsf(v[m][r]));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const int e = f16_split_exponent(mx);
  const float sc = ldexpf(1.f, -e);
  if (tid == 0) row_scale[node] = ldexpf(1.f, e);
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int ct = wave + 4 * m;
    if (ct >= n_ct) break;
    uint32_t hv[PN], lv[PN];  // fp16 bits of the hi and lo parts
#pragma unroll
    for (int r = 0; r < PN; ++r) {
      const float y = v[m][r] * sc;
      const _Float16 hi = static_cast<_Float16>(y);
      hv[r] = __builtin_bit_cast(uint16_t, hi);
      lv[r] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(y - float(hi)));
    }
    uint32_t w[PN];
#pragma unroll
    for (int j = 0; j < PN; ++j) {
      const int s0 = 2 * j, s1 = 2 * j + 1;
      w[j] = (s0 < PN ? hv[s0] : lv[s0 - PN]) | ((s1 < PN ? hv[s1] : lv[s1 - PN]) << 16);
    }
    uint32_t* o = xp + (size_t(node) * n_ct + ct) * 64 * PN;
    constexpr int NQ = PN / 4, NT = PN % 4;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      *reinterpret_cast<u32x4*>(o + (q * 64 + lane) * 4) = u32x4{w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]};
#pragma unroll
    for (int t = 0; t < NT; ++t) o[NQ * 256 + lane * NT + t] = w[4 * NQ + t];
  }
}

template <int PN>
hipError_t launch_packed_pn(int N, int d, int C, const float* x, uint32_t* xp, float* row_scale, hipStream_t s) {
  if (C <= 128)
    k_feature_layout_packed<PN, 1><<<dim3(N), dim3(256), 0, s>>>(d, C, x, xp, row_scale);
  else
    k_feature_layout_packed<PN, 2><<<dim3(N), dim3(256), 0, s>>>(d, C, x, xp, row_scale);
  return hipGetLastError();
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

// xd[n][p][s][h][k][i] = part p of x[n][k][c(s, h, i)] (zero from channel C):
// the operand blocks of a 32x32x16 MFMA contracting channels, lane (h, k)
// holding eight channels of K-step s.  c(s, h, i) = 16 s + 8 h + i (plain),
// or with PERM 16 s + 8 (i/4) + 4 h + i%4, the order in which the backward's
// direct kernel holds Gh^T in accumulator registers.  P = 2: fp16 hi and lo of x[n] 2^-e_n with
// 2^e_n (the row's largest |x| to [2^13, 2^14)) in row_scale[n]; P = 1:
// bf16.  One block per node: its [d, C] rows staged in LDS with their
// maximum, then one thread per (s, h, k) run of eight channels.  The staged
// rows are C + 1 floats apart: the threads of a wave read one channel of
// consecutive rows, which with rows C floats apart (C a multiple of 16) all
// fell in one or two LDS banks.
template <int P, typename TI, bool PERM>
__global__ __launch_bounds__(256) void k_direct_layout(int d, int C, int Cp, const TI* __restrict__ x,
                                                       uint16_t* __restrict__ xd, float* __restrict__ row_scale) {
  extern __shared__ __align__(16) float tile[];  // [d][C + 1], then four floats for the row maximum
  const int S = C + 1;
  float* red = tile + d * S;
  const int n = blockIdx.x;
  const TI* src = x + size_t(n) * d * C;
  float mx = stage_node(src, d * C, tile, C);  // row k at k (C + 1)
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
      const int c0 = PERM ? 16 * st + 8 * (i0 / 4) + 4 * h + i0 % 4 : 16 * st + 8 * h + i0;
      const float v0 = c0 < C ? tile[k * S + c0] : 0.f;
      const float v1 = c0 + 1 < C ? tile[k * S + c0 + 1] : 0.f;
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
hipError_t launch_direct_p(int N, int d, int C, int Cp, const TI* x, void* xd, float* row_scale, bool perm,
                           hipStream_t s) {
  const size_t lds = (size_t(d) * (C + 1) + 4) * 4;
  auto k = perm ? k_direct_layout<P, TI, true> : k_direct_layout<P, TI, false>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(N), dim3(256), lds, s>>>(d, C, Cp, x, static_cast<uint16_t*>(xd), row_scale);
  return hipGetLastError();
}

}  // namespace

int edge_kpad(int d) { return d <= 32 ? 32 : 64; }

hipError_t launch_direct_layout(int N, int d, int C, int Cp, const void* x, bool x_is_f32, int parts, void* xd,
                                float* row_scale, bool perm_channels, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (Cp < C || Cp % 16 || size_t(d) * (C + 1) * 4 + 16 > 160 * 1024) return hipErrorInvalidValue;
  const bool pm = perm_channels;
  if (parts == 2) {
    if (!x_is_f32 || !row_scale) return hipErrorInvalidValue;
    return launch_direct_p<2>(N, d, C, Cp, static_cast<const float*>(x), xd, row_scale, pm, s);
  }
  if (parts != 1) return hipErrorInvalidValue;
  return x_is_f32 ? launch_direct_p<1>(N, d, C, Cp, static_cast<const float*>(x), xd, nullptr, pm, s)
                  : launch_direct_p<1>(N, d, C, Cp, static_cast<const uint16_t*>(x), xd, nullptr, pm, s);
}

hipError_t launch_feature_layout_packed(int N, int d, int C, const float* x, void* xp, float* row_scale,
                                        hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (!x || !xp || !row_scale || C < 1 || C > 256) return hipErrorInvalidValue;
  uint32_t* w = static_cast<uint32_t*>(xp);
  switch (pk_rows(d)) {  // d = (L + 1)^2, L = 0 .. 6
    case 1: return launch_packed_pn<1>(N, d, C, x, w, row_scale, s);
    case 2: return launch_packed_pn<2>(N, d, C, x, w, row_scale, s);
    case 5: return launch_packed_pn<5>(N, d, C, x, w, row_scale, s);
    case 8: return launch_packed_pn<8>(N, d, C, x, w, row_scale, s);
    case 13: return launch_packed_pn<13>(N, d, C, x, w, row_scale, s);
    case 18: return launch_packed_pn<18>(N, d, C, x, w, row_scale, s);
    case 25: return launch_packed_pn<25>(N, d, C, x, w, row_scale, s);
    default: return hipErrorInvalidValue;
  }
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
