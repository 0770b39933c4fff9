// Per-node channel GEMMs of the layer.
//
// Path-weight sharing (Sec. 3.2) gives one W for every path; W acts only on
// the channel index, so it commutes with the sum over edges and with D and is
// applied once per node row: out[n*d + m, :] = Z[n*d + m, :] W.  In the
// backward, Gz = grad_out W^T (same kernel, W read transposed) and
// grad_W = sum_rows Z^T grad_out, split over fixed row chunks whose partial
// C x C products are summed in a fixed order (deterministic, no atomics).
//
// All of them stage operands through LDS for MFMA: a 128 x 128 output tile
// per workgroup, four waves of 64 x 64 (2 x 2 MFMA tiles, so every operand
// read from LDS feeds two MFMAs), contraction staged in chunks of 32.  The
// fp32 node GEMMs run on 32x32x16 fp16 MFMA over scaled two-part splits
// (k_node_gemm_f16); the Gram products of fp32 problems use 32x32x2 fp32
// MFMA; bf16 problems (bf16 W) use 32x32x16 bf16 MFMA with the fp32 operand
// rounded to bf16 while it is staged.  Without path-weight sharing, each
// path has its own channel matrix; the path GEMM applies them to the per-path
// node sums (they too commute with the edge sum) on 32x32x2 fp32 MFMA.
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;  // output rows per block
constexpr int kBN = 128;  // output columns per block
constexpr int kBK = 32;   // contraction chunk
constexpr int kSF = kBK + 1;  // fp32 LDS row stride (floats)
constexpr int kSH = kBK + 8;  // bf16 LDS row stride (halves): 80-byte rows

__device__ __forceinline__ uint16_t bf16_bits(float v) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v)); }

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 16 consecutive elements as floats (zero when out of range; `n_ok` of them
// valid).  Element types: float (four float4 loads) or bf16 bits (two 16-byte
// loads).
template <typename T>
__device__ __forceinline__ void load16(const T* p, int n_ok, float (&v)[16]);
template <>
__device__ __forceinline__ void load16<float>(const float* p, int n_ok, float (&v)[16]) {
  if (n_ok >= 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 t = *reinterpret_cast<const f32x4*>(p + 4 * q);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * q + i] = t[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n_ok ? p[i] : 0.f;
  }
}
template <>
__device__ __forceinline__ void load16<uint16_t>(const uint16_t* p, int n_ok, float (&v)[16]) {
  if (n_ok >= 16) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const u32x4 t = *reinterpret_cast<const u32x4*>(p + 8 * q);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[8 * q + 2 * i] = __uint_as_float(t[i] << 16);
        v[8 * q + 2 * i + 1] = __uint_as_float(t[i] & 0xffff0000u);
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n_ok ? __uint_as_float(uint32_t(p[i]) << 16) : 0.f;
  }
}

// out[m][n] = sum_k L(m, k) R(k, n) for one 128 x 128 tile, k in
// [k_begin, k_end):
//   L(m, k) = lhs[(m0 + m) * ldl + k]  (LT = false)   or lhs[k * ldl + m0 + m]  (LT = true)
//   R(k, n) = rhs[k * ldr + n0 + n]    (RT = false)   or rhs[(n0 + n) * ldr + k] (RT = true)
// Each 32-deep chunk is staged "contraction-fastest" in LDS (sa[m][k],
// sb[n][k]); every thread brings 16 consecutive elements of each operand with
// vector loads, and the next chunk's loads are issued before the current
// chunk's MFMAs (register double buffer).  BF16 rounds both operands to bf16
// at staging and runs 32x32x16 bf16 MFMA; otherwise 32x32x2 fp32 MFMA.
template <bool BF16, bool LT, bool RT, typename TL, typename TR>
__device__ inline void gemm_tile(const TL* __restrict__ lhs, int ldl, int M, const TR* __restrict__ rhs, int ldr,
                                 int Ncols, int k_begin, int k_end, int m0, int n0, f32x16 (&acc)[2][2], void* smem) {
  constexpr int SS = BF16 ? kSH : kSF;  // LDS row stride in elements
  float* sa_f = static_cast<float*>(smem);
  float* sb_f = sa_f + kBM * kSF;
  uint16_t* sa_h = static_cast<uint16_t*>(smem);
  uint16_t* sb_h = sa_h + kBM * kSH;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int wr = wave >> 1, wc = wave & 1;
  // this thread's 16-element runs: along k (rows of 32 -> 2 runs per row) or
  // along m/n (k fixed, 128 wide -> 8 runs per k)
  const int a_r = LT ? tid / 8 : tid / 2, a_c = LT ? (tid % 8) * 16 : (tid % 2) * 16;
  const int b_r = RT ? tid / 2 : tid / 8, b_c = RT ? (tid % 2) * 16 : (tid % 8) * 16;
  float va[16], vb[16];
  auto fetch = [&](int k0) {
    if constexpr (LT) {  // run: k = k0 + a_r, m = m0 + a_c .. +15
      const int gk = k0 + a_r;
      const int n_ok = gk < k_end ? min(16, M - (m0 + a_c)) : 0;
      load16<TL>(lhs + size_t(gk < k_end ? gk : k_begin) * ldl + (m0 + a_c < M ? m0 + a_c : 0), n_ok, va);
    } else {             // run: m = m0 + a_r, k = k0 + a_c .. +15
      const int gm = m0 + a_r;
      const int n_ok = gm < M ? min(16, k_end - (k0 + a_c)) : 0;
      load16<TL>(lhs + size_t(gm < M ? gm : 0) * ldl + (k0 + a_c < k_end ? k0 + a_c : k_begin), n_ok, va);
    }
    if constexpr (RT) {  // run: n = n0 + b_r, k = k0 + b_c .. +15
      const int gn = n0 + b_r;
      const int n_ok = gn < Ncols ? min(16, k_end - (k0 + b_c)) : 0;
      load16<TR>(rhs + size_t(gn < Ncols ? gn : 0) * ldr + (k0 + b_c < k_end ? k0 + b_c : k_begin), n_ok, vb);
    } else {             // run: k = k0 + b_r, n = n0 + b_c .. +15
      const int gk = k0 + b_r;
      const int n_ok = gk < k_end ? min(16, Ncols - (n0 + b_c)) : 0;
      load16<TR>(rhs + size_t(gk < k_end ? gk : k_begin) * ldr + (n0 + b_c < Ncols ? n0 + b_c : 0), n_ok, vb);
    }
  };
  auto put = [&]() {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int am = LT ? a_c + i : a_r, ak = LT ? a_r : a_c + i;
      const int bn = RT ? b_r : b_c + i, bk = RT ? b_c + i : b_r;
      if constexpr (BF16) {
        sa_h[am * SS + ak] = bf16_bits(va[i]);
        sb_h[bn * SS + bk] = bf16_bits(vb[i]);
      } else {
        sa_f[am * SS + ak] = va[i];
        sb_f[bn * SS + bk] = vb[i];
      }
    }
  };
  if (k_begin >= k_end) return;
  fetch(k_begin);
  for (int k0 = k_begin; k0 < k_end; k0 += kBK) {
    __syncthreads();  // the previous chunk's operands are consumed
    put();
    __syncthreads();
    if (k0 + kBK < k_end) fetch(k0 + kBK);
    if constexpr (BF16) {
#pragma unroll
      for (int s = 0; s < kBK / 16; ++s) {
        bf16x8 av[2], bv[2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          av[i] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(sa_h + (wr * 64 + i * 32 + l32) * SS + 16 * s + 8 * h));
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bv[j] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(sb_h + (wc * 64 + j * 32 + l32) * SS + 16 * s + 8 * h));
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma32_bf16(av[i], bv[j], acc[i][j]);
      }
    } else {
#pragma unroll
      for (int s = 0; s < kBK / 2; ++s) {
        const int k = 2 * s + h;
        float av[2], bv[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) av[i] = sa_f[(wr * 64 + i * 32 + l32) * SS + k];
#pragma unroll
        for (int j = 0; j < 2; ++j) bv[j] = sb_f[(wc * 64 + j * 32 + l32) * SS + k];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(av[i], bv[j], acc[i][j]);
      }
    }
  }
}

__device__ inline void store_tile(const f32x16 (&acc)[2][2], float* __restrict__ out, int ldo, int M, int Ncols, int m0,
                                  int n0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int wr = wave >> 1, wc = wave & 1;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wc * 64 + j * 32 + l32;
      if (col >= Ncols) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wr * 64 + i * 32 + acc_row(v, h);
        if (row < M) out[size_t(row) * ldo + col] = acc[i][j][v];
      }
    }
}

// ---- fp32 problems: the node GEMM on fp16 MFMA over two-part splits.
// W (or W^T) is split once per call into wp[p][n][k] (fp16 parts of
// W 2^-e_W, contraction fastest; 2^e_W after them); every row of `in` is
// scaled by the power of two that puts its largest |value| in [2^13, 2^14)
// and split while it is staged; out = (sum of the three part products with
// i + j <= 3) x 2^(e_row + e_W).
__global__ __launch_bounds__(1024) void k_w_parts(int C, int transpose_w, const float* __restrict__ W,
                                                  uint16_t* __restrict__ wp) {
  __shared__ float red[16];
  const int tid = threadIdx.x;
  // every block finds W's largest magnitude itself (C*C <= 65536 floats,
  // float4 loads, independent iterations), then splits its slice of pairs
  float mx = 0.f;
  const int n4 = C * C / 4;
#pragma unroll 4
  for (int i = tid; i < n4; i += blockDim.x) {
    const f32x4 v = reinterpret_cast<const f32x4*>(W)[i];
    mx = fmaxf(mx, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  for (int w = 0; w < int(blockDim.x >> 6); ++w) mx = fmaxf(mx, red[w]);
  const int e = f16_split_exponent(mx);
  const float sc = ldexpf(1.f, -e);
  // pair i: element (n, k), (n, k + 1) of the B operand: W[k][n] (out = in W)
  // or W[n][k] (in W^T)
  const int i = blockIdx.x * blockDim.x + tid;
  if (i < C * C / 2) {
    const int n = (2 * i) / C, k = (2 * i) % C;
    const float v0 = transpose_w ? W[n * C + k] : W[k * C + n];
    const float v1 = transpose_w ? W[n * C + k + 1] : W[(k + 1) * C + n];
    uint32_t hi, lo;
    split_f16x2_pair(v0 * sc, v1 * sc, hi, lo);
    reinterpret_cast<uint32_t*>(wp)[i] = hi;
    reinterpret_cast<uint32_t*>(wp)[C * C / 2 + i] = lo;
  }
  if (blockIdx.x == 0 && tid == 0) *reinterpret_cast<float*>(wp + 2 * C * C) = ldexpf(1.f, e);
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma32_f16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0,
                                                0);
}

// out[rows, C] = in[rows, C] B with B given as the parts wp (k_w_parts), for
// C <= 32 NCH.  BM x 128 output tile per workgroup (BM = 128 or 64), four
// waves of BM/2 x 64.
// The block loads all NCH 32-wide chunks of its rows at once (coalesced,
// straight into registers), so each row's largest magnitude needs one
// memory latency; then per 32-deep chunk both operands are staged in LDS as
// fp16 parts (the row parts split on the way, W's next chunk loaded one
// chunk ahead) and every 16-deep step runs the three part products.
template <int NCH, int BM>
__global__ __launch_bounds__(256) void k_node_gemm_f16(int rows, int C, const float* __restrict__ in,
                                                       const uint16_t* __restrict__ wp, float* __restrict__ out) {
  constexpr int JR = BM / 32;  // 32-row groups of the block's row loads
  constexpr int MI = BM / 64;  // 32-row MFMA tiles per wave
  __shared__ __align__(16) uint16_t sa[2][BM * kSH];
  __shared__ __align__(16) uint16_t sb[2][kBN * kSH];
  __shared__ float s_unscale[BM];
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * kBN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int wr = wave >> 1, wc = wave & 1;
  // row chunk loads, coalesced: per 32-wide chunk the block's BM x 32
  // floats are BM * 8 float4, thread t taking float4 f = t + 256 j
  // (j < BM / 32): row (t >> 3) + 32 j, columns 4 (t & 7) .. +3; eight
  // consecutive lanes cover one row's 128 bytes
  const int c4 = tid & 7;
  f32x4 va[NCH][JR];
#pragma unroll
  for (int it = 0; it < NCH; ++it)
#pragma unroll
    for (int j = 0; j < JR; ++j) {
      const int r = (tid >> 3) + 32 * j, k = it * kBK + 4 * c4;
      va[it][j] = (m0 + r < rows && k < C) ? *reinterpret_cast<const f32x4*>(in + size_t(m0 + r) * C + k) : f32x4{};
    }
  float rsc[JR];
#pragma unroll
  for (int j = 0; j < JR; ++j) {
    float mx = 0.f;
#pragma unroll
    for (int it = 0; it < NCH; ++it)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, fabsf(va[it][j][i]));
    mx = fmaxf(mx, __shfl_xor(mx, 1));
    mx = fmaxf(mx, __shfl_xor(mx, 2));
    mx = fmaxf(mx, __shfl_xor(mx, 4));
    const int er = f16_split_exponent(mx);
    rsc[j] = ldexpf(1.f, -er);
    if (c4 == 0) s_unscale[(tid >> 3) + 32 * j] = ldexpf(1.f, er);
  }
  const float w_unscale = *reinterpret_cast<const float*>(wp + 2 * C * C);
  // B runs: n = n0 + tid / 2, k = k0 + (tid % 2) * 16 .. +15, both parts
  const int b_r = tid / 2, b_c = (tid % 2) * 16;
  const int gn = n0 + b_r;
  f32x16 acc[MI][2];
#pragma unroll
  for (int i = 0; i < MI; ++i) acc[i][0] = acc[i][1] = f32x16{};
  u32x4 vb[2][2][2];  // [buffer][part][half of the run]
  auto fetch_b = [&](int k0, u32x4 (&b)[2][2]) {
    const int kb = k0 + b_c;
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int q = 0; q < 2; ++q)
        b[p][q] = (gn < C && kb + 8 * q < C)
                      ? *reinterpret_cast<const u32x4*>(wp + size_t(p) * C * C + size_t(gn) * C + kb + 8 * q)
                      : u32x4{};
  };
  fetch_b(0, vb[0]);
#pragma unroll
  for (int it = 0; it < NCH; ++it) {
    const int k0 = it * kBK;
    if (k0 >= C) break;
    __syncthreads();  // the previous chunk's operands are consumed
#pragma unroll
    for (int j = 0; j < JR; ++j) {
      uint32_t hi[2], lo[2];
      split_f16x2_pair(va[it][j][0] * rsc[j], va[it][j][1] * rsc[j], hi[0], lo[0]);
      split_f16x2_pair(va[it][j][2] * rsc[j], va[it][j][3] * rsc[j], hi[1], lo[1]);
      const int r = (tid >> 3) + 32 * j;
      *reinterpret_cast<uint2*>(&sa[0][r * kSH + 4 * c4]) = make_uint2(hi[0], hi[1]);
      *reinterpret_cast<uint2*>(&sa[1][r * kSH + 4 * c4]) = make_uint2(lo[0], lo[1]);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int p = 0; p < 2; ++p) *reinterpret_cast<u32x4*>(&sb[p][b_r * kSH + b_c + 8 * q]) = vb[it & 1][p][q];
    __syncthreads();
    if (it + 1 < NCH && k0 + kBK < C) fetch_b(k0 + kBK, vb[(it + 1) & 1]);
#pragma unroll
    for (int s2 = 0; s2 < kBK / 16; ++s2) {
      u32x4 av[2][MI], bv[2][2];  // [part][tile]
#pragma unroll
      for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
          av[p][i] = *reinterpret_cast<const u32x4*>(&sa[p][(wr * (BM / 2) + i * 32 + l32) * kSH + 16 * s2 + 8 * h]);
#pragma unroll
        for (int i = 0; i < 2; ++i)
          bv[p][i] = *reinterpret_cast<const u32x4*>(&sb[p][(wc * 64 + i * 32 + l32) * kSH + 16 * s2 + 8 * h]);
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = mfma32_f16(av[1][i], bv[0][j], acc[i][j]);
          acc[i][j] = mfma32_f16(av[0][i], bv[1][j], acc[i][j]);
          acc[i][j] = mfma32_f16(av[0][i], bv[0][j], acc[i][j]);
        }
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wc * 64 + j * 32 + l32;
      if (col >= C) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int rl = wr * (BM / 2) + i * 32 + acc_row(v, h);
        if (m0 + rl < rows) out[size_t(m0 + rl) * C + col] = acc[i][j][v] * (s_unscale[rl] * w_unscale);
      }
    }
}

// out[rows, C] = in[rows, C] @ W   (TW: W[k][n])   or   in @ W^T   (W[n][k])
template <typename TW, bool BF16, bool WT>
__global__ __launch_bounds__(256) void k_node_gemm(int rows, int C, const float* __restrict__ in,
                                                   const TW* __restrict__ W, float* __restrict__ out) {
  __shared__ __align__(16) float smem[2 * kBM * kSF];
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  f32x16 acc[2][2] = {{f32x16{}, f32x16{}}, {f32x16{}, f32x16{}}};
  gemm_tile<BF16, false, WT>(in, C, rows, W, C, C, 0, C, m0, n0, acc, smem);
  store_tile(acc, out, C, rows, C, m0, n0);
}

// partial[p][ci][co] = sum over rows of chunk p of Z[row][ci] G[row][co]:
// L(m = ci, k = row) = Z[row][ci] (transposed left operand),
// R(k = row, n = co) = G[row][co].
// The product without path-weight sharing: out[n][k][:] = sum over the paths
// p of degree l3 = deg k of zp[n][row[p] + k - l3^2][:] W_paths[p], one
// (row tile, column tile, k) per block, the paths accumulated in order.
__global__ __launch_bounds__(256) void k_path_gemm(int N, int C, int d, PathRows pt, const float* __restrict__ zp,
                                                   const float* __restrict__ W_paths, float* __restrict__ out) {
  __shared__ __align__(16) float smem[2 * kBM * kSF];
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN, k = blockIdx.z;
  int l3 = 0;
  while ((l3 + 1) * (l3 + 1) <= k) ++l3;
  f32x16 acc[2][2] = {{f32x16{}, f32x16{}}, {f32x16{}, f32x16{}}};
  for (int p = 0; p < pt.n_path; ++p) {
    if (pt.l3[p] != l3) continue;
    gemm_tile<false, false, false>(zp + size_t(pt.row[p] + k - l3 * l3) * C, pt.n_rows * C, N,
                                   W_paths + size_t(p) * C * C, C, C, 0, C, m0, n0, acc, smem);
  }
  store_tile(acc, out + size_t(k) * C, d * C, N, C, m0, n0);
}

template <bool BF16>
__global__ __launch_bounds__(256) void k_gram_partial(int rows, int C, int rows_per_part, const float* __restrict__ Z,
                                                      const float* __restrict__ G, float* __restrict__ partial) {
  __shared__ __align__(16) float smem[2 * kBM * kSF];
  const int p = blockIdx.x;
  const int m0 = blockIdx.y * kBM, n0 = blockIdx.z * kBN;
  const int lo = p * rows_per_part, hi = min(rows, lo + rows_per_part);
  f32x16 acc[2][2] = {{f32x16{}, f32x16{}}, {f32x16{}, f32x16{}}};
  gemm_tile<BF16, true, false>(Z, C, C, G, C, C, lo, hi, m0, n0, acc, smem);
  store_tile(acc, partial + size_t(p) * C * C, C, C, C, m0, n0);
}

// 16 outputs per workgroup, 16 slices per output: slice k sums parts
// k, k + 16, ... in order (part p at row p * stride), then the slices are
// added in order (the result does not depend on scheduling).
__global__ __launch_bounds__(256) void k_sum_parts(int n_part, int CC, int stride, const float* __restrict__ partial,
                                                   float* __restrict__ out) {
  __shared__ float sl[16][17];
  const int o = threadIdx.x & 15, k = threadIdx.x >> 4;
  const int i = blockIdx.x * 16 + o;
  float s = 0.f;
  if (i < CC)
    for (int p = k; p < n_part; p += 16) s += partial[size_t(p) * stride * CC + i];
  sl[k][o] = s;
  __syncthreads();
  if (k == 0 && i < CC) {
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) t += sl[j][o];
    out[i] = t;
  }
}

// First stage for many parts: group g (parts g kGroup .. g kGroup + kGroup
// - 1) summed in order by one thread per output, the sum written over the
// group's first part (each entry read and written by its one thread).
constexpr int kGroup = 64;
__global__ __launch_bounds__(256) void k_sum_groups(int n_part, int CC, float* __restrict__ partial) {
  const int i = blockIdx.x * 256 + threadIdx.x, g = blockIdx.y;
  if (i >= CC) return;
  const int p0 = g * kGroup, p1 = min(p0 + kGroup, n_part);
  float s = 0.f;
#pragma unroll 8
  for (int p = p0; p < p1; ++p) s += partial[size_t(p) * CC + i];
  partial[size_t(p0) * CC + i] = s;
}

}  // namespace

size_t node_gemm_ws_bytes(int C) { return size_t(2) * C * C * 2 + 256; }

hipError_t launch_node_gemm(int rows, int C, const float* in, const void* W, bool w_bf16, int transpose_w, float* out,
                            void* ws, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (C % 16) return hipErrorInvalidValue;
  const dim3 grid((rows + kBM - 1) / kBM, (C + kBN - 1) / kBN);
  if (w_bf16) {
    const uint16_t* wh = static_cast<const uint16_t*>(W);
    if (transpose_w)
      k_node_gemm<uint16_t, true, true><<<grid, dim3(256), 0, s>>>(rows, C, in, wh, out);
    else
      k_node_gemm<uint16_t, true, false><<<grid, dim3(256), 0, s>>>(rows, C, in, wh, out);
    return hipGetLastError();
  }
  if (!ws) return hipErrorInvalidValue;
  uint16_t* wp = static_cast<uint16_t*>(ws);
  k_w_parts<<<dim3((C * C / 2 + 1023) / 1024), dim3(1024), 0, s>>>(C, transpose_w, static_cast<const float*>(W), wp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // 64-row tiles: twice the workgroups of 128-row ones, so the last round of
  // workgroups on the CUs is less uneven
  constexpr int BM = 64;
  const dim3 grid_f((rows + BM - 1) / BM, (C + kBN - 1) / kBN);
  const int nch = (C + kBK - 1) / kBK;
  if (nch <= 1)
    k_node_gemm_f16<1, BM><<<grid_f, dim3(256), 0, s>>>(rows, C, in, wp, out);
  else if (nch <= 2)
    k_node_gemm_f16<2, BM><<<grid_f, dim3(256), 0, s>>>(rows, C, in, wp, out);
  else if (nch <= 4)
    k_node_gemm_f16<4, BM><<<grid_f, dim3(256), 0, s>>>(rows, C, in, wp, out);
  else
    k_node_gemm_f16<8, BM><<<grid_f, dim3(256), 0, s>>>(rows, C, in, wp, out);
  return hipGetLastError();
}

// Row parts of the Gram product: about 512 workgroups over the 128 x 128
// output tiles (two per CU), each part at least 64 rows.
int gram_parts(int rows, int C) {
  const int tiles = ((C + kBM - 1) / kBM) * ((C + kBN - 1) / kBN);
  int p = 512 / tiles;
  const int by_rows = rows / 64;
  if (p > by_rows) p = by_rows;
  return p < 1 ? 1 : p;
}

hipError_t launch_sum_parts(int n_part, int n, float* partial, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (n_part < 1 || n < 0 || !partial || !out) return hipErrorInvalidValue;
  if (n_part > 4 * kGroup) {
    // many parts: groups of kGroup summed in place first, then the groups
    const int groups = (n_part + kGroup - 1) / kGroup;
    k_sum_groups<<<dim3((n + 255) / 256, groups), dim3(256), 0, s>>>(n_part, n, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_sum_parts<<<dim3((n + 15) / 16), dim3(256), 0, s>>>(groups, n, kGroup, partial, out);
    return hipGetLastError();
  }
  k_sum_parts<<<dim3((n + 15) / 16), dim3(256), 0, s>>>(n_part, n, 1, partial, out);
  return hipGetLastError();
}

hipError_t launch_path_gemm(int N, int L, int C, const float* zp, const float* W_paths, float* out, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (L < 0 || L > 6 || C < 1 || !zp || !W_paths || !out) return hipErrorInvalidValue;
  const int d = (L + 1) * (L + 1);
  const dim3 grid((N + kBM - 1) / kBM, (C + kBN - 1) / kBN, d);
  k_path_gemm<<<grid, dim3(256), 0, s>>>(N, C, d, path_rows(L), zp, W_paths, out);
  return hipGetLastError();
}

hipError_t launch_gram(int rows, int C, const float* Z, const float* G, bool bf16, float* partial, float* grad_W,
                       hipStream_t s) {
  if (rows <= 0) return launch_zero(grad_W, size_t(C) * C * 4, s);
  const int parts = gram_parts(rows, C);
  int rpp = (rows + parts - 1) / parts;
  rpp = (rpp + kBK - 1) / kBK * kBK;
  const dim3 grid(parts, (C + kBM - 1) / kBM, (C + kBN - 1) / kBN);
  if (bf16)
    k_gram_partial<true><<<grid, dim3(256), 0, s>>>(rows, C, rpp, Z, G, partial);
  else
    k_gram_partial<false><<<grid, dim3(256), 0, s>>>(rows, C, rpp, Z, G, partial);
  k_sum_parts<<<dim3((C * C + 15) / 16), dim3(256), 0, s>>>(parts, C * C, 1, partial, grad_W);
  return hipGetLastError();
}

}  // namespace tdn
