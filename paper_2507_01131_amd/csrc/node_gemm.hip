// Per-node channel GEMMs of the layer.
//
// Path-weight sharing (Sec. 3.2) gives one W for every path; W acts only on
// the channel index, so it commutes with the sum over edges and with D and is
// applied once per node row: out[n*d + m, :] = Z[n*d + m, :] W.  In the
// backward, Gz = grad_out W^T (same kernel, W read transposed) and
// grad_W = sum_rows Z^T grad_out, split over fixed row chunks whose partial
// C x C products are summed in a fixed order (deterministic, no atomics).
#include "common.hpp"
#include "kernels.h"

namespace tdn {

namespace {

constexpr int kBM = 64;   // rows per block
constexpr int kBN = 128;  // columns per block
constexpr int kBK = 32;   // contraction chunk staged in LDS

template <typename TW>
__global__ __launch_bounds__(256) void k_node_gemm(int rows, int C, const float* __restrict__ in,
                                                   const TW* __restrict__ W, int transpose_w,
                                                   float* __restrict__ out) {
  __shared__ float sA[kBM][kBK + 1];
  __shared__ float sW[kBK][kBN + 4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int r0 = blockIdx.x * kBM, c0 = blockIdx.y * kBN;
  const int wr = wave >> 1, wc = wave & 1;
  f32x16 acc[2] = {f32x16{}, f32x16{}};
  for (int k0 = 0; k0 < C; k0 += kBK) {
    {  // 64 x 32 tile of `in`: thread -> (row, 8 consecutive columns)
      const int row = tid >> 2, kq = (tid & 3) * 8;
      const int gr = r0 + row, gk = k0 + kq;
      for (int i = 0; i < 8; ++i) sA[row][kq + i] = (gr < rows && gk + i < C) ? in[size_t(gr) * C + gk + i] : 0.f;
    }
    if (!transpose_w) {  // sW[k][n] = W[k0+k][c0+n]
      const int kr = tid >> 3, n0 = (tid & 7) * 16;
      const int gk = k0 + kr;
      for (int i = 0; i < 16; ++i) {
        const int gn = c0 + n0 + i;
        sW[kr][n0 + i] = (gk < C && gn < C) ? load_feat<TW>(W + size_t(gk) * C + gn) : 0.f;
      }
    } else {  // sW[k][n] = W[c0+n][k0+k]
      const int n = tid >> 1, kk = (tid & 1) * 16;
      const int gn = c0 + n;
      for (int i = 0; i < 16; ++i) {
        const int gk = k0 + kk + i;
        sW[kk + i][n] = (gk < C && gn < C) ? load_feat<TW>(W + size_t(gn) * C + gk) : 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kBK / 2; ++s) {
      const float av = sA[wr * 32 + l32][2 * s + h];
#pragma unroll
      for (int t = 0; t < 2; ++t) acc[t] = mfma32(av, sW[2 * s + h][wc * 64 + t * 32 + l32], acc[t]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int col = c0 + wc * 64 + t * 32 + l32;
    if (col >= C) continue;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = r0 + wr * 32 + acc_row(v, h);
      if (row < rows) out[size_t(row) * C + col] = acc[t][v];
    }
  }
}

// partial[p][ci][co] = sum over rows of chunk p of Z[row][ci] G[row][co].
// One wave per (chunk, ci tile, group of up to 4 co tiles).
__global__ __launch_bounds__(64) void k_gram_partial(int rows, int C, int rows_per_part, const float* __restrict__ Z,
                                                     const float* __restrict__ G, float* __restrict__ partial) {
  const int p = blockIdx.x, cit = blockIdx.y, cog = blockIdx.z;
  const int lane = threadIdx.x, h = lane >> 5, l32 = lane & 31;
  const int lo = p * rows_per_part, hi = min(rows, lo + rows_per_part);
  const int ci = cit * kTile + l32;
  f32x16 acc[4] = {f32x16{}, f32x16{}, f32x16{}, f32x16{}};
  for (int r = lo; r < hi; r += 2) {
    const int row = r + h;
    const bool ok = row < hi;
    const float av = (ok && ci < C) ? Z[size_t(row) * C + ci] : 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int co = (cog * 4 + t) * kTile + l32;
      const float bv = (ok && co < C) ? G[size_t(row) * C + co] : 0.f;
      acc[t] = mfma32(av, bv, acc[t]);
    }
  }
  float* out = partial + size_t(p) * C * C;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int co = (cog * 4 + t) * kTile + l32;
    if (co >= C) continue;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = cit * kTile + acc_row(v, h);
      if (r < C) out[size_t(r) * C + co] = acc[t][v];
    }
  }
}

__global__ void k_sum_parts(int n_part, int CC, const float* __restrict__ partial, float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CC) return;
  float s = 0.f;
  for (int p = 0; p < n_part; ++p) s += partial[size_t(p) * CC + i];
  out[i] = s;
}

}  // namespace

hipError_t launch_node_gemm(int rows, int C, const float* in, const void* W, bool w_bf16, int transpose_w, float* out,
                            hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((rows + kBM - 1) / kBM, (C + kBN - 1) / kBN);
  if (w_bf16)
    k_node_gemm<uint16_t><<<grid, dim3(256), 0, s>>>(rows, C, in, static_cast<const uint16_t*>(W), transpose_w, out);
  else
    k_node_gemm<float><<<grid, dim3(256), 0, s>>>(rows, C, in, static_cast<const float*>(W), transpose_w, out);
  return hipGetLastError();
}

int gram_parts(int rows) {
  int p = (rows + 255) / 256;
  return p < 1 ? 1 : (p > 256 ? 256 : p);
}

hipError_t launch_gram(int rows, int C, const float* Z, const float* G, float* partial, float* grad_W, hipStream_t s) {
  const int parts = gram_parts(rows);
  int rpp = (rows + parts - 1) / parts;
  rpp += rpp & 1;
  const int ct = (C + kTile - 1) / kTile;
  if (rows > 0) k_gram_partial<<<dim3(parts, ct, (ct + 3) / 4), dim3(64), 0, s>>>(rows, C, rpp, Z, G, partial);
  else return launch_zero(grad_W, size_t(C) * C * 4, s);
  k_sum_parts<<<dim3((C * C + 255) / 256), dim3(256), 0, s>>>(parts, C * C, partial, grad_W);
  return hipGetLastError();
}

}  // namespace tdn
