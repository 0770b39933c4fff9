// Gradient of the radial weights.  The layer's per-edge radial weight is
// rho_e = phi_e Wrad (phi_e: the Gaussian radial basis of |r_e|, Wrad:
// [n_radial, R], one weight per rank of the CP product of Sec. 3.1), so
//   grad_Wrad[q, r] = sum_e phi_e[q] drho_e[r],
// with drho_e = dg_e * v_e stored per edge by the backward destination pass.
// Workgroup b takes the edge range [b E / B, (b+1) E / B) (B = E / 256, at
// most 2048) in chunks of 64:
// phi for the chunk into LDS, then fp32 MFMA (rows: radial functions, columns:
// ranks, contraction over the chunk's edges, two per step), one 32-rank tile
// per wave (two for R > 128).  The partial sums are added in a fixed order
// (launch_sum_parts), so the result does not depend on scheduling.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

constexpr int kGradChunk = 64;
constexpr int kEdgesPerBlock = 256;
constexpr int kMaxBlocks = 2048;

__global__ __launch_bounds__(256) void k_wrad_partial(int E, int n_blocks, int R, int nr, float sigma,
                                                      const float* __restrict__ edge_vec,
                                                      const float* __restrict__ drho, float* __restrict__ partial) {
  __shared__ float sPhi[kGradChunk * 16];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave, h = lane >> 5, l32 = lane & 31;
  const int e0 = int(int64_t(b) * E / n_blocks), e1 = int(int64_t(b + 1) * E / n_blocks);
  const int RT = (R + kTile - 1) / kTile;
  f32x16 acc[2] = {f32x16{}, f32x16{}};
  for (int cb = e0; cb < e1; cb += kGradChunk) {
    const int n = min(kGradChunk, e1 - cb);
    __syncthreads();  // the previous chunk's phi consumed
    for (int t = tid; t < n * nr; t += blockDim.x) {
      const int e = t / nr, q = t - e * nr;
      const float vx = edge_vec[3 * size_t(cb + e)], vy = edge_vec[3 * size_t(cb + e) + 1],
                  vz = edge_vec[3 * size_t(cb + e) + 2];
      sPhi[t] = radial_phi(sqrtf(vx * vx + vy * vy + vz * vz), q, sigma);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int rt = wave + 4 * j;
      if (rt < RT) {
        const int r = rt * kTile + l32;
        // every drho load of the chunk issued before the first product
        float bv[kGradChunk / 2];
#pragma unroll
        for (int s2 = 0; s2 < kGradChunk / 2; ++s2) {
          const int e = 2 * s2 + h;
          bv[s2] = (e < n && r < R) ? drho[size_t(cb + e) * R + r] : 0.f;
        }
#pragma unroll
        for (int s2 = 0; s2 < kGradChunk / 2; ++s2) {
          const int e = 2 * s2 + h;
          const float av = (e < n && l32 < nr) ? sPhi[e * nr + l32] : 0.f;
          acc[j] = mfma32(av, bv[s2], acc[j]);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int rt = wave + 4 * j;
    if (rt < RT) {
      const int r = rt * kTile + l32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int q = acc_row(v, h);
        if (q < nr && r < R) partial[(size_t(b) * nr + q) * R + r] = acc[j][v];
      }
    }
  }
}

}  // namespace

int radial_grad_blocks(int E) {
  const int b = (E + kEdgesPerBlock - 1) / kEdgesPerBlock;
  return b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b);
}

hipError_t launch_radial_grad(int E, int R, int n_radial, float sigma, const float* edge_vec, const float* drho,
                              float* partial, float* grad_radial_w, hipStream_t s) {
  if (R < 1 || R > 8 * kTile || n_radial < 1 || n_radial > 16) return hipErrorInvalidValue;
  const int n_out = n_radial * R;
  if (E == 0) return launch_zero(grad_radial_w, size_t(n_out) * 4, s);
  const int nb = radial_grad_blocks(E);
  k_wrad_partial<<<dim3(nb), dim3(256), 0, s>>>(E, nb, R, n_radial, sigma, edge_vec, drho, partial);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_sum_parts(nb, n_out, partial, grad_radial_w, s);
}

}  // namespace tdn
