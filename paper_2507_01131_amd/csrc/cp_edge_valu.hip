// Measurement ablation of the edge pass: the contraction on the vector ALUs.
// The same layer as launch_cp_edge (eq. approximate of Sec. 3.1 summed over a
// destination's edges, D applied once per node),
//   Z[t] = D sum_{e: t_e = t} diag(g_e) A^T x[s_e],  g_e = (B^T Y_e) * (phi_e Wrad),
// but every product is an fp32 fused multiply-add on the VALU instead of
// fp16 MFMA over two-part splits: one workgroup per destination node; thread
// (i, j) of 16 x 16 holds H[8i .. 8i+7][8j .. 8j+7] (ranks x channels) in
// registers over the node's edges; per edge the gathered row x[s_e] and
// g_e-scaled A columns come from LDS.  At the end H goes to LDS and Z = D H
// is formed one output per thread and step.  R <= 128, C <= 128, L <= 4.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

constexpr int kVR = 128, kVC = 128;  // rank and channel capacity
constexpr int kVHs = kVC + 1;        // row stride of H in LDS

template <int L>
__global__ __launch_bounds__(256) void k_cp_edge_valu(EdgeArgs a, const float* __restrict__ x) {
  constexpr int d = (L + 1) * (L + 1);
  extern __shared__ float smem[];
  float* sA = smem;                 // [d][kVR]  A, zero past R
  float* sX = sA + d * kVR;         // [d][kVC]  the gathered row, zero past C
  float* sG = sX + d * kVC;         // [kVR]     g_e
  float* sY = sG + kVR;             // [d]
  float* sPhi = sY + d;             // [16]
  int* sRow = reinterpret_cast<int*>(sPhi + 16);
  float* sH = smem;                 // [kVR][kVHs] at the end (aliases the above)
  const int tid = threadIdx.x, ti = tid / 16, tj = tid % 16;
  const int t = xcd_remap(blockIdx.x, a.n_seg);
  const int e0 = a.offsets[t], e1 = a.offsets[t + 1];
  const int R = a.R, C = a.C, nr = a.n_radial;
  for (int i = tid; i < d * kVR; i += blockDim.x) {
    const int k = i / kVR, r = i - k * kVR;
    sA[i] = r < R ? a.KF[k * R + r] : 0.f;
  }
  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  for (int e = e0; e < e1; ++e) {
    __syncthreads();  // A staged / the previous edge consumed
    if (tid == 0) {
      const int eid = a.perm[e];
      sRow[0] = a.gather[eid];
      const float vx = a.edge_vec[3 * size_t(eid)], vy = a.edge_vec[3 * size_t(eid) + 1],
                  vz = a.edge_vec[3 * size_t(eid) + 2];
      const float len = sqrtf(vx * vx + vy * vy + vz * vz), inv = 1.f / len;
      sh_unit_all<L>(vx * inv, vy * inv, vz * inv, sY);
      for (int q = 0; q < nr; ++q) sPhi[q] = radial_phi(len, q, a.sigma);
    }
    __syncthreads();
    const float* xr = x + size_t(sRow[0]) * d * C;
    for (int i = tid; i < d * kVC; i += blockDim.x) {
      const int k = i / kVC, c = i - k * kVC;
      sX[i] = c < C ? xr[k * C + c] : 0.f;
    }
    if (tid < kVR) {
      float v = 0.f, rho = 0.f;
      if (tid < R) {
        for (int k = 0; k < d; ++k) v = fmaf(sY[k], a.Bf[k * R + tid], v);
        for (int q = 0; q < nr; ++q) rho = fmaf(sPhi[q], a.radial_w[q * R + tid], rho);
      }
      sG[tid] = v * rho;
    }
    __syncthreads();
    float g[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) g[i] = sG[8 * ti + i];
    for (int k = 0; k < d; ++k) {
      float av[8], xv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) av[i] = g[i] * sA[k * kVR + 8 * ti + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) xv[j] = sX[k * kVC + 8 * tj + j];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(av[i], xv[j], acc[i][j]);
    }
  }
  __syncthreads();  // the last edge's operands consumed; H replaces them
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) sH[(8 * ti + i) * kVHs + 8 * tj + j] = acc[i][j];
  __syncthreads();
  float* out = a.out + size_t(t) * d * C;
  for (int o = tid; o < d * C; o += blockDim.x) {
    const int k = o / C, c = o - k * C;
    float z = 0.f;
    for (int r = 0; r < R; ++r) z = fmaf(a.EF[k * R + r], sH[r * kVHs + c], z);
    out[o] = z;
  }
}

template <int L>
hipError_t launch_valu_l(const EdgeArgs& a, const float* x, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const size_t lds_edge = size_t(d * kVR + d * kVC + kVR + d + 16 + 1) * 4;
  const size_t lds_h = size_t(kVR) * kVHs * 4;
  const size_t lds = lds_edge > lds_h ? lds_edge : lds_h;
  auto k = k_cp_edge_valu<L>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(a.n_seg), dim3(256), lds, s>>>(a, x);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cp_edge_valu(const EdgeArgs& a, const float* x, hipStream_t s) {
  if (a.n_seg == 0) return hipSuccess;
  if (a.R < 1 || a.R > kVR || a.C < 1 || a.C > kVC || a.n_radial < 1 || a.n_radial > 16 || !x || !a.out ||
      !a.offsets || (a.E > 0 && (!a.perm || !a.gather || !a.edge_vec)))
    return hipErrorInvalidValue;
  switch (a.L) {
    case 2: return launch_valu_l<2>(a, x, s);
    case 3: return launch_valu_l<3>(a, x, s);
    case 4: return launch_valu_l<4>(a, x, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
