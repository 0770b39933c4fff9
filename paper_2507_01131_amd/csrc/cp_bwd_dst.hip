// Backward of the CP tensor-product layer with respect to the edge vectors.
//
// With Gz = grad_out W^T and Gh_t = D^T Gz[t] (per destination node, [R, C]),
// the cotangent of g_e (eq. approximate, Sec. 3.1) is
//   dg_e[r] = sum_c Gh_t[r, c] (A^T x[s_e])[r, c] = sum_k A[k, r] P_e[k, r],
//   P_e = x[s_e] Gh_t^T   ([d, R], contraction over the C channels)
// and then  dv = dg * rho,  drho = dg * v,  dY = B dv,  dphi = Wrad drho,
//   grad r_e = J_Y(r_e)^T dY + (sum_q dphi_q phi'_q(|r_e|)) r_e/|r_e|.
//
// One workgroup per destination segment, one wave per 32-rank tile.  Each
// wave first forms its Gh^T tiles with MFMA (K = d) and keeps them in
// registers: in accumulator layout lane l holds Gh^T[ct*32 + acc_row(v, l/32)]
// [rt*32 + l%32], which is exactly the B operand of P_e^T = x_e Gh^T when
// K-step (ct, v) contracts channel ct*32 + acc_row(v, half) in each half-wave.
// x[s_e] is staged in LDS per edge (padded rows) for the A operand; dg is a
// 16-term dot product per lane with the factor A held in registers, plus one
// cross-half add.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

constexpr int kMaxCT = 8;   // channel tiles held in registers (C <= 256)
constexpr int kMaxMT = 2;   // k tiles (d <= 64)
constexpr int kChunk = 8;   // edges per chunk

struct DstSmem {
  int Rp, xs, off_b, off_dx, off_v, off_rho, off_dg, off_y, off_phi, off_dy, off_dphi, off_j, off_idx, floats;
};

__host__ __device__ inline DstSmem dst_smem(int RT, int d, int n_radial, int C) {
  DstSmem s{};
  s.Rp = RT * kTile;
  s.xs = C + 1;
  int o = 0;
  s.off_b = o;          // B [d][Rp] then Wrad [n_radial][Rp]
  o += (d + n_radial) * s.Rp;
  s.off_dx = o;         // D [d][Rp] during the Gh phase, then x_e [d][C+1]
  const int dsz = d * s.Rp, xsz = d * s.xs;
  o += dsz > xsz ? dsz : xsz;
  s.off_v = o;
  o += kChunk * s.Rp;
  s.off_rho = o;
  o += kChunk * s.Rp;
  s.off_dg = o;
  o += kChunk * s.Rp;
  s.off_y = o;
  o += kChunk * d;
  s.off_phi = o;
  o += kChunk * n_radial;
  s.off_dy = o;
  o += kChunk * d;
  s.off_dphi = o;
  o += kChunk * n_radial;
  s.off_j = o;
  o += kChunk * 3 * d;
  s.off_idx = o;
  o += 2 * kChunk;
  s.floats = o;
  return s;
}

template <int RT, typename TX>
__global__ __launch_bounds__(512) void k_bwd_dst(BwdDstArgs a) {
  extern __shared__ float smem[];
  const DstSmem S = dst_smem(RT, a.d, a.n_radial, a.C);
  constexpr int Rp = RT * kTile;
  float* sB = smem + S.off_b;
  float* sWr = sB + a.d * Rp;
  float* sDX = smem + S.off_dx;
  float* sV = smem + S.off_v;
  float* sRho = smem + S.off_rho;
  float* sDG = smem + S.off_dg;
  float* sY = smem + S.off_y;
  float* sPhi = smem + S.off_phi;
  float* sDY = smem + S.off_dy;
  float* sDPhi = smem + S.off_dphi;
  float* sJ = smem + S.off_j;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);
  int* sEid = sIdx + kChunk;

  const int seg = xcd_remap(blockIdx.x, a.n_seg);
  const int e_begin = a.offsets[seg], e_end = a.offsets[seg + 1];
  if (e_begin == e_end) return;
  const int tid = threadIdx.x, lane = tid & 63, rt = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int d = a.d, C = a.C, nr = a.n_radial, R = a.R;
  const int nct = (C + kTile - 1) / kTile, MT = (d + kTile - 1) / kTile;
  const int r = rt * kTile + l32;
  const TX* __restrict__ x = static_cast<const TX*>(a.x);

  for (int i = tid; i < (d + nr) * Rp; i += blockDim.x) {
    const int k = i / Rp, rr = i - k * Rp;
    sB[i] = rr < R ? (k < d ? a.Bf[k * R + rr] : a.radial_w[(k - d) * R + rr]) : 0.f;
  }
  for (int i = tid; i < d * Rp; i += blockDim.x) {
    const int k = i / Rp, rr = i - k * Rp;
    sDX[i] = rr < R ? a.D[k * R + rr] : 0.f;
  }
  // factor A in registers, in P^T accumulator layout: Areg[kt][v] = A[kt*32 + acc_row(v,h)][r]
  float Areg[kMaxMT][16];
#pragma unroll
  for (int kt = 0; kt < kMaxMT; ++kt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int k = kt * kTile + acc_row(v, h);
      Areg[kt][v] = (kt < MT && k < d && r < R) ? a.A[k * R + r] : 0.f;
    }
  __syncthreads();

  // Gh^T tiles: gh[ct] = Gz[seg]^T D restricted to (channel tile ct, rank tile rt)
  f32x16 gh[kMaxCT];
#pragma unroll
  for (int ct = 0; ct < kMaxCT; ++ct) {
    gh[ct] = f32x16{};
    if (ct < nct) {
      const int cc = ct * kTile + l32;
      for (int s = 0; s < (d + 1) / 2; ++s) {
        const int k = 2 * s + h;
        const float av = (k < d && cc < C) ? a.Gz[(size_t(seg) * d + k) * C + cc] : 0.f;
        const float bv = k < d ? sDX[k * Rp + r] : 0.f;
        gh[ct] = mfma32(av, bv, gh[ct]);
      }
    }
  }

  for (int cb = e_begin; cb < e_end; cb += kChunk) {
    const int n = min(kChunk, e_end - cb);
    __syncthreads();
    if (tid < n) {
      const int eid = a.perm[cb + tid];
      sEid[tid] = eid;
      sIdx[tid] = a.src[eid];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float rn = sqrtf(vx * vx + vy * vy + vz * vz);
      const float inv = 1.f / rn;
      sh_unit_jacobian(a.L, vx * inv, vy * inv, vz * inv, inv, sY + tid * d, sJ + tid * 3 * d);
      for (int q = 0; q < nr; ++q) sPhi[tid * nr + q] = radial_phi(rn, q, a.sigma);
    }
    __syncthreads();
    for (int i = tid; i < n * Rp; i += blockDim.x) {
      const int e = i / Rp, rr = i - e * Rp;
      float v = 0.f, rho = 0.f;
      for (int k = 0; k < d; ++k) v += sB[k * Rp + rr] * sY[e * d + k];
      for (int q = 0; q < nr; ++q) rho += sWr[q * Rp + rr] * sPhi[e * nr + q];
      sV[i] = v;
      sRho[i] = rho;
    }
    for (int j = 0; j < n; ++j) {
      __syncthreads();  // previous x_e consumed (and the D staging on the first edge)
      const size_t base = size_t(sIdx[j]) * d * C;
      for (int i = tid; i < d * C; i += blockDim.x) {
        const int k = i / C, cc = i - k * C;
        sDX[k * S.xs + cc] = load_feat<TX>(x + base + i);
      }
      __syncthreads();
      float part = 0.f;
#pragma unroll
      for (int kt = 0; kt < kMaxMT; ++kt) {
        if (kt < MT) {
          f32x16 p = f32x16{};
          const int krow = kt * kTile + l32;
          const float* xr = sDX + krow * S.xs;
#pragma unroll
          for (int ct = 0; ct < kMaxCT; ++ct) {
            if (ct < nct) {
#pragma unroll
              for (int v = 0; v < 16; ++v) {
                const int cc = ct * kTile + acc_row(v, h);
                const float av = (krow < d && cc < C) ? xr[cc] : 0.f;
                p = mfma32(av, gh[ct][v], p);
              }
            }
          }
#pragma unroll
          for (int v = 0; v < 16; ++v) part += Areg[kt][v] * p[v];
        }
      }
      part += __shfl_xor(part, 32);
      if (h == 0) sDG[j * Rp + r] = part;
    }
    __syncthreads();
    for (int i = tid; i < n * Rp; i += blockDim.x) {
      const float dg = sDG[i];
      const float dv = dg * sRho[i], drho = dg * sV[i];
      sV[i] = dv;
      sRho[i] = drho;
    }
    __syncthreads();
    for (int i = tid; i < n * (d + nr); i += blockDim.x) {
      const int e = i / (d + nr), k = i - e * (d + nr);
      float s = 0.f;
      if (k < d) {
        for (int rr = 0; rr < Rp; ++rr) s += sB[k * Rp + rr] * sV[e * Rp + rr];
        sDY[e * d + k] = s;
      } else {
        const int q = k - d;
        for (int rr = 0; rr < Rp; ++rr) s += sWr[q * Rp + rr] * sRho[e * Rp + rr];
        sDPhi[e * nr + q] = s;
      }
    }
    __syncthreads();
    if (tid < n) {
      const int eid = sEid[tid];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float rn = sqrtf(vx * vx + vy * vy + vz * vz);
      float gx = 0.f, gy = 0.f, gz = 0.f;
      for (int k = 0; k < d; ++k) {
        const float dy = sDY[tid * d + k];
        gx += dy * sJ[tid * 3 * d + 3 * k];
        gy += dy * sJ[tid * 3 * d + 3 * k + 1];
        gz += dy * sJ[tid * 3 * d + 3 * k + 2];
      }
      float dr = 0.f;
      for (int q = 0; q < nr; ++q) {
        const float t = (rn - float(q) * a.sigma) / a.sigma;
        dr += sDPhi[tid * nr + q] * (-t / a.sigma) * sPhi[tid * nr + q];
      }
      const float inv = 1.f / rn;
      a.grad_vec[3 * eid] = gx + dr * vx * inv;
      a.grad_vec[3 * eid + 1] = gy + dr * vy * inv;
      a.grad_vec[3 * eid + 2] = gz + dr * vz * inv;
    }
  }
}

template <int RT>
hipError_t launch_rt(const BwdDstArgs& a, bool bf16, hipStream_t s) {
  const size_t lds = size_t(dst_smem(RT, a.d, a.n_radial, a.C).floats) * 4;
  if (a.n_seg == 0) return hipSuccess;
  if (bf16) {
    auto k = k_bwd_dst<RT, uint16_t>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(a.n_seg), dim3(RT * kWave), lds, s>>>(a);
  } else {
    auto k = k_bwd_dst<RT, float>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(a.n_seg), dim3(RT * kWave), lds, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

size_t bwd_dst_lds_bytes(int R, int d, int n_radial, int C) {
  return size_t(dst_smem((R + kTile - 1) / kTile, d, n_radial, C).floats) * 4;
}

hipError_t launch_bwd_dst(const BwdDstArgs& a, bool x_bf16, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_rt<1>(a, x_bf16, s);
    case 2: return launch_rt<2>(a, x_bf16, s);
    case 3: return launch_rt<3>(a, x_bf16, s);
    case 4: return launch_rt<4>(a, x_bf16, s);
    case 5: return launch_rt<5>(a, x_bf16, s);
    case 6: return launch_rt<6>(a, x_bf16, s);
    case 7: return launch_rt<7>(a, x_bf16, s);
    case 8: return launch_rt<8>(a, x_bf16, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
