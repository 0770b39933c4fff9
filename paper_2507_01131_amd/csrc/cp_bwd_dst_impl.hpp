// Backward of the CP tensor-product layer with respect to the edge vectors,
// direct form (used for d > 32; d <= 32 takes the factored form in
// cp_bwd_sg_impl.hpp).
//
// With Gz = grad_out W^T and Gh_t = D^T Gz[t] (per destination node, [R, C]),
// the cotangent of g_e (eq. approximate, Sec. 3.1) is
//   dg_e[r] = sum_c Gh_t[r, c] (A^T x[s_e])[r, c] = sum_k A[k, r] P_e[k, r],
//   P_e = x[s_e] Gh_t^T   ([d, R], contraction over the C channels)
// and then  dv = dg * rho,  drho = dg * v,  dY = B dv,  dphi = Wrad drho,
//   grad r_e = J_Y(r_e)^T dY + (sum_q dphi_q phi'_q(|r_e|)) r_e/|r_e|.
//
// One workgroup per destination segment, one wave per 32-rank tile.  Each
// wave forms its Gh^T tiles once (MFMA, K = d) and keeps them in registers:
// in accumulator layout lane l holds Gh^T[ct*32 + acc_row(v, l/32)]
// [rt*32 + l%32], which is exactly the B operand of P_e^T = x[s_e] Gh^T when
// K-step (ct, v) contracts channel ct*32 + acc_row(v, half) in each
// half-wave.  The matching A operand, x[s_e][k][ct*32 + acc_row(v, half)],
// is four groups of four consecutive channels per lane, so it is loaded
// straight from global memory with float4 loads (no LDS staging), one
// (edge, channel tile) step ahead into alternating register buffers.  dg is
// then a 16-term dot product with A held in registers plus one cross-half
// add.  The channel-tile count NCT and k-tile count MT are compile-time.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace bwd_detail {

constexpr int kChunk = 16;  // edges per chunk

struct DstSmem {
  int Rp, off_b, off_v, off_rho, off_dg, off_y, off_phi, off_dy, off_dphi, off_j, off_idx, floats;
};

__host__ __device__ inline DstSmem dst_smem(int RT, int d, int n_radial) {
  DstSmem s{};
  s.Rp = RT * kTile;
  int o = 0;
  s.off_b = o;  // B [d][Rp] then Wrad [n_radial][Rp]
  o += (d + n_radial) * s.Rp;
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

template <typename TX>
__device__ __forceinline__ void load4(const TX* p, float* out);
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* out) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(p);
  out[0] = v[0];
  out[1] = v[1];
  out[2] = v[2];
  out[3] = v[3];
}
template <>
__device__ __forceinline__ void load4<uint16_t>(const uint16_t* p, float* out) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  out[0] = __uint_as_float(v.x << 16);
  out[1] = __uint_as_float(v.x & 0xffff0000u);
  out[2] = __uint_as_float(v.y << 16);
  out[3] = __uint_as_float(v.y & 0xffff0000u);
}

template <int MT, int RT, int NCT, typename TX>
__global__ __launch_bounds__(RT* kWave) void k_bwd_dst(BwdDstArgs a) {
  extern __shared__ float smem[];
  const DstSmem S = dst_smem(RT, a.d, a.n_radial);
  constexpr int Rp = RT * kTile;
  float* sB = smem + S.off_b;
  float* sWr = sB + a.d * Rp;
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
  const int r = rt * kTile + l32;
  const TX* __restrict__ x = static_cast<const TX*>(a.x);

  for (int i = tid; i < (d + nr) * Rp; i += blockDim.x) {
    const int k = i / Rp, rr = i - k * Rp;
    sB[i] = rr < R ? (k < d ? a.Bf[k * R + rr] : a.radial_w[(k - d) * R + rr]) : 0.f;
  }
  // factor A in registers, in P^T accumulator layout: Areg[kt][v] = A[kt*32 + acc_row(v,h)][r]
  float Areg[MT][16];
#pragma unroll
  for (int kt = 0; kt < MT; ++kt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int k = kt * kTile + acc_row(v, h);
      Areg[kt][v] = (k < d && r < R) ? a.A[k * R + r] : 0.f;
    }

  // Gh^T tiles: gh[ct] = Gz[seg]^T D restricted to (channel tile ct, rank tile rt)
  f32x16 gh[NCT];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    gh[ct] = f32x16{};
    const int cc = ct * kTile + l32;
    for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
      const int k = 2 * s2 + h;
      const float av = (k < d && cc < C) ? a.Gz[(size_t(seg) * d + k) * C + cc] : 0.f;
      const float bv = (k < d && r < R) ? a.D[k * R + r] : 0.f;
      gh[ct] = mfma32(av, bv, gh[ct]);
    }
  }

  // A operand of step (edge row `row`, channel tile ct): for k tile kt,
  // x[row][kt*32 + l32][ct*32 + 8q + 4h + i] -> xb[kt*16 + 4q + i].  Rows past
  // d are clamped (their P rows meet A = 0); channels past C are clamped
  // (they meet Gh = 0).
  auto load_step = [&](int row, int ct, float (&xb)[MT * 16]) {
#pragma unroll
    for (int kt = 0; kt < MT; ++kt) {
      const int kr = kt * kTile + l32 < d ? kt * kTile + l32 : d - 1;
      const TX* p = x + (size_t(row) * d + kr) * C;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c0 = ct * kTile + 8 * q + 4 * h;
        load4<TX>(p + (c0 < C ? c0 : C - 4), &xb[kt * 16 + 4 * q]);
      }
    }
  };

  for (int cb = e_begin; cb < e_end; cb += kChunk) {
    const int n = min(kChunk, e_end - cb);
    __syncthreads();
    // harmonics and Jacobian per (edge, order m) column; radial basis per
    // (edge, function); indices per edge
    for (int t = tid; t < n * (a.L + 1); t += blockDim.x) {
      const int e = t / (a.L + 1), m = t - e * (a.L + 1);
      const int eid = a.perm[cb + e];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float inv = 1.f / sqrtf(vx * vx + vy * vy + vz * vz);
      sh_unit_jacobian_column(a.L, m, vx * inv, vy * inv, vz * inv, inv, sY + e * d, sJ + e * 3 * d);
    }
    for (int t = tid; t < n * nr; t += blockDim.x) {
      const int e = t / nr, q = t - e * nr;
      const int eid = a.perm[cb + e];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      sPhi[t] = radial_phi(sqrtf(vx * vx + vy * vy + vz * vz), q, a.sigma);
    }
    for (int t = tid; t < n; t += blockDim.x) {
      const int eid = a.perm[cb + t];
      sEid[t] = eid;
      sIdx[t] = a.src[eid];
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

    // P_e^T tiles and dg, edges in pairs so that the buffer of every
    // (edge, ct) step is a compile-time choice; an odd last edge is paired
    // with a copy of itself whose result is dropped.
    float xb0[MT * 16], xb1[MT * 16];
    f32x16 p[MT];
    load_step(sIdx[0], 0, xb0);
    for (int e0 = 0; e0 < n; e0 += 2) {
      const int e1 = e0 + 1 < n ? e0 + 1 : e0;
      const int e2 = e0 + 2 < n ? e0 + 2 : e1;
#pragma unroll
      for (int half_e = 0; half_e < 2; ++half_e) {
        const int e = half_e ? e1 : e0;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          // the step index s decides the buffer: s & 1 (compile-time here)
          const int s = half_e * NCT + ct;
          // issue the loads of the next step
          {
            const bool last_ct = ct + 1 == NCT;
            const int nrow = last_ct ? sIdx[half_e ? e2 : e1] : sIdx[e];
            const int nct = last_ct ? 0 : ct + 1;
            if ((s + 1) & 1)
              load_step(nrow, nct, xb1);
            else
              load_step(nrow, nct, xb0);
          }
          __builtin_amdgcn_sched_barrier(0);
          if (ct == 0) {
#pragma unroll
            for (int kt = 0; kt < MT; ++kt) p[kt] = f32x16{};
          }
#pragma unroll
          for (int kt = 0; kt < MT; ++kt)
#pragma unroll
            for (int v = 0; v < 16; ++v) p[kt] = mfma32(s & 1 ? xb1[kt * 16 + v] : xb0[kt * 16 + v], gh[ct][v], p[kt]);
          __builtin_amdgcn_sched_barrier(0);
          if (ct + 1 == NCT && (half_e == 0 || e1 != e0)) {
            float part = 0.f;
#pragma unroll
            for (int kt = 0; kt < MT; ++kt)
#pragma unroll
              for (int v = 0; v < 16; ++v) part += Areg[kt][v] * p[kt][v];
            part += __shfl_xor(part, 32);
            if (h == 0) sDG[e * Rp + r] = part;
          }
        }
      }
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
      // each thread starts at its own rank so that a wave's LDS reads of the
      // factor rows (stride Rp) fall in distinct banks
      const float* fr = k < d ? sB + k * Rp : sWr + (k - d) * Rp;
      const float* vr = (k < d ? sV : sRho) + e * Rp;
      float s2 = 0.f;
      int rr = k % Rp;
      for (int j = 0; j < Rp; ++j) {
        s2 += fr[rr] * vr[rr];
        rr = rr + 1 == Rp ? 0 : rr + 1;
      }
      if (k < d)
        sDY[e * d + k] = s2;
      else
        sDPhi[e * nr + (k - d)] = s2;
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

template <int MT, int RT, int NCT, typename TX>
hipError_t launch_k(const BwdDstArgs& a, hipStream_t s) {
  const size_t lds = size_t(dst_smem(RT, a.d, a.n_radial).floats) * 4;
  auto k = k_bwd_dst<MT, RT, NCT, TX>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(a.n_seg), dim3(RT * kWave), lds, s>>>(a);
  return hipGetLastError();
}

template <int MT, typename TX>
hipError_t launch_mt(const BwdDstArgs& a, hipStream_t s) {
  const int rt = (a.R + kTile - 1) / kTile;
  const int nct = (a.C + kTile - 1) / kTile;
  const int NC = nct <= 2 ? 2 : (nct <= 4 ? 4 : 8);
#define TDN_BWD_CASE(RTV)                                   \
  case RTV:                                                 \
    if (NC == 2) return launch_k<MT, RTV, 2, TX>(a, s);     \
    if (NC == 4) return launch_k<MT, RTV, 4, TX>(a, s);     \
    return launch_k<MT, RTV, 8, TX>(a, s);
  switch (rt) {
    TDN_BWD_CASE(1)
    TDN_BWD_CASE(2)
    TDN_BWD_CASE(3)
    TDN_BWD_CASE(4)
    TDN_BWD_CASE(5)
    TDN_BWD_CASE(6)
    TDN_BWD_CASE(7)
    TDN_BWD_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef TDN_BWD_CASE
}

}  // namespace bwd_detail

}  // namespace tdn
