// Destination-side backward for d <= 32 through the factored form of dg.
//
// With Gz = grad_out W^T and Gh_t = D^T Gz[t], the cotangent of g_e
// (eq. approximate, Sec. 3.1) factors as
//   dg_e[r] = sum_{k,j} S_e[k, j] A[k, r] D[j, r],   S_e = x[s_e] Gz[t]^T
// (d x d, contraction over the C channels), so an edge costs d*d*C + d*d*R
// multiply-adds instead of R*d*C.  Then dv = dg * rho, drho = dg * v,
// dY = B dv, dphi = Wrad drho and
//   grad r_e = J_Y(r_e)^T dY + (sum_q dphi_q phi'_q(|r_e|)) r_e/|r_e|.
//
// One workgroup per destination segment, edges in chunks of 32:
//  * geometry: harmonics and their Jacobian per (edge, m) column, radial
//    basis per (edge, function);
//  * v = Y B and rho = Phi Wrad as small MFMA GEMMs (32 edges x 32 ranks per
//    tile);
//  * per edge (each wave takes whole edges, no barriers): S_e as one 32x32
//    MFMA tile with Gz[t] held in registers; its accumulator layout (lane l
//    holds S_e[acc_row(v, l/32)][l%32]) is the A operand of T_e = S_e^T A,
//    so S never leaves the registers; dg_e[r] = sum_j D[j, r] T_e[j, r] and
//    immediately dv, drho;
//  * dY = dV B^T and dphi = dRho Wrad^T as MFMA GEMMs (K = ranks), then the
//    edge-vector gradient per edge.
// fp32 features use 32x32x2 fp32 MFMA; bf16 features use 32x32x16 bf16 MFMA
// for S (x is bf16, Gz rounded to bf16) and T (S and A rounded to bf16),
// fp32 accumulation throughout.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace bwd_sg_detail {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxChunk = 32;  // edges per chunk: one 32-row MFMA tile
constexpr int kWaves = 4;

struct SgSmem {
  int Rp, bs, off_b, off_wr, off_a, off_d, off_v, off_rho, off_y, off_phi, off_dy, off_dphi, off_j, off_idx, floats;
};

// bf16: A is kept permuted as bf16 [2][2][Rp][8] (half the floats)
__host__ __device__ inline SgSmem sg_smem(int RT, int d, int n_radial, bool bf16, int kChunk) {
  SgSmem s{};
  s.Rp = RT * kTile;
  s.bs = s.Rp + 1;  // padded rows: row-wise operand reads across lanes hit distinct banks
  int o = 0;
  s.off_b = o;
  o += d * s.bs;
  s.off_wr = o;
  o += n_radial * s.bs;
  s.off_a = o;
  o += bf16 ? kTile * s.Rp / 2 : kTile * s.Rp;
  s.off_d = o;
  o += kTile * s.Rp;
  s.off_v = o;
  o += kChunk * s.bs;
  s.off_rho = o;
  o += kChunk * s.bs;
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

__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return uint32_t(__builtin_bit_cast(uint16_t, static_cast<__bf16>(lo))) |
         (uint32_t(__builtin_bit_cast(uint16_t, static_cast<__bf16>(hi))) << 16);
}

// Contraction row of K-step q (0, 1), half h, element i in the bf16 T = S^T A
// step: the rows lane half h holds in accumulator registers 8q .. 8q+7.
__host__ __device__ inline int t_row(int q, int h, int i) { return 16 * q + 8 * (i / 4) + 4 * h + (i % 4); }

// NCT: channel tiles (fp32: 32 channels per tile; bf16: 16 channels per
// K-step, NCT*2 K-steps)
template <int RT, int NCT, bool BF16>
__global__ __launch_bounds__(kWaves* kWave) void k_bwd_dst_sg(BwdDstArgs a, int kChunk) {
  extern __shared__ float smem[];
  const SgSmem S = sg_smem(RT, a.d, a.n_radial, BF16, kChunk);
  constexpr int Rp = RT * kTile;
  const int bs = S.bs;
  float* sB = smem + S.off_b;
  float* sWr = smem + S.off_wr;
  float* sA = smem + S.off_a;
  uint16_t* sAp = reinterpret_cast<uint16_t*>(smem + S.off_a);
  float* sD = smem + S.off_d;
  float* sV = smem + S.off_v;
  float* sRho = smem + S.off_rho;
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
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int d = a.d, C = a.C, nr = a.n_radial, R = a.R;

  for (int i = tid; i < d * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    sB[k * bs + r] = r < R ? a.Bf[k * R + r] : 0.f;
  }
  for (int i = tid; i < nr * Rp; i += blockDim.x) {
    const int q = i / Rp, r = i - q * Rp;
    sWr[q * bs + r] = r < R ? a.radial_w[q * R + r] : 0.f;
  }
  for (int i = tid; i < kTile * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    const bool ok = r < R && k < d;
    sD[i] = ok ? a.D[k * R + r] : 0.f;
    if constexpr (!BF16) sA[i] = ok ? a.A[k * R + r] : 0.f;
  }
  if constexpr (BF16) {
    // sAp[((q*2 + h)*Rp + r)*8 + i] = bf16(A[t_row(q, h, i)][r])
    for (int i = tid; i < 4 * Rp; i += blockDim.x) {
      const int qh = i / Rp, r = i - qh * Rp, q = qh >> 1, hh = qh & 1;
      uint32_t w[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int k0 = t_row(q, hh, 2 * p), k1 = t_row(q, hh, 2 * p + 1);
        const float v0 = (k0 < d && r < R) ? a.A[k0 * R + r] : 0.f;
        const float v1 = (k1 < d && r < R) ? a.A[k1 * R + r] : 0.f;
        w[p] = pack_bf16(v0, v1);
      }
      *reinterpret_cast<u32x4*>(sAp + size_t(i) * 8) = u32x4{w[0], w[1], w[2], w[3]};
    }
  }

  // Gz[seg] rows j = l32 as the B operand of S.
  //  fp32: gz[ct*16 + v] = Gz[j][ct*32 + acc_row(v, h)]   (permuted channel K-steps)
  //  bf16: gzb[s] = bf16(Gz[j][16s + 8h .. +7])            (16 channels per K-step)
  constexpr int NG = BF16 ? NCT * 2 * 4 : NCT * 16;  // registers
  uint32_t gzb[BF16 ? NCT * 2 : 1][4];
  float gz[BF16 ? 1 : NG];
  {
    const int jr = l32 < d ? l32 : d - 1;
    const bool jok = l32 < d;
    const float* p = a.Gz + (size_t(seg) * d + jr) * C;
    if constexpr (BF16) {
#pragma unroll
      for (int s2 = 0; s2 < NCT * 2; ++s2) {
        const int c0 = 16 * s2 + 8 * h;
        const bool cok = jok && c0 < C;
        const f32x4 v0 = *reinterpret_cast<const f32x4*>(p + (c0 < C ? c0 : C - 8));
        const f32x4 v1 = *reinterpret_cast<const f32x4*>(p + (c0 < C ? c0 : C - 8) + 4);
        gzb[s2][0] = cok ? pack_bf16(v0[0], v0[1]) : 0u;
        gzb[s2][1] = cok ? pack_bf16(v0[2], v0[3]) : 0u;
        gzb[s2][2] = cok ? pack_bf16(v1[0], v1[1]) : 0u;
        gzb[s2][3] = cok ? pack_bf16(v1[2], v1[3]) : 0u;
      }
    } else {
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c0 = ct * kTile + 8 * q + 4 * h;
          const bool cok = jok && c0 < C;
          const f32x4 v = *reinterpret_cast<const f32x4*>(p + (c0 < C ? c0 : C - 4));
#pragma unroll
          for (int i = 0; i < 4; ++i) gz[ct * 16 + 4 * q + i] = cok ? v[i] : 0.f;
        }
    }
  }

  // x[row] as the A operand of S (rows past d clamp: they meet zero rows of
  // Gz, A and D).  bf16: all channels, one 16-byte load per K-step of 16
  // channels; fp32: one 32-channel tile (four float4 loads) at a time.
  const int kr_ld = l32 < d ? l32 : d - 1;
  auto load_x_bf16 = [&](int row, u32x4 (&xb)[NCT * 2]) {
    const uint16_t* p = static_cast<const uint16_t*>(a.x) + (size_t(row) * d + kr_ld) * C;
#pragma unroll
    for (int s2 = 0; s2 < NCT * 2; ++s2) {
      const int c0 = 16 * s2 + 8 * h;
      xb[s2] = *reinterpret_cast<const u32x4*>(p + (c0 < C ? c0 : C - 8));
    }
  };
  auto load_x_tile = [&](int row, int ct, u32x4 (&xb)[4]) {
    const float* p = static_cast<const float*>(a.x) + (size_t(row) * d + kr_ld) * C;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c0 = ct * kTile + 8 * q + 4 * h;
      xb[q] = *reinterpret_cast<const u32x4*>(p + (c0 < C ? c0 : C - 4));
    }
  };

  for (int cb = e_begin; cb < e_end; cb += kChunk) {
    const int n = min(kChunk, e_end - cb);
    __syncthreads();
    // ---- geometry
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
    // ---- v = Y B, rho = Phi Wrad (rows: edges, columns: ranks)
    for (int item = wave; item < 2 * RT; item += kWaves) {
      const int rt = item >> 1;
      const bool is_v = (item & 1) == 0;
      const int K = is_v ? d : nr;
      const float* src = is_v ? sY : sPhi;
      const float* fac = is_v ? sB : sWr;
      f32x16 T = f32x16{};
      for (int s2 = 0; s2 < (K + 1) / 2; ++s2) {
        const int k = 2 * s2 + h;
        const float av = (l32 < n && k < K) ? src[l32 * K + k] : 0.f;
        const float bv = k < K ? fac[k * bs + rt * kTile + l32] : 0.f;
        T = mfma32(av, bv, T);
      }
      float* dst = is_v ? sV : sRho;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int e = acc_row(v, h);
        if (e < n) dst[e * bs + rt * kTile + l32] = T[v];
      }
    }
    __syncthreads();
    // ---- per edge: S_e, T_e, dg -> dv, drho (each wave takes whole edges)
    // T_e = S_e^T A and dg from the S accumulators
    auto finish_edge = [&](int e, const f32x16& Sacc) {
      bf16x8 sa[2];
      if constexpr (BF16) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
          sa[q] = __builtin_bit_cast(bf16x8, u32x4{pack_bf16(Sacc[8 * q + 0], Sacc[8 * q + 1]),
                                                   pack_bf16(Sacc[8 * q + 2], Sacc[8 * q + 3]),
                                                   pack_bf16(Sacc[8 * q + 4], Sacc[8 * q + 5]),
                                                   pack_bf16(Sacc[8 * q + 6], Sacc[8 * q + 7])});
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int r = rt * kTile + l32;
        f32x16 T = f32x16{};
        if constexpr (BF16) {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const u32x4 bv = *reinterpret_cast<const u32x4*>(sAp + (size_t(q * 2 + h) * Rp + r) * 8);
            T = mfma32_bf16(sa[q], __builtin_bit_cast(bf16x8, bv), T);
          }
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) T = mfma32(Sacc[v], sA[acc_row(v, h) * Rp + r], T);
        }
        float part = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) part += sD[acc_row(v, h) * Rp + r] * T[v];
        part += __shfl_xor(part, 32);
        if (h == 0) {
          const float dv = part * sRho[e * bs + r], drho = part * sV[e * bs + r];
          sV[e * bs + r] = dv;
          sRho[e * bs + r] = drho;
        }
      }
    };
    if constexpr (BF16) {
      // whole-edge operands, alternating buffers one edge ahead
      u32x4 xb0[NCT * 2], xb1[NCT * 2];
      auto s_of = [&](const u32x4 (&xb)[NCT * 2]) {
        f32x16 Sacc = f32x16{};
#pragma unroll
        for (int s2 = 0; s2 < NCT * 2; ++s2)
          Sacc = mfma32_bf16(__builtin_bit_cast(bf16x8, xb[s2]),
                             __builtin_bit_cast(bf16x8, u32x4{gzb[s2][0], gzb[s2][1], gzb[s2][2], gzb[s2][3]}),
                             Sacc);
        return Sacc;
      };
      int e = wave;
      if (e < n) load_x_bf16(sIdx[e], xb0);
      for (; e < n; e += 2 * kWaves) {
        const int e1 = e + kWaves;
        const int e2 = e + 2 * kWaves;
        load_x_bf16(sIdx[e1 < n ? e1 : e], xb1);
        __builtin_amdgcn_sched_barrier(0);
        finish_edge(e, s_of(xb0));
        __builtin_amdgcn_sched_barrier(0);
        if (e1 < n) {
          load_x_bf16(sIdx[e2 < n ? e2 : e1], xb0);
          __builtin_amdgcn_sched_barrier(0);
          finish_edge(e1, s_of(xb1));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    } else {
      // one 32-channel tile per step, alternating buffers one step ahead; NCT
      // is even, so every edge starts on buffer 0
      u32x4 xb0[4], xb1[4];
      int e = wave;
      if (e < n) load_x_tile(sIdx[e], 0, xb0);
      for (; e < n; e += kWaves) {
        const int en = e + kWaves < n ? e + kWaves : e;  // last edge reloads itself; unused
        f32x16 Sacc = f32x16{};
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          if (ct + 1 < NCT) {
            if ((ct + 1) & 1)
              load_x_tile(sIdx[e], ct + 1, xb1);
            else
              load_x_tile(sIdx[e], ct + 1, xb0);
          } else {
            load_x_tile(sIdx[en], 0, xb0);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              Sacc = mfma32(__builtin_bit_cast(float, ct & 1 ? xb1[q][i] : xb0[q][i]), gz[ct * 16 + 4 * q + i], Sacc);
          __builtin_amdgcn_sched_barrier(0);
        }
        finish_edge(e, Sacc);
      }
    }
    __syncthreads();
    // ---- dY = dV B^T (k < d), dphi = dRho Wrad^T (q < nr); K = ranks
    for (int item = wave; item < 2; item += kWaves) {
      const bool is_y = item == 0;
      const int K2 = is_y ? d : nr;
      const float* src = is_y ? sV : sRho;
      const float* fac = is_y ? sB : sWr;
      f32x16 T = f32x16{};
      for (int s2 = 0; s2 < Rp / 2; ++s2) {
        const int r = 2 * s2 + h;
        const float av = l32 < n ? src[l32 * bs + r] : 0.f;
        const float bv = l32 < K2 ? fac[l32 * bs + r] : 0.f;
        T = mfma32(av, bv, T);
      }
      float* dst = is_y ? sDY : sDPhi;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int ee = acc_row(v, h);
        if (ee < n && l32 < K2) dst[ee * K2 + l32] = T[v];
      }
    }
    __syncthreads();
    for (int t = tid; t < n; t += blockDim.x) {
      const int eid = sEid[t];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float rn = sqrtf(vx * vx + vy * vy + vz * vz);
      float gx = 0.f, gy = 0.f, gzv = 0.f;
      for (int k = 0; k < d; ++k) {
        const float dy = sDY[t * d + k];
        gx += dy * sJ[t * 3 * d + 3 * k];
        gy += dy * sJ[t * 3 * d + 3 * k + 1];
        gzv += dy * sJ[t * 3 * d + 3 * k + 2];
      }
      float dr = 0.f;
      for (int q = 0; q < nr; ++q) {
        const float u = (rn - float(q) * a.sigma) / a.sigma;
        dr += sDPhi[t * nr + q] * (-u / a.sigma) * sPhi[t * nr + q];
      }
      const float inv = 1.f / rn;
      a.grad_vec[3 * eid] = gx + dr * vx * inv;
      a.grad_vec[3 * eid + 1] = gy + dr * vy * inv;
      a.grad_vec[3 * eid + 2] = gzv + dr * vz * inv;
    }
    if (a.drho) {  // drho rows for the radial-weight gradient (sRho is rewritten after the next barrier)
      for (int i = tid; i < n * R; i += blockDim.x) {
        const int t = i / R, r = i - t * R;
        a.drho[size_t(sEid[t]) * R + r] = sRho[t * bs + r];
      }
    }
  }
}

template <int RT, int NCT, bool BF16>
hipError_t launch_sg(const BwdDstArgs& a, hipStream_t s) {
  // the largest chunk (<= 32 edges) whose layout fits the 160 KB of LDS
  int chunk = kMaxChunk;
  while (chunk > 4 && sg_smem(RT, a.d, a.n_radial, BF16, chunk).floats * 4 > 160 * 1024) chunk >>= 1;
  const size_t lds = size_t(sg_smem(RT, a.d, a.n_radial, BF16, chunk).floats) * 4;
  auto k = k_bwd_dst_sg<RT, NCT, BF16>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(a.n_seg), dim3(kWaves * kWave), lds, s>>>(a, chunk);
  return hipGetLastError();
}

template <bool BF16>
hipError_t launch_sg_any(const BwdDstArgs& a, hipStream_t s) {
  const int rt = (a.R + kTile - 1) / kTile;
  const int nct = (a.C + kTile - 1) / kTile;
  const int NC = nct <= 2 ? 2 : (nct <= 4 ? 4 : 8);
#define TDN_SG_CASE(RTV)                                     \
  case RTV:                                                  \
    if (NC == 2) return launch_sg<RTV, 2, BF16>(a, s);       \
    if (NC == 4) return launch_sg<RTV, 4, BF16>(a, s);       \
    return launch_sg<RTV, 8, BF16>(a, s);
  switch (rt) {
    TDN_SG_CASE(1)
    TDN_SG_CASE(2)
    TDN_SG_CASE(3)
    TDN_SG_CASE(4)
    TDN_SG_CASE(5)
    TDN_SG_CASE(6)
    TDN_SG_CASE(7)
    TDN_SG_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef TDN_SG_CASE
}

}  // namespace bwd_sg_detail

}  // namespace tdn
