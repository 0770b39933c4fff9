// The CP tensor-product edge pass as one Khatri-Rao GEMM per segment.
//
// For a destination node t with incoming edges e (eq. approximate of
// Sec. 3.1 per channel, radial weight on the rank index):
//   H_t[r, c] = sum_e g_e[r] sum_k A[k, r] x[s_e][k, c]
//             = (K_t^T X_t)[r, c],  K_t[(e,k), r] = g_e[r] A[k, r],
//                                    X_t[(e,k), c] = x[s_e][k, c]
// so the projection A^T x, the Hadamard product with g_e = (B^T Y_e)*rho_e
// and the sum over the segment are a single fp32 MFMA contraction of length
// n_t * d whose partial sums never leave the accumulators (no atomics, fixed
// order).  The output factor is applied once per node, Z_t = D H_t, because D
// commutes with the sum over edges; the shared channel mix W (Sec. 3.2) is a
// separate node GEMM.
//
// The same kernel computes grad_x on the source-sorted graph:
//   grad_x[s] = A sum_{e: s_e = s} diag(g_e) D^T Gz[t_e],  Gz = grad_out W^T,
// i.e. K uses D, the epilogue uses A and the gathered rows are Gz[t_e].
//
// Work decomposition: one workgroup per (segment, group of up to four
// 32-channel tiles); wave w owns channel tile w and all R rank rows, so its
// accumulators are RT = ceil(R/32) MFMA tiles of 32x32.  Per chunk of edges
// the block evaluates the harmonics and radial basis (one lane per edge), then
// g_e[r] for every rank (all lanes), into LDS.  The MFMA loop then walks the
// chunk edge by edge: each edge's contraction over its d feature rows is
// padded to an even length (a zero row when d is odd), so one 32x32x2 K-step
// always covers rows 2j and 2j+1 of one edge; g_e is held in registers for the
// edge, the K operand is g_e[r] * KF[k][r] with KF resident in LDS, and the B
// operand x[s_e][k][c] comes straight from global memory (each half-wave
// reads one contiguous 128-byte row slice), loaded one edge ahead.
//
// The degree L is a template parameter so that the per-edge K-step count
// DH = ceil(d/2) and the harmonic recurrences are compile-time constants.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace edge_detail {

constexpr int kMaxWavesPerBlock = 4;

struct EdgeSmem {
  int Rp, kstride, estride, off_k, off_be, off_g, off_y, off_phi, off_idx, floats;
};

__host__ __device__ inline EdgeSmem edge_smem(int RT, int d, int n_radial, int chunk) {
  EdgeSmem s{};
  const int dpad = d + (d & 1);
  s.Rp = RT * kTile;
  s.kstride = s.Rp + 32;  // rows 2j and 2j+1 land 32 banks apart
  s.estride = s.Rp + 1;   // the epilogue reads a column across 32 rows
  int o = 0;
  s.off_k = o;
  o += dpad * s.kstride;
  s.off_be = o;
  const int be_b = (d + n_radial) * s.Rp, be_e = d * s.estride;
  o += be_b > be_e ? be_b : be_e;
  s.off_g = o;
  o += chunk * s.Rp;
  s.off_y = o;
  o += chunk * d;
  s.off_phi = o;
  o += chunk * n_radial;
  s.off_idx = o;
  o += chunk;
  s.floats = o;
  return s;
}

// Stage a [rows_src, R] factor into LDS rows of `stride` floats; zero beyond
// R and for rows rows_src..rows_dst-1.
__device__ inline void stage_factor(float* dst, const float* __restrict__ src, int rows_src, int rows_dst, int R,
                                    int Rp, int stride) {
  for (int i = threadIdx.x; i < rows_dst * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    dst[k * stride + r] = (r < R && k < rows_src) ? src[k * R + r] : 0.f;
  }
}

// Two waves per SIMD when the register-resident K factor fits beside the
// accumulators; one otherwise (large R at high L), where spilling would cost
// more than the lost occupancy.
template <int L, int RT>
constexpr int edge_waves_per_eu() {
  return ((L + 1) * (L + 1) + 1) / 2 * RT <= 64 ? 2 : 1;
}

template <int L, int RT, typename TF>
__global__ __launch_bounds__(kMaxWavesPerBlock* kWave) __attribute__((amdgpu_waves_per_eu(edge_waves_per_eu<L, RT>())))
void k_cp_edge(EdgeArgs a, int n_cgrp, int waves, int chunk) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DH = (d + 1) / 2;  // K-steps per edge
  constexpr int Rp = RT * kTile;
  extern __shared__ float smem[];
  const EdgeSmem S = edge_smem(RT, d, a.n_radial, chunk);
  float* sK = smem + S.off_k;
  float* sBE = smem + S.off_be;
  float* sG = smem + S.off_g;
  float* sY = smem + S.off_y;
  float* sPhi = smem + S.off_phi;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);

  const int total = a.n_seg * n_cgrp;
  const int logical = xcd_remap(blockIdx.x, total);
  const int seg = logical / n_cgrp, cgrp = logical - seg * n_cgrp;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int h = lane >> 5, l32 = lane & 31;
  const int C = a.C, nr = a.n_radial;
  const int c = (cgrp * waves + wave) * kTile + l32;
  const bool cvalid = c < C;
  const TF* __restrict__ feat = static_cast<const TF*>(a.feat);

  stage_factor(sK, a.KF, d, d + (d & 1), a.R, Rp, S.kstride);
  stage_factor(sBE, a.Bf, d, d, a.R, Rp, Rp);
  stage_factor(sBE + d * Rp, a.radial_w, nr, nr, a.R, Rp, Rp);

  f32x16 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x16{};

  // When it fits (DH*RT <= 64 values per lane) the K factor of this lane,
  // KF[2j + h][rt*32 + l32], lives in registers for the whole segment, so
  // the MFMA loop touches LDS only for g_e.
  constexpr bool kRegK = DH * RT <= 64;
  float kreg[kRegK ? DH : 1][kRegK ? RT : 1];
  const float* kr = sK + h * S.kstride + l32;
  if constexpr (kRegK) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < DH; ++j)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) kreg[j][rt] = kr[2 * j * S.kstride + rt * kTile];
  }

  // B operand of K-step j of one edge: x[row][2j + h][c].  The loads are
  // unconditional with clamped addresses and no select on the value, so
  // nothing forces a wait before the operand is used one edge later: the pad
  // row (2j + h == d) meets an all-zero K row in LDS, and a lane with c >= C
  // only feeds result column c, which is never stored.
  const int c_ld = cvalid ? c : C - 1;
  auto load_edge = [&](int row, float (&b)[DH]) {
    const TF* p = feat + size_t(row) * d * C + c_ld;
#pragma unroll
    for (int j = 0; j < DH; ++j) {
      const int k = 2 * j + h < d ? 2 * j + h : d - 1;
      b[j] = load_feat<TF>(p + size_t(k) * C);
    }
  };

  const int e_begin = a.offsets[seg], e_end = a.offsets[seg + 1];
  for (int cb = e_begin; cb < e_end; cb += chunk) {
    const int n = min(chunk, e_end - cb);
    __syncthreads();  // factors staged / previous chunk consumed
    // harmonics: one thread per (edge, order m) column; radial basis: one
    // thread per (edge, function); gathered row: one thread per edge
    for (int t = tid; t < n * (L + 1); t += blockDim.x) {
      const int e = t / (L + 1), m = t - e * (L + 1);
      const int eid = a.perm[cb + e];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float inv = 1.f / sqrtf(vx * vx + vy * vy + vz * vz);
      sh_unit_column(L, m, vx * inv, vy * inv, vz * inv, sY + e * d);
    }
    for (int t = tid; t < n * nr; t += blockDim.x) {
      const int e = t / nr, q = t - e * nr;
      const int eid = a.perm[cb + e];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      sPhi[t] = radial_phi(sqrtf(vx * vx + vy * vy + vz * vz), q, a.sigma);
    }
    for (int t = tid; t < n; t += blockDim.x) sIdx[t] = a.gather[a.perm[cb + t]];
    __syncthreads();
    // g = (Y B) * (Phi Wrad) for the chunk's edges (rows) and all ranks
    // (columns): two small MFMA GEMMs per 32x32 tile, one rank tile per wave.
    const int n_et = (n + kTile - 1) / kTile;
    for (int item = wave; item < n_et * RT; item += waves) {
      const int et = item / RT, rt = item - et * RT;
      const int er = et * kTile + l32;  // this lane's edge row
      const bool row_ok = er < n;
      f32x16 T = f32x16{};
#pragma unroll 1
      for (int s2 = 0; s2 < (nr + 1) / 2; ++s2) {
        const int q = 2 * s2 + h;
        const float av = (row_ok && q < nr) ? sPhi[er * nr + q] : 0.f;
        const float bv = q < nr ? sBE[(d + q) * Rp + rt * kTile + l32] : 0.f;
        T = mfma32(av, bv, T);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int e = et * kTile + acc_row(v, h);
        if (e < n) sG[e * Rp + rt * kTile + l32] = T[v];
      }
      T = f32x16{};
#pragma unroll 1
      for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
        const int k = 2 * s2 + h;
        const float av = (row_ok && k < d) ? sY[er * d + k] : 0.f;
        const float bv = k < d ? sBE[k * Rp + rt * kTile + l32] : 0.f;
        T = mfma32(av, bv, T);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int e = et * kTile + acc_row(v, h);
        if (e < n) sG[e * Rp + rt * kTile + l32] *= T[v];
      }
    }
    __syncthreads();

    // Two operand buffers used alternately: the loads for edge e+1 are issued
    // before the MFMAs of edge e, and the scheduling barriers keep the
    // compiler from sinking them next to their use.
    auto edge_mfma = [&](int e, const float (&b)[DH]) {
      float g[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) g[rt] = sG[e * Rp + rt * kTile + l32];
#pragma unroll
      for (int j = 0; j < DH; ++j) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          float kv;
          if constexpr (kRegK)
            kv = kreg[j][rt];
          else
            kv = kr[2 * j * S.kstride + rt * kTile];
          acc[rt] = mfma32(g[rt] * kv, b[j], acc[rt]);
        }
      }
    };
    float b0[DH], b1[DH];
    load_edge(sIdx[0], b0);
    int e = 0;
    for (; e + 1 < n; e += 2) {
      load_edge(sIdx[e + 1], b1);
      __builtin_amdgcn_sched_barrier(0);
      edge_mfma(e, b0);
      __builtin_amdgcn_sched_barrier(0);
      load_edge(sIdx[e + 2 < n ? e + 2 : e + 1], b0);  // the last pair reloads; unused
      __builtin_amdgcn_sched_barrier(0);
      edge_mfma(e + 1, b1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (e < n) edge_mfma(e, b0);
  }

  // Epilogue: out[seg][m][c] = sum_r EF[m][r] H[r][c].  The contraction over r
  // pairs accumulator register v of the two half-waves: lanes 0-31 contribute
  // rank rt*32 + acc_row(v,0), lanes 32-63 rank rt*32 + acc_row(v,1), which is
  // exactly the B-operand layout, so H never leaves the registers.
  __syncthreads();
  stage_factor(sBE, a.EF, d, d, a.R, Rp, S.estride);
  __syncthreads();
  constexpr int MT = (d + kTile - 1) / kTile;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    f32x16 z = f32x16{};
    const int row = mt * kTile + l32;
    const float* er = sBE + row * S.estride;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float av = row < d ? er[rt * kTile + acc_row(v, h)] : 0.f;
        z = mfma32(av, acc[rt][v], z);
      }
    }
    if (cvalid) {
      float* o = a.out + size_t(seg) * d * C + c;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = mt * kTile + acc_row(v, h);
        if (m < d) o[size_t(m) * C] = z[v];
      }
    }
  }
}

template <int L, int RT>
hipError_t launch_l_rt(const EdgeArgs& a, bool bf16, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const int ntiles = (a.C + kTile - 1) / kTile;
  const int waves = ntiles < kMaxWavesPerBlock ? ntiles : kMaxWavesPerBlock;
  const int n_cgrp = (ntiles + waves - 1) / waves;
  // largest edge chunk (<= 64) that keeps LDS within 80 KB (two blocks per
  // CU), at least 8: typical in-degrees then need a single chunk per segment
  int chunk = 64;
  while (chunk > 8 && edge_smem(RT, d, a.n_radial, chunk).floats * 4 > 80 * 1024) chunk >>= 1;
  const size_t lds = size_t(edge_smem(RT, d, a.n_radial, chunk).floats) * 4;
  const int total = a.n_seg * n_cgrp;
  if (total == 0) return hipSuccess;
  if (bf16) {
    auto k = k_cp_edge<L, RT, uint16_t>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(total), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  } else {
    auto k = k_cp_edge<L, RT, float>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(total), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  }
  return hipGetLastError();
}

template <int L>
hipError_t launch_cp_edge_l(const EdgeArgs& a, bool bf16, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt<L, 1>(a, bf16, s);
    case 2: return launch_l_rt<L, 2>(a, bf16, s);
    case 3: return launch_l_rt<L, 3>(a, bf16, s);
    case 4: return launch_l_rt<L, 4>(a, bf16, s);
    case 5: return launch_l_rt<L, 5>(a, bf16, s);
    case 6: return launch_l_rt<L, 6>(a, bf16, s);
    case 7: return launch_l_rt<L, 7>(a, bf16, s);
    case 8: return launch_l_rt<L, 8>(a, bf16, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace edge_detail

}  // namespace tdn
