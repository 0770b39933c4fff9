// The edge pass for bfloat16 node features: the same Khatri-Rao contraction
// per destination segment as cp_edge_impl.hpp,
//   H_t[r, c] = sum_e sum_k (g_e[r] KF[k, r]) x[s_e][k, c],
// on bf16 MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulation).  The K operand
// g_e[r] KF[k, r] is formed in fp32 and rounded to bf16 once; x is already
// bf16.  A bf16 32x32x16 step wants eight consecutive contraction rows per
// lane, so x arrives transposed as xT[n][c][k] (k padded to 32 or 64 with
// zeros, launch_feature_layout with one part): then one lane's operand is a
// single 16-byte load.  Each wave owns
// two 32-channel tiles so that every K operand built in registers feeds two
// MFMAs.  The per-node output factor runs in fp32 as in the fp32 kernel.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace edge_bf16_detail {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

constexpr int kWavesMax = 4;
// channel tiles per wave: two while the accumulators fit (R <= 128)
template <int RT>
constexpr int ctw() {
  return RT <= 4 ? 2 : 1;
}

struct Bf16Smem {
  int Rp, kstride, estride, off_k, off_be, off_g, off_y, off_phi, off_idx, floats;
};

__host__ __device__ inline Bf16Smem bf16_smem(int RT, int d, int dp, int n_radial, int chunk) {
  Bf16Smem s{};
  s.Rp = RT * kTile;
  s.kstride = s.Rp;
  s.estride = s.Rp + 1;
  int o = 0;
  s.off_k = o;  // KF [dp][Rp] fp32, rows >= d zero
  o += dp * s.kstride;
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

__device__ inline void stage(float* dst, const float* __restrict__ src, int rows_src, int rows_dst, int R, int Rp,
                             int stride) {
  for (int i = threadIdx.x; i < rows_dst * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    dst[k * stride + r] = (r < R && k < rows_src) ? src[k * R + r] : 0.f;
  }
}

template <int L, int RT>
__global__ __launch_bounds__(kWavesMax* kWave) void k_cp_edge_bf16(EdgeArgs a, int n_cgrp, int waves, int chunk) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DP = d <= 32 ? 32 : 64;
  constexpr int KS = DP / 16;  // K-steps per edge
  constexpr int Rp = RT * kTile;
  constexpr int kCtw = ctw<RT>();
  constexpr bool kRegK = KS * RT * 8 <= 64;  // K factor in registers when it fits
  extern __shared__ float smem[];
  const Bf16Smem S = bf16_smem(RT, d, DP, a.n_radial, chunk);
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
  const int ct0 = (cgrp * waves + wave) * kCtw;  // first channel tile of this wave
  const uint16_t* __restrict__ xT = static_cast<const uint16_t*>(a.feat);

  stage(sK, a.KF, d, DP, a.R, Rp, S.kstride);
  stage(sBE, a.Bf, d, d, a.R, Rp, Rp);
  stage(sBE + d * Rp, a.radial_w, nr, nr, a.R, Rp, Rp);
  __syncthreads();

  // K factor of this lane: KF[16j + 8h + i][rt*32 + l32], from registers
  // when it fits, else from LDS
  float kreg[kRegK ? KS : 1][kRegK ? RT : 1][8];
  if constexpr (kRegK) {
#pragma unroll
    for (int j = 0; j < KS; ++j)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 8; ++i) kreg[j][rt][i] = sK[(16 * j + 8 * h + i) * S.kstride + rt * kTile + l32];
  }
  auto kval = [&](int j, int rt, int i) -> float {
    if constexpr (kRegK)
      return kreg[j][rt][i];
    else
      return sK[(16 * j + 8 * h + i) * S.kstride + rt * kTile + l32];
  };

  f32x16 acc[RT][kCtw];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < kCtw; ++t) acc[rt][t] = f32x16{};

  // B operand of K-step j, channel tile t: xT[row][c][16j + 8h .. +7] (one
  // 16-byte load; channels past C clamp to C-1, whose results are dropped)
  auto load_edge = [&](int row, u32x4 (&b)[KS][ctw<RT>()]) {
#pragma unroll
    for (int t = 0; t < kCtw; ++t) {
      int c = (ct0 + t) * kTile + l32;
      c = c < C ? c : C - 1;
      const uint16_t* p = xT + (size_t(row) * C + c) * DP + 8 * h;
#pragma unroll
      for (int j = 0; j < KS; ++j) b[j][t] = *reinterpret_cast<const u32x4*>(p + 16 * j);
    }
  };

  const int e_begin = a.offsets[seg], e_end = a.offsets[seg + 1];
  for (int cb = e_begin; cb < e_end; cb += chunk) {
    const int n = min(chunk, e_end - cb);
    __syncthreads();
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
    // g = (Y B) * (Phi Wrad), fp32 MFMA, one (32 edges x 32 ranks) tile per item
    const int n_et = (n + kTile - 1) / kTile;
    for (int item = wave; item < n_et * RT; item += waves) {
      const int et = item / RT, rt = item - et * RT;
      const int er = et * kTile + l32;
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

    auto edge_mfma = [&](int e, const u32x4 (&b)[KS][ctw<RT>()]) {
      float g[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) g[rt] = sG[e * Rp + rt * kTile + l32];
#pragma unroll
      for (int j = 0; j < KS; ++j) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          bf16x8 av;
#pragma unroll
          for (int i = 0; i < 8; ++i) av[i] = static_cast<__bf16>(g[rt] * kval(j, rt, i));
#pragma unroll
          for (int t = 0; t < kCtw; ++t)
            acc[rt][t] = mfma32_bf16(av, __builtin_bit_cast(bf16x8, b[j][t]), acc[rt][t]);
        }
      }
    };
    u32x4 b0[KS][kCtw], b1[KS][kCtw];
    load_edge(sIdx[0], b0);
    int e = 0;
    for (; e + 1 < n; e += 2) {
      load_edge(sIdx[e + 1], b1);
      __builtin_amdgcn_sched_barrier(0);
      edge_mfma(e, b0);
      __builtin_amdgcn_sched_barrier(0);
      load_edge(sIdx[e + 2 < n ? e + 2 : e + 1], b0);
      __builtin_amdgcn_sched_barrier(0);
      edge_mfma(e + 1, b1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (e < n) edge_mfma(e, b0);
  }

  // Epilogue (fp32 MFMA): out[seg][m][c] = sum_r EF[m][r] H[r][c], H taken
  // straight from the accumulators as the B operand (see cp_edge_impl.hpp).
  __syncthreads();
  stage(sBE, a.EF, d, d, a.R, Rp, S.estride);
  __syncthreads();
  constexpr int MT = (d + kTile - 1) / kTile;
#pragma unroll
  for (int t = 0; t < kCtw; ++t) {
    const int c = (ct0 + t) * kTile + l32;
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
          z = mfma32(av, acc[rt][t][v], z);
        }
      }
      if (c < C) {
        float* o = a.out + size_t(seg) * d * C + c;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = mt * kTile + acc_row(v, h);
          if (m < d) o[size_t(m) * C] = z[v];
        }
      }
    }
  }
}

template <int L, int RT>
hipError_t launch_l_rt(const EdgeArgs& a, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DP = d <= 32 ? 32 : 64;
  constexpr int kCtw = ctw<RT>();
  const int ntiles = (a.C + kTile - 1) / kTile;
  const int pairs = (ntiles + kCtw - 1) / kCtw;
  const int waves = pairs < kWavesMax ? pairs : kWavesMax;
  const int n_cgrp = (pairs + waves - 1) / waves;
  int chunk = 64;
  while (chunk > 8 && bf16_smem(RT, d, DP, a.n_radial, chunk).floats * 4 > 80 * 1024) chunk >>= 1;
  const size_t lds = size_t(bf16_smem(RT, d, DP, a.n_radial, chunk).floats) * 4;
  const int total = a.n_seg * n_cgrp;
  if (total == 0) return hipSuccess;
  auto k = k_cp_edge_bf16<L, RT>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(total), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  return hipGetLastError();
}

template <int L>
hipError_t launch_bf16_l(const EdgeArgs& a, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt<L, 1>(a, s);
    case 2: return launch_l_rt<L, 2>(a, s);
    case 3: return launch_l_rt<L, 3>(a, s);
    case 4: return launch_l_rt<L, 4>(a, s);
    case 5: return launch_l_rt<L, 5>(a, s);
    case 6: return launch_l_rt<L, 6>(a, s);
    case 7: return launch_l_rt<L, 7>(a, s);
    case 8: return launch_l_rt<L, 8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace edge_bf16_detail

}  // namespace tdn
