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
// g_e[r] for every rank (all lanes), into LDS; the MFMA loop builds the K
// operand on the fly from g and the LDS-resident factor and streams the B
// operand x[s_e][k, c] straight from global memory (each half-wave reads one
// contiguous 128-byte row slice), software-pipelined U steps ahead.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

constexpr int kMaxWavesPerBlock = 4;
constexpr int kPipe = 4;  // B-operand loads in flight per lane

struct EdgeSmem {
  int Rp, kstride, estride, d, n_radial, chunk;
  int off_k, off_be, off_g, off_y, off_phi, off_idx;
  int floats;
};

__host__ __device__ inline EdgeSmem edge_smem(int RT, int d, int n_radial, int chunk) {
  EdgeSmem s{};
  s.Rp = RT * kTile;
  s.kstride = s.Rp + 32;  // consecutive K rows land 32 banks apart
  s.estride = s.Rp + 1;   // epilogue reads a column across 32 rows
  s.d = d;
  s.n_radial = n_radial;
  s.chunk = chunk;
  int o = 0;
  s.off_k = o;
  o += d * s.kstride;
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

// Stage a [d, R] factor into LDS rows of `stride` floats, zero beyond R.
__device__ inline void stage_factor(float* dst, const float* __restrict__ src, int rows, int R, int Rp, int stride) {
  for (int i = threadIdx.x; i < rows * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    dst[k * stride + r] = r < R ? src[k * R + r] : 0.f;
  }
}

template <int RT, typename TF>
__global__ __launch_bounds__(kMaxWavesPerBlock* kWave) void k_cp_edge(EdgeArgs a, int n_cgrp, int waves, int chunk) {
  extern __shared__ float smem[];
  const EdgeSmem L = edge_smem(RT, a.d, a.n_radial, chunk);
  constexpr int Rp = RT * kTile;
  float* sK = smem + L.off_k;
  float* sBE = smem + L.off_be;
  float* sG = smem + L.off_g;
  float* sY = smem + L.off_y;
  float* sPhi = smem + L.off_phi;
  int* sIdx = reinterpret_cast<int*>(smem + L.off_idx);

  const int total = a.n_seg * n_cgrp;
  const int logical = xcd_remap(blockIdx.x, total);
  const int seg = logical / n_cgrp, cgrp = logical - seg * n_cgrp;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int h = lane >> 5, l32 = lane & 31;
  const int d = a.d, C = a.C, nr = a.n_radial;
  const int c = (cgrp * waves + wave) * kTile + l32;
  const bool cvalid = c < C;
  const TF* __restrict__ feat = static_cast<const TF*>(a.feat);

  stage_factor(sK, a.KF, d, a.R, Rp, L.kstride);
  stage_factor(sBE, a.Bf, d, a.R, Rp, Rp);
  stage_factor(sBE + d * Rp, a.radial_w, nr, a.R, Rp, Rp);

  f32x16 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x16{};

  const int e_begin = a.offsets[seg], e_end = a.offsets[seg + 1];
  for (int cb = e_begin; cb < e_end; cb += chunk) {
    const int n = min(chunk, e_end - cb);
    __syncthreads();  // factors staged / previous chunk consumed
    if (tid < n) {
      const int eid = a.perm[cb + tid];
      const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
      const float rn = sqrtf(vx * vx + vy * vy + vz * vz);
      const float inv = 1.f / rn;
      sh_unit(a.L, vx * inv, vy * inv, vz * inv, sY + tid * d);
      for (int q = 0; q < nr; ++q) sPhi[tid * nr + q] = radial_phi(rn, q, a.sigma);
      sIdx[tid] = a.gather[eid];
    }
    __syncthreads();
    // g_e[r] = (sum_k B[k,r] Y_e[k]) * (sum_q Wrad[q,r] phi_e[q])
    for (int i = tid; i < n * Rp; i += blockDim.x) {
      const int e = i / Rp, r = i - e * Rp;
      float v = 0.f, rho = 0.f;
      for (int k = 0; k < d; ++k) v += sBE[k * Rp + r] * sY[e * d + k];
      for (int q = 0; q < nr; ++q) rho += sBE[(d + q) * Rp + r] * sPhi[e * nr + q];
      sG[e * Rp + r] = v * rho;
    }
    __syncthreads();

    // MFMA over the flattened contraction index j = e*d + k; K-step s covers
    // j = 2s (lanes 0-31) and j = 2s+1 (lanes 32-63).
    const int T = n * d;
    const int S = (T + 1) >> 1;
    int le = h / d, lk = h - (h / d) * d;  // load cursor
    int ce = le, ck = lk;                  // compute cursor
    float bq[kPipe];
#pragma unroll
    for (int u = 0; u < kPipe; ++u) {
      float v = 0.f;
      if (le < n && cvalid) v = load_feat<TF>(feat + (size_t(sIdx[le]) * d + lk) * C + c);
      bq[u] = v;
      lk += 2;
      while (lk >= d) { lk -= d; ++le; }
    }
    for (int s0 = 0; s0 < S; s0 += kPipe) {
      float bn[kPipe];
#pragma unroll
      for (int u = 0; u < kPipe; ++u) {
        float v = 0.f;
        if (le < n && cvalid) v = load_feat<TF>(feat + (size_t(sIdx[le]) * d + lk) * C + c);
        bn[u] = v;
        lk += 2;
        while (lk >= d) { lk -= d; ++le; }
      }
#pragma unroll
      for (int u = 0; u < kPipe; ++u) {
        if (s0 + u < S) {
          const bool valid = ce < n;
          const float* gr = sG + ce * Rp + l32;
          const float* kr = sK + ck * L.kstride + l32;
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            const float av = valid ? gr[rt * kTile] * kr[rt * kTile] : 0.f;
            acc[rt] = mfma32(av, bq[u], acc[rt]);
          }
          ck += 2;
          while (ck >= d) { ck -= d; ++ce; }
        }
      }
#pragma unroll
      for (int u = 0; u < kPipe; ++u) bq[u] = bn[u];
    }
  }

  // Epilogue: out[seg][m][c] = sum_r EF[m][r] H[r][c].  The contraction over r
  // pairs accumulator register v of the two half-waves: lanes 0-31 contribute
  // rank rt*32 + acc_row(v,0), lanes 32-63 rank rt*32 + acc_row(v,1), which is
  // exactly the B-operand layout, so H never leaves the registers.
  __syncthreads();
  stage_factor(sBE, a.EF, d, a.R, Rp, L.estride);
  __syncthreads();
  const int MT = (d + kTile - 1) / kTile;
  for (int mt = 0; mt < MT; ++mt) {
    f32x16 z = f32x16{};
    const int row = mt * kTile + l32;
    const float* er = sBE + row * L.estride;
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

template <int RT>
hipError_t launch_rt(const EdgeArgs& a, bool bf16, hipStream_t s) {
  const int ntiles = (a.C + kTile - 1) / kTile;
  const int waves = ntiles < kMaxWavesPerBlock ? ntiles : kMaxWavesPerBlock;
  const int n_cgrp = (ntiles + waves - 1) / waves;
  // largest edge chunk (<= 32) that keeps LDS within 80 KB, at least 4
  int chunk = 32;
  while (chunk > 4 && edge_smem(RT, a.d, a.n_radial, chunk).floats * 4 > 80 * 1024) chunk >>= 1;
  const size_t lds = size_t(edge_smem(RT, a.d, a.n_radial, chunk).floats) * 4;
  const int total = a.n_seg * n_cgrp;
  if (total == 0) return hipSuccess;
  if (bf16) {
    auto k = k_cp_edge<RT, uint16_t>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(total), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  } else {
    auto k = k_cp_edge<RT, float>;
    hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    k<<<dim3(total), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_cp_edge(const EdgeArgs& a, bool feat_bf16, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_rt<1>(a, feat_bf16, s);
    case 2: return launch_rt<2>(a, feat_bf16, s);
    case 3: return launch_rt<3>(a, feat_bf16, s);
    case 4: return launch_rt<4>(a, feat_bf16, s);
    case 5: return launch_rt<5>(a, feat_bf16, s);
    case 6: return launch_rt<6>(a, feat_bf16, s);
    case 7: return launch_rt<7>(a, feat_bf16, s);
    case 8: return launch_rt<8>(a, feat_bf16, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
