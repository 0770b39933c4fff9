// The exact CG tensor product over the edges, the comparator of the CP edge
// pass: for every destination node n,
//   Z[n] = sum over edges e into n of K_e x[s_e],
//   K_e[k][i] = sum_j C[k; i, j] Y_e[j] rho_e[path(k, i, j)],
// with C the real CG coefficients of every path (l1, l2, l3) of degree <= L
// (Sec. 2, eq. clebsch_gordan and the direct sum over paths), Y_e the real
// harmonics of the edge direction and rho_e = phi_e Wpath one radial weight
// per path (Sec. 3.2; the channel weight W is applied by the node GEMM).
//
// One workgroup per destination node, edges in batches of EB:
//   1. per edge: harmonics and radial basis into LDS;
//   2. rho_e = phi_e Wpath, one thread per (edge, path);
//   3. K_e in LDS: thread q takes the (k, i) pairs q, q + threads, ...,
//      loads each pair's coefficients (j, path, value) once and applies them
//      to all edges of the batch; the largest |K_e| per edge sets the power of
//      two that puts K_e in the fp16 split's range;
//   4. per edge and 32-channel tile: U = K_e x[s_e] on 32x32x16 fp16 MFMA from
//      the three part products of the two-part splits (K_e split on the fly
//      from LDS, x from the edge pass's operand blocks), then
//      acc += 2^(e_K + e_x) U in fp32.
// The node's d x C sum is stored once.  Work per edge: nnz(C) multiply-adds
// for K_e (independent of C) and 2 d^2 C flops of contraction (d padded to
// 32 or 64).
//
// UN (the product without path-weight sharing): the output rows are the
// paths' own blocks, row[p] + m3 over all paths (PathRows), so that each
// path's channel matrix can be applied afterwards (launch_path_gemm).  K_e
// then has those rows; a launch covers a chunk of dense_un_rows of them (the
// kernel runs once per chunk), and a coefficient entry (k, i, j) goes to row
// row[p] + m3(k) of the chunk, p the path (deg i, deg j, deg k) in the order
// l1, l2, l3 (each ascending); the table's own path field is not used.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace dense_detail {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma_f16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0,
                                                0);
}

constexpr int kMaxWaves = 4;

__host__ __device__ constexpr int dense_dp(int d) { return d <= 32 ? 32 : 64; }  // MFMA rows and K, padded
// K_e in LDS: the d rows only, columns up to the next multiple of 8 (zero
// past d), row stride 4 floats more (16-byte aligned, fewer bank conflicts)
__host__ __device__ constexpr int dense_kc(int d) { return (d + 7) / 8 * 8; }
__host__ __device__ constexpr int dense_ks(int d) { return dense_kc(d) + 4; }
// edges per batch (16 at d = 16 measured 13 % faster than 8; 32 at d <= 9
// cost occupancy and was slower)
__host__ __device__ constexpr int dense_eb(int d) { return d <= 9 ? 8 : (d <= 16 ? 16 : (d <= 32 ? 8 : 4)); }

// UN: output row tiles per launch (the 1, 11, 51 and 156 path rows of
// L = 0..3 in one launch; 8 at L = 4, 4 at d = 36 and 49, where the operand
// blocks are twice as large and 8 tiles spill) and edges per batch
__host__ __device__ constexpr int dense_un_tiles(int d) {
  return d == 1 || d == 4 ? 1 : (d == 9 ? 2 : (d == 16 ? 5 : (d <= 32 ? 8 : 4)));
}
__host__ __device__ constexpr int dense_un_rows(int d) { return dense_un_tiles(d) * kTile; }
__host__ __device__ constexpr int dense_eb_un(int) { return 2; }

struct DenseSmem {
  int off_k, off_y, off_phi, off_rho, off_row, off_sc, off_ksc, off_max, off_pre, floats;
};
__host__ __device__ inline DenseSmem dense_smem(int d, int n_path, bool un = false) {
  const int eb = un ? dense_eb_un(d) : dense_eb(d);
  DenseSmem s{};
  int o = 0;
  s.off_k = o;
  o += eb * (un ? dense_un_rows(d) : d) * dense_ks(d);
  s.off_y = o;
  o += eb * d;
  s.off_phi = o;
  o += eb * 16;
  s.off_rho = o;
  o += eb * n_path;
  s.off_row = o;
  o += eb;
  s.off_sc = o;
  o += eb;
  s.off_ksc = o;
  o += eb;
  s.off_max = o;
  o += kMaxWaves * eb;
  s.off_pre = o;  // UN: first item of each of the launch's paths
  o += un ? kMaxPaths + 1 : 0;
  s.floats = o;
  return s;
}

template <int L, int CTW, bool UN = false>
__global__ __launch_bounds__(256) void k_dense_edge(DenseArgs a, int waves, PathRows pt, int row0, int p_lo, int p_hi,
                                                    float* zp) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DP = dense_dp(d), KC = dense_kc(d), KS = dense_ks(d), EB = UN ? dense_eb_un(d) : dense_eb(d);
  constexpr int KB = DP / 16, RK = UN ? dense_un_tiles(d) : DP / 32;
  constexpr int KR = UN ? dense_un_rows(d) : d;  // rows of K_e held in LDS
  extern __shared__ float smem[];
  const DenseSmem sm = dense_smem(d, a.n_path, UN);
  float* sK = smem + sm.off_k;
  float* sY = smem + sm.off_y;
  float* sPhi = smem + sm.off_phi;
  float* sRho = smem + sm.off_rho;
  int* sRow = reinterpret_cast<int*>(smem + sm.off_row);
  float* sSc = smem + sm.off_sc;
  float* sKsc = smem + sm.off_ksc;
  float* sMax = smem + sm.off_max;

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int h = lane >> 5, l32 = lane & 31;
  const int nthr = blockDim.x;
  const int n = xcd_remap(blockIdx.x, a.N);
  const int e0 = a.offsets[n], e1 = a.offsets[n + 1];
  const int P = a.n_path, nr = a.n_radial;

  // K's padding columns (d .. KC-1) stay zero; every (k, i) with k, i < d is
  // rewritten for each batch
  for (int t = tid; t < EB * KR * KS; t += nthr) sK[t] = 0.f;
  // UN over part of the paths (several launches): the launch's (path, m3,
  // m1) items, path p_lo + u from item pre[u]; over all paths (one launch):
  // the (k, i) rows, each walked once
  const bool un_items = UN && p_hi - p_lo < pt.n_path;
  int* sPre = reinterpret_cast<int*>(smem + sm.off_pre);
  if (un_items && tid == 0) {
    int acc = 0;
    for (int p = p_lo; p < p_hi; ++p) {
      sPre[p - p_lo] = acc;
      acc += (2 * pt.l3[p] + 1) * (2 * pt.l1[p] + 1);
    }
    sPre[p_hi - p_lo] = acc;
  }

  f32x16 acc[RK][CTW];
#pragma unroll
  for (int r = 0; r < RK; ++r)
#pragma unroll
    for (int c = 0; c < CTW; ++c) acc[r][c] = f32x16{};

  const char* __restrict__ xs = static_cast<const char*>(a.feat);
  const int n_ct = (a.C + kTile - 1) / kTile;
  const size_t row_bytes = size_t(n_ct) * 2 * KB * 1024;
  uint32_t lane_off[CTW];
#pragma unroll
  for (int c = 0; c < CTW; ++c) {
    const int ct = min(wave * CTW + c, n_ct - 1);
    lane_off[c] = uint32_t(ct * 2 * KB * 1024 + h * 512 + l32 * 16);
  }
  // x[row] operand blocks of this wave's channel tiles: [tile][part][K-block]
  auto load_x = [&](int row, u32x4 (&xb)[CTW][2][KB]) {
    const char* p = xs + size_t(row) * row_bytes;
#pragma unroll
    for (int c = 0; c < CTW; ++c)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int b = 0; b < KB; ++b)
          xb[c][s][b] = *reinterpret_cast<const u32x4*>(p + lane_off[c] + uint32_t((s * KB + b) * 1024));
  };
  auto edge_compute = [&](int t, const u32x4 (&xb)[CTW][2][KB]) {
    const float ksc = sKsc[t], usc = sSc[t];
#pragma unroll
    for (int r = 0; r < RK; ++r) {
      u32x4 hi[KB], lo[KB];
      const int row = r * kTile + l32;
      const float* kp = sK + (t * KR + (row < KR ? row : 0)) * KS + 8 * h;
#pragma unroll
      for (int b = 0; b < KB; ++b) {
        // rows >= d (UN: past the chunk) and column groups >= KC are zero
        // (not stored)
        const bool in = row < KR && 16 * b + 8 * h < KC;
        float4 f0 = make_float4(0.f, 0.f, 0.f, 0.f), f1 = f0;
        if (in) {
          f0 = *reinterpret_cast<const float4*>(kp + 16 * b);
          f1 = *reinterpret_cast<const float4*>(kp + 16 * b + 4);
        }
        uint32_t h0, h1, h2, h3, m0, m1, m2, m3;
        split_f16x2_pair(f0.x * ksc, f0.y * ksc, h0, m0);
        split_f16x2_pair(f0.z * ksc, f0.w * ksc, h1, m1);
        split_f16x2_pair(f1.x * ksc, f1.y * ksc, h2, m2);
        split_f16x2_pair(f1.z * ksc, f1.w * ksc, h3, m3);
        hi[b] = u32x4{h0, h1, h2, h3};
        lo[b] = u32x4{m0, m1, m2, m3};
      }
#pragma unroll
      for (int c = 0; c < CTW; ++c) {
        f32x16 u = f32x16{};
#pragma unroll
        for (int b = 0; b < KB; ++b) u = mfma_f16(lo[b], xb[c][0][b], u);
#pragma unroll
        for (int b = 0; b < KB; ++b) u = mfma_f16(hi[b], xb[c][1][b], u);
#pragma unroll
        for (int b = 0; b < KB; ++b) u = mfma_f16(hi[b], xb[c][0][b], u);
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[r][c][v] = fmaf(usc, u[v], acc[r][c][v]);
      }
    }
  };

  for (int b0 = e0; b0 < e1; b0 += EB) {
    const int nb = min(EB, e1 - b0);
    __syncthreads();  // the previous batch's K consumed (and the zero fill done)
    // 1. per edge: gathered row, harmonics, radial basis
    if (tid < nb) {
      const int eid = a.perm[b0 + tid];
      sRow[tid] = a.src[eid];
      const float vx = a.edge_vec[3 * size_t(eid)], vy = a.edge_vec[3 * size_t(eid) + 1],
                  vz = a.edge_vec[3 * size_t(eid) + 2];
      const float len = sqrtf(vx * vx + vy * vy + vz * vz);
      const float inv = 1.f / len;
      sh_unit_all<L>(vx * inv, vy * inv, vz * inv, sY + tid * d);
      for (int q = 0; q < nr; ++q) sPhi[tid * 16 + q] = radial_phi(len, q, a.sigma);
    }
    __syncthreads();
    // 2. rho = phi Wpath
    for (int t = tid; t < nb * P; t += nthr) {
      const int e = t / P, p = t - e * P;
      float s = 0.f;
      for (int q = 0; q < nr; ++q) s = fmaf(sPhi[e * 16 + q], a.path_w[q * P + p], s);
      sRho[e * P + p] = s;
    }
    __syncthreads();
    // 3. K_e for the batch, and the largest |K_e| of each edge
    float mx[EB];
#pragma unroll
    for (int e = 0; e < EB; ++e) mx[e] = 0.f;
    if (un_items) {
      // item (p, m3, m1) sums the entries of row (k, i) = (l3^2 + m3,
      // l1^2 + m1) whose j has degree l2 and writes row row[p] + m3 - row0,
      // column i, zero where the table holds no entry (every row position of
      // the launch's paths is written; rows outside the chunk are skipped)
      const int n_item = sPre[p_hi - p_lo];
      for (int it = tid; it < n_item; it += nthr) {
        int u = 0;  // the path of item it: the last u with pre[u] <= it
        for (int step = 128; step > 0; step >>= 1)  // kMaxPaths <= 256
          if (u + step < p_hi - p_lo && sPre[u + step] <= it) u += step;
        const int p = p_lo + u, r = it - sPre[u];
        const int l1 = pt.l1[p], l2 = pt.l2[p], l3 = pt.l3[p];
        const int m3 = r / (2 * l1 + 1), m1 = r - m3 * (2 * l1 + 1);
        const int row = pt.row[p] + m3 - row0;
        if (row < 0 || row >= KR) continue;
        const int k = l3 * l3 + m3, i = l1 * l1 + m1, q = k * d + i;
        int s0 = a.cg_row[q], s1 = a.cg_row[q + 1];
        s0 = max(0, min(s0, a.cg_nnz));
        s1 = max(s0, min(s1, a.cg_nnz));
        float v[EB];
#pragma unroll
        for (int e = 0; e < EB; ++e) v[e] = 0.f;
        for (int s = s0; s < s1; ++s) {
          const int j = a.cg_col[s] & 0xffff;
          if (j >= (l2 + 1) * (l2 + 1)) break;
          if (j < l2 * l2) continue;
          const float cv = a.cg_val[s];
#pragma unroll
          for (int e = 0; e < EB; ++e)
            if (e < nb) v[e] = fmaf(cv, sY[e * d + j] * sRho[e * P + p], v[e]);
        }
#pragma unroll
        for (int e = 0; e < EB; ++e)
          if (e < nb) {
            sK[(e * KR + row) * KS + i] = v[e];
            mx[e] = fmaxf(mx[e], fabsf(v[e]));
          }
      }
    }
    for (int q = tid; q < (un_items ? 0 : d * d); q += nthr) {
      const int k = q / d, i = q - k * d;
      int s0 = a.cg_row[q], s1 = a.cg_row[q + 1];
      s0 = max(0, min(s0, a.cg_nnz));
      s1 = max(s0, min(s1, a.cg_nnz));
      float v[EB];
#pragma unroll
      for (int e = 0; e < EB; ++e) v[e] = 0.f;
      if constexpr (UN) {
        // one K row per (path, m3): for k of degree l3 and i of degree l1,
        // the rows of the paths (l1, l2, l3), l2 = |l1 - l3| .. min(l1 + l3, L),
        // each summing the entries whose j has degree l2 (consecutive, as the
        // row lists j in order).  Every such row position is written, zero
        // where the table holds no entry, so no value of the previous batch
        // stays behind; rows outside this launch's chunk are skipped.
        const int l3k = int(sqrtf(float(k) + 0.5f)), l1i = int(sqrtf(float(i) + 0.5f));
        const int lo2 = l1i > l3k ? l1i - l3k : l3k - l1i, hi2 = l1i + l3k < L ? l1i + l3k : L;
        int s = s0;
        for (int l2 = lo2; l2 <= hi2; ++l2) {
          const int p = pt.first[l1i * (L + 1) + l2] + (l3k - (l1i > l2 ? l1i - l2 : l2 - l1i));
#pragma unroll
          for (int e = 0; e < EB; ++e) v[e] = 0.f;
          for (; s < s1; ++s) {
            const int j = a.cg_col[s] & 0xffff;
            if (j >= d) continue;  // malformed: ignored
            const int l2j = int(sqrtf(float(j) + 0.5f));
            if (l2j > l2) break;
            if (l2j < l2) continue;  // no path with this degree: ignored
            const float cv = a.cg_val[s];
#pragma unroll
            for (int e = 0; e < EB; ++e)
              if (e < nb) v[e] = fmaf(cv, sY[e * d + j] * sRho[e * P + p], v[e]);
          }
          const int row = pt.row[p] + (k - l3k * l3k) - row0;
          if (row >= 0 && row < KR) {
#pragma unroll
            for (int e = 0; e < EB; ++e)
              if (e < nb) {
                sK[(e * KR + row) * KS + i] = v[e];
                mx[e] = fmaxf(mx[e], fabsf(v[e]));
              }
          }
        }
        continue;
      }
      // for d > 32 (rows of ~5 entries) four entries' loads issued together,
      // then applied in order; one at a time below (fewer registers, more
      // waves)
      constexpr int U = d > 32 ? 4 : 1;
      for (int s = s0; s < s1; s += U) {
        int cl[U];
        float cv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int su = s + u < s1 ? s + u : s0;
          cl[u] = a.cg_col[su];
          cv[u] = a.cg_val[su];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int j = cl[u] & 0xffff, p = cl[u] >> 16;
          if (s + u >= s1 || j >= d || p < 0 || p >= P) continue;  // past the row, or malformed: ignored
#pragma unroll
          for (int e = 0; e < EB; ++e)
            if (e < nb) v[e] = fmaf(cv[u], sY[e * d + j] * sRho[e * P + p], v[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < EB; ++e)
        if (e < nb) {
          sK[(e * d + k) * KS + i] = v[e];
          mx[e] = fmaxf(mx[e], fabsf(v[e]));
        }
    }
#pragma unroll
    for (int e = 0; e < EB; ++e) {
      float m = mx[e];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
      if (lane == 0) sMax[wave * EB + e] = m;
    }
    __syncthreads();
    if (tid < nb) {
      float m = 0.f;
      for (int w = 0; w < waves; ++w) m = fmaxf(m, sMax[w * EB + tid]);
      const int ek = f16_split_exponent(m);
      sKsc[tid] = ldexpf(1.f, -ek);
      sSc[tid] = ldexpf(a.row_scale[sRow[tid]], ek);
    }
    __syncthreads();
    // 4. the contraction, x of edge t + 1 loaded while edge t computes
    u32x4 x0[CTW][2][KB], x1[CTW][2][KB];
    load_x(__builtin_amdgcn_readfirstlane(sRow[0]), x0);
    int t = 0;
    for (; t + 1 < nb; t += 2) {
      load_x(__builtin_amdgcn_readfirstlane(sRow[t + 1]), x1);
      __builtin_amdgcn_sched_barrier(0);
      edge_compute(t, x0);
      __builtin_amdgcn_sched_barrier(0);
      load_x(__builtin_amdgcn_readfirstlane(sRow[t + 2 < nb ? t + 2 : t + 1]), x0);  // past the end: unused
      __builtin_amdgcn_sched_barrier(0);
      edge_compute(t + 1, x1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (t < nb) edge_compute(t, x0);
  }
  // Z[n] rows k < d (UN: the chunk's path rows), channels of this wave's tiles
#pragma unroll
  for (int c = 0; c < CTW; ++c) {
    const int ct = wave * CTW + c;
    const int ch = ct * kTile + l32;
    if (ct >= n_ct || ch >= a.C) continue;
#pragma unroll
    for (int r = 0; r < RK; ++r)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int k = r * kTile + acc_row(v, h);
        if constexpr (UN) {
          if (row0 + k < pt.n_rows) zp[(size_t(n) * pt.n_rows + row0 + k) * a.C + ch] = acc[r][c][v];
        } else {
          if (k < d) a.out[(size_t(n) * d + k) * a.C + ch] = acc[r][c][v];
        }
      }
  }
}

template <int L, int CTW>
hipError_t launch_l_ctw(const DenseArgs& a, int waves, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const size_t lds = size_t(dense_smem(d, a.n_path).floats) * 4;
  auto k = k_dense_edge<L, CTW>;
  hipError_t e =
      hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  PathRows none{};
  k<<<dim3(a.N), dim3(waves * kWave), lds, s>>>(a, waves, none, 0, 0, 0, nullptr);
  return hipGetLastError();
}

// UN: one launch per chunk of kUnRows path rows (one 32-channel tile per
// wave, C <= 128)
template <int L>
hipError_t launch_l_un(const DenseArgs& a, float* zp, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const int n_ct = (a.C + kTile - 1) / kTile;
  const PathRows pt = path_rows(L);
  const size_t lds = size_t(dense_smem(d, a.n_path, true).floats) * 4;
  auto k = k_dense_edge<L, 1, true>;
  hipError_t e =
      hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  for (int row0 = 0; row0 < pt.n_rows; row0 += dense_un_rows(d)) {
    // the paths whose rows meet [row0, row0 + rows of a launch)
    int p_lo = 0;
    while (p_lo < pt.n_path && pt.row[p_lo] + 2 * pt.l3[p_lo] + 1 <= row0) ++p_lo;
    int p_hi = p_lo;
    while (p_hi < pt.n_path && pt.row[p_hi] < row0 + dense_un_rows(d)) ++p_hi;
    k<<<dim3(a.N), dim3(n_ct * kWave), lds, s>>>(a, n_ct, pt, row0, p_lo, p_hi, zp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int L>
hipError_t launch_l(const DenseArgs& a, hipStream_t s) {
  const int n_ct = (a.C + kTile - 1) / kTile;
  const int waves = n_ct < kMaxWaves ? n_ct : kMaxWaves;
  return n_ct <= kMaxWaves ? launch_l_ctw<L, 1>(a, waves, s) : launch_l_ctw<L, 2>(a, waves, s);
}

}  // namespace dense_detail

int dense_path_count(int L) {
  int n = 0;
  for (int l1 = 0; l1 <= L; ++l1)
    for (int l2 = 0; l2 <= L; ++l2) {
      const int lo = l1 > l2 ? l1 - l2 : l2 - l1, hi = l1 + l2 < L ? l1 + l2 : L;
      n += hi - lo + 1;
    }
  return n;
}

PathRows path_rows(int L) {
  PathRows t{};
  int p = 0, row = 0;
  for (int l1 = 0; l1 <= L; ++l1)
    for (int l2 = 0; l2 <= L; ++l2) {
      const int lo = l1 > l2 ? l1 - l2 : l2 - l1, hi = l1 + l2 < L ? l1 + l2 : L;
      if (l1 * (L + 1) + l2 < kMaxDegPairs) t.first[l1 * (L + 1) + l2] = p;
      for (int l3 = lo; l3 <= hi && p < kMaxPaths; ++l3, ++p) {
        t.l1[p] = l1;
        t.l2[p] = l2;
        t.l3[p] = l3;
        t.row[p] = row;
        row += 2 * l3 + 1;
      }
    }
  t.n_path = p;
  t.n_rows = row;
  return t;
}

hipError_t launch_dense_edge_unshared(const DenseArgs& a, float* zp, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  if (a.C < 1 || a.C > 4 * kTile || a.n_radial < 1 || a.n_radial > 16 || a.n_path != dense_path_count(a.L) ||
      a.feat == nullptr || a.row_scale == nullptr || zp == nullptr)
    return hipErrorInvalidValue;
  switch (a.L) {
    case 0: return dense_detail::launch_l_un<0>(a, zp, s);
    case 1: return dense_detail::launch_l_un<1>(a, zp, s);
    case 2: return dense_detail::launch_l_un<2>(a, zp, s);
    case 3: return dense_detail::launch_l_un<3>(a, zp, s);
    case 4: return dense_detail::launch_l_un<4>(a, zp, s);
    case 5: return dense_detail::launch_l_un<5>(a, zp, s);
    case 6: return dense_detail::launch_l_un<6>(a, zp, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_dense_edge(const DenseArgs& a, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  if (a.C < 1 || a.C > 8 * kTile || a.n_radial < 1 || a.n_radial > 16 || a.n_path != dense_path_count(a.L) ||
      a.feat == nullptr || a.row_scale == nullptr)
    return hipErrorInvalidValue;
  switch (a.L) {
    case 0: return dense_detail::launch_l<0>(a, s);
    case 1: return dense_detail::launch_l<1>(a, s);
    case 2: return dense_detail::launch_l<2>(a, s);
    case 3: return dense_detail::launch_l<3>(a, s);
    case 4: return dense_detail::launch_l<4>(a, s);
    case 5: return dense_detail::launch_l<5>(a, s);
    case 6: return dense_detail::launch_l<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
