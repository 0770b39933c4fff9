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
// Work decomposition.  The sorted edge list is cut into n_range equal ranges,
// as many as the device holds workgroups at once (over the channel groups),
// so every workgroup gets the same number of edges and the launch has no
// tail; the factors are staged once per workgroup.  A workgroup covers one
// range for up to four 32-channel tiles: wave w owns channel tile w and all R
// rank rows, so its accumulators are RT = ceil(R/32) MFMA tiles of 32x32.
// Per chunk of edges the block evaluates the harmonics and radial basis, then
// g_e[r] for every rank, into LDS, and marks where in the chunk a new segment
// starts.  The MFMA loop then walks the chunk edge by edge: each edge's
// contraction over its d feature rows is padded to an even length (a zero row
// when d is odd), so one 32x32x2 K-step always covers rows 2j and 2j+1 of one
// edge; g_e is held in registers for the edge, the K operand is
// g_e[r] * KF[k][r], and the B operand x[s_e][k][c] comes straight from
// global memory (each half-wave reads one contiguous 128-byte row slice),
// loaded one edge ahead.  Where a segment ends the epilogue Z = EF H runs on
// the accumulators and they restart from zero.  A segment wholly inside the
// range is written to its output row; the first segment of a range, when it
// began in an earlier range, and the last one, when it continues into a later
// range, go to two per-range partial slots that a small second kernel adds
// up in range order (fixed order, deterministic); that kernel also writes the
// zero rows of segments without edges.
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

// Whether this lane's share of the K factor, KF[2j + h][rt*32 + l32] for all
// K-steps j and rank tiles rt, fits in registers beside the accumulators.
__host__ __device__ constexpr bool edge_reg_k(int d, int RT) { return (d + 1) / 2 * RT <= 64; }

// Two waves per SIMD (two workgroups per CU) when the K factor is register
// resident; one otherwise (large R at high L), where spilling would cost more
// than the lost occupancy.
__host__ __device__ constexpr int edge_waves_per_eu(int L, int RT) {
  return edge_reg_k((L + 1) * (L + 1), RT) ? 2 : 1;
}

struct EdgeSmem {
  int Rp, kstride, estride, off_k, off_be, off_ef, off_g, off_y, off_vec, off_phi, off_idx, off_bnd, floats;
};

// LDS regions: the K factor (only when it is not register resident), the
// harmonic and radial factors B and radial_w, the output factor EF (only
// when the K factor is in registers; otherwise the epilogue reads EF from
// global memory), g for a chunk of edges (rows rounded up to a whole 32-row
// tile), harmonics, normalised edge vectors with their lengths, radial basis,
// gathered rows, and the segment starts of the chunk (positions, keys, count
// and the two partial-segment flags).
__host__ __device__ inline EdgeSmem edge_smem(int RT, int d, int n_radial, int chunk) {
  EdgeSmem s{};
  const int dpad = d + (d & 1);
  const bool reg_k = edge_reg_k(d, RT);
  s.Rp = RT * kTile;
  s.kstride = s.Rp + 32;  // rows 2j and 2j+1 land 32 banks apart
  s.estride = s.Rp + 1;   // the epilogue reads a column across 32 rows
  int o = 0;
  s.off_k = o;
  if (!reg_k) o += dpad * s.kstride;
  s.off_be = o;
  o += (d + n_radial) * s.Rp;
  s.off_ef = o;
  if (reg_k) o += d * s.estride;
  s.off_g = o;
  o += (chunk + kTile - 1) / kTile * kTile * s.Rp;
  s.off_y = o;
  o += chunk * d;
  o = (o + 3) & ~3;  // float4 rows
  s.off_vec = o;
  o += chunk * 4;
  s.off_phi = o;
  o += chunk * n_radial;
  s.off_idx = o;
  o += chunk;
  s.off_bnd = o;
  o += 2 * chunk + 4;
  s.floats = o;
  return s;
}

// Stage a [rows_src, R] factor into LDS rows of `stride` floats; zero beyond
// R and for rows rows_src..rows_dst-1.  Eight loads per thread are in flight
// at once (clamped addresses, zeroing by select) before any store.
__device__ inline void stage_factor(float* dst, const float* __restrict__ src, int rows_src, int rows_dst, int R,
                                    int Rp, int stride) {
  constexpr int U = 8;
  const int total = rows_dst * Rp;
  for (int i0 = threadIdx.x; i0 < total; i0 += U * blockDim.x) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * blockDim.x;
      const int k = i / Rp, r = i - k * Rp;
      const int kc = k < rows_src ? k : rows_src - 1, rc = r < R ? r : R - 1;
      v[u] = src[kc * R + rc];
      v[u] = (k < rows_src && r < R) ? v[u] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * blockDim.x;
      const int k = i / Rp, r = i - k * Rp;
      if (i < total) dst[k * stride + r] = v[u];
    }
  }
}

template <int L, int RT>
__global__ __launch_bounds__(kMaxWavesPerBlock* kWave) __attribute__((amdgpu_waves_per_eu(edge_waves_per_eu(L, RT))))
void k_cp_edge(EdgeArgs a, int n_cgrp, int waves, int chunk) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DH = (d + 1) / 2;  // K-steps per edge
  constexpr int Rp = RT * kTile;
  constexpr int MT = (d + kTile - 1) / kTile;
  constexpr bool kRegK = edge_reg_k(d, RT);
  extern __shared__ float smem[];
  const EdgeSmem S = edge_smem(RT, d, a.n_radial, chunk);
  float* sK = smem + S.off_k;
  float* sBE = smem + S.off_be;
  float* sEF = smem + S.off_ef;
  float* sG = smem + S.off_g;
  float* sY = smem + S.off_y;
  float4* sVec = reinterpret_cast<float4*>(smem + S.off_vec);
  float* sPhi = smem + S.off_phi;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);
  int* sBnd = reinterpret_cast<int*>(smem + S.off_bnd);  // [chunk] chunk positions where a segment starts
  int* sBndKey = sBnd + chunk;                          // [chunk] that segment
  int* sMeta = sBndKey + chunk;                         // start count, first partial, last partial

  const int total = a.n_range * n_cgrp;
  const int logical = xcd_remap(blockIdx.x, total);
  const int range = logical / n_cgrp, cgrp = logical - range * n_cgrp;
  const int e_lo = int(int64_t(range) * a.E / a.n_range), e_hi = int(int64_t(range + 1) * a.E / a.n_range);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int h = lane >> 5, l32 = lane & 31;
  const int C = a.C, nr = a.n_radial, R = a.R;
  const int c = (cgrp * waves + wave) * kTile + l32;
  const bool cvalid = c < C;
  const float* __restrict__ feat = static_cast<const float*>(a.feat);

  // When it fits (DH*RT <= 64 values per lane) the K factor of this lane
  // lives in registers for the whole range, read straight from global
  // memory; the pad row (2j + h == d) and ranks beyond R are zero.
  // Otherwise the factor is staged in LDS and read per K-step.
  float kreg[kRegK ? DH : 1][kRegK ? RT : 1];
  const float* kr = sK + h * S.kstride + l32;
  if constexpr (kRegK) {
#pragma unroll
    for (int j = 0; j < DH; ++j)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int k = 2 * j + h, r = rt * kTile + l32;
        const float v = a.KF[(k < d ? k : d - 1) * R + (r < R ? r : R - 1)];
        kreg[j][rt] = (k < d && r < R) ? v : 0.f;
      }
    stage_factor(sEF, a.EF, d, d, R, Rp, S.estride);
  } else {
    stage_factor(sK, a.KF, d, d + (d & 1), R, Rp, S.kstride);
  }
  stage_factor(sBE, a.Bf, d, d, R, Rp, Rp);
  stage_factor(sBE + d * Rp, a.radial_w, nr, nr, R, Rp, Rp);

  f32x16 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x16{};

  // Segment epilogue: Z[m][c] = sum_r EF[m][r] H[r][c].  The contraction over
  // r pairs accumulator register v of the two half-waves: lanes 0-31
  // contribute rank rt*32 + acc_row(v,0), lanes 32-63 rank rt*32 +
  // acc_row(v,1), which is exactly the B-operand layout, so H never leaves
  // the registers.  The A operand comes in groups of 16 values, one group per
  // (row tile mt, rank tile rt), the next group loaded while the current
  // one's MFMAs run; EF is read from LDS when staged there, else from global
  // memory.  slot < 0 writes the segment's output row, slot 0 or 1 the
  // range's partial slot; the accumulators restart from zero.
  auto finish = [&](int seg, int slot) {
    float* dst = slot < 0 ? a.out + size_t(seg) * d * C : a.partial + (size_t(range) * 2 + slot) * d * C;
    constexpr int NG = MT * RT;
    auto ef_load = [&](int g, float (&ev)[16]) {
      const int mt = g / RT, rt = g - mt * RT;
      const int row = mt * kTile + l32, rowc = row < d ? row : d - 1;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = rt * kTile + acc_row(v, h);
        if constexpr (kRegK)
          ev[v] = sEF[rowc * S.estride + r];  // zero beyond R
        else
          ev[v] = a.EF[rowc * R + (r < R ? r : R - 1)];
      }
    };
    f32x16 z = f32x16{};
    auto ef_mfma = [&](int g, const float (&ev)[16]) {
      const int mt = g / RT, rt = g - mt * RT;
      const int row = mt * kTile + l32;
      if (rt == 0) z = f32x16{};
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = rt * kTile + acc_row(v, h);
        z = mfma32((row < d && r < R) ? ev[v] : 0.f, acc[rt][v], z);
      }
      if (rt == RT - 1 && cvalid) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = mt * kTile + acc_row(v, h);
          if (m < d) dst[size_t(m) * C + c] = z[v];
        }
      }
    };
    float ev0[16], ev1[16];
    ef_load(0, ev0);
#pragma unroll
    for (int g = 0; g < NG; g += 2) {
      if (g + 1 < NG) ef_load(g + 1, ev1);
      __builtin_amdgcn_sched_barrier(0);
      ef_mfma(g, ev0);
      __builtin_amdgcn_sched_barrier(0);
      if (g + 1 < NG) {
        if (g + 2 < NG) ef_load(g + 2, ev0);
        __builtin_amdgcn_sched_barrier(0);
        ef_mfma(g + 1, ev1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x16{};
  };

  // B operand of K-step j of one edge: x[row][2j + h][c].  The gathered row
  // is wave-uniform, so the row base lives in scalar registers and each load
  // takes one 32-bit lane offset.  The loads are unconditional with clamped
  // addresses and no select on the value, so nothing forces a wait before
  // the operand is used one edge later: the pad row (2j + h == d) meets an
  // all-zero K row, and a lane with c >= C only feeds result column c, which
  // is never stored.
  const uint32_t c_ld = cvalid ? c : C - 1;
  auto load_edge = [&](int row, float (&b)[DH]) {
    const char* p = reinterpret_cast<const char*>(feat + size_t(row) * (d * C));
#pragma unroll
    for (int j = 0; j < DH; ++j) {
      const uint32_t k = 2 * j + h < d ? 2 * j + h : d - 1;
      b[j] = *reinterpret_cast<const float*>(p + (k * uint32_t(C) + c_ld) * 4u);
    }
  };
  auto load_g = [&](int e, float (&g)[RT]) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) g[rt] = sG[e * Rp + rt * kTile + l32];
  };
  auto edge_mfma = [&](const float (&g)[RT], const float (&b)[DH]) {
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

  int cur = -1;           // segment in the accumulators
  bool first_seg = true;  // cur is the range's first segment
  int first_partial = 0, last_partial = 0;
  for (int cb = e_lo; cb < e_hi; cb += chunk) {
    const int n = min(chunk, e_hi - cb);
    __syncthreads();  // factors staged / previous chunk consumed
    // wave 0, one lane per edge: gathered row, unit direction and length,
    // and the segment starts (a key differing from the previous edge's, and
    // the range's first edge)
    if (wave == 0) {
      const int t = lane;
      int key = -1;
      if (t < n) {
        const int eid = a.perm[cb + t];
        sIdx[t] = a.gather[eid];
        key = a.key[eid];
        const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
        const float len = sqrtf(vx * vx + vy * vy + vz * vz);
        const float inv = 1.f / len;
        sVec[t] = make_float4(vx * inv, vy * inv, vz * inv, len);
      }
      int prev = __shfl_up(key, 1);
      if (t == 0) prev = cb > 0 ? a.key[a.perm[cb - 1]] : -1;
      const int last_key = __shfl(key, n - 1);
      const bool start = t < n && (key != prev || (cb == e_lo && t == 0));
      const unsigned long long m = __ballot(start);
      if (start) {
        const int pos = __popcll(m & ((1ull << t) - 1));
        sBnd[pos] = t;
        sBndKey[pos] = key;
      }
      if (t == 0) {
        sMeta[0] = __popcll(m);
        sMeta[1] = cb == e_lo && cb > 0 && key == prev;
        sMeta[2] = cb + n == e_hi && e_hi < a.E && a.key[a.perm[e_hi]] == last_key;
      }
    }
    __syncthreads();
    // harmonics: one thread per (edge, order m) column; radial basis: one
    // thread per (edge, function)
    for (int t = tid; t < n * (L + 1); t += blockDim.x) {
      const int e = t / (L + 1), m = t - e * (L + 1);
      const float4 u = sVec[e];
      sh_unit_column(L, m, u.x, u.y, u.z, sY + e * d);
    }
    for (int t = tid; t < n * nr; t += blockDim.x) {
      const int e = t / nr, q = t - e * nr;
      sPhi[t] = radial_phi(sVec[e].w, q, a.sigma);
    }
    __syncthreads();
    // g = (Y B) * (Phi Wrad) for the chunk's edges (rows) and all ranks
    // (columns): two small MFMA GEMMs per 32x32 tile, one rank tile per wave.
    // Rows beyond n hold zeros (their A operand is masked) and are never read.
    const int n_et = (n + kTile - 1) / kTile;
    for (int item = wave; item < n_et * RT; item += waves) {
      const int et = item / RT, rt = item - et * RT;
      const int er = et * kTile + l32;  // this lane's edge row
      const bool row_ok = er < n;
      f32x16 Tr = f32x16{}, Ty = f32x16{};
#pragma unroll 1
      for (int s2 = 0; s2 < (nr + 1) / 2; ++s2) {
        const int q = 2 * s2 + h;
        const float av = (row_ok && q < nr) ? sPhi[er * nr + q] : 0.f;
        const float bv = q < nr ? sBE[(d + q) * Rp + rt * kTile + l32] : 0.f;
        Tr = mfma32(av, bv, Tr);
      }
#pragma unroll
      for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
        const int k = 2 * s2 + h;
        const float av = (row_ok && k < d) ? sY[er * d + k] : 0.f;
        const float bv = k < d ? sBE[k * Rp + rt * kTile + l32] : 0.f;
        Ty = mfma32(av, bv, Ty);
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) sG[(et * kTile + acc_row(v, h)) * Rp + rt * kTile + l32] = Tr[v] * Ty[v];
    }
    __syncthreads();

    const int nb = __builtin_amdgcn_readfirstlane(sMeta[0]);
    if (cb == e_lo) first_partial = __builtin_amdgcn_readfirstlane(sMeta[1]);
    if (cb + n == e_hi) last_partial = __builtin_amdgcn_readfirstlane(sMeta[2]);
    int bi = 0;
    int next = nb > 0 ? __builtin_amdgcn_readfirstlane(sBnd[0]) : n;
    // The chunk in pieces that each lie in one segment; the segment in the
    // accumulators is closed where the next one starts, before any operand
    // of the next piece is loaded.
    for (int e = 0; e < n;) {
      if (e == next) {
        if (cur >= 0) {
          finish(cur, first_seg && first_partial ? 0 : -1);
          first_seg = false;
        }
        cur = __builtin_amdgcn_readfirstlane(sBndKey[bi]);
        ++bi;
        next = bi < nb ? __builtin_amdgcn_readfirstlane(sBnd[bi]) : n;
      }
      const int pe = next;
      // Two operand buffers used alternately: the loads of edge f+1 (its
      // feature rows and g) are issued before the MFMAs of edge f, and the
      // gathered row of each edge is read from LDS one edge earlier still,
      // so no wait falls between the MFMA chains of consecutive edges; the
      // scheduling barriers keep the compiler from sinking the loads next to
      // their use.
      float b0[DH], b1[DH], g0[RT], g1[RT];
      load_edge(__builtin_amdgcn_readfirstlane(sIdx[e]), b0);
      load_g(e, g0);
      int row_a = sIdx[e + 1 < pe ? e + 1 : e];
      int f = e;
      for (; f + 1 < pe; f += 2) {
        load_edge(__builtin_amdgcn_readfirstlane(row_a), b1);
        load_g(f + 1, g1);
        const int f2 = f + 2 < pe ? f + 2 : f + 1, f3 = f + 3 < pe ? f + 3 : f2;  // past the end: reloads, unused
        const int row_b = sIdx[f2];
        __builtin_amdgcn_sched_barrier(0);
        edge_mfma(g0, b0);
        __builtin_amdgcn_sched_barrier(0);
        load_edge(__builtin_amdgcn_readfirstlane(row_b), b0);
        load_g(f2, g0);
        row_a = sIdx[f3];
        __builtin_amdgcn_sched_barrier(0);
        edge_mfma(g1, b1);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (f < pe) edge_mfma(g0, b0);
      e = pe;
    }
  }
  if (cur >= 0) finish(cur, first_seg && first_partial ? 0 : (last_partial ? 1 : -1));
}

// Edge chunk of a block: the largest power of two <= 64 (at least 8) whose
// LDS fits the block's share of the CU (160 KB over the blocks per CU).
inline int edge_chunk(int L, int RT, int n_radial) {
  const int d = (L + 1) * (L + 1);
  const int budget = 160 * 1024 / edge_waves_per_eu(L, RT);
  int chunk = 64;
  while (chunk > 8 && edge_smem(RT, d, n_radial, chunk).floats * 4 > budget) chunk >>= 1;
  return chunk;
}

template <int L, int RT>
hipError_t launch_l_rt(const EdgeArgs& a, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const int ntiles = (a.C + kTile - 1) / kTile;
  const int waves = ntiles < kMaxWavesPerBlock ? ntiles : kMaxWavesPerBlock;
  const int n_cgrp = (ntiles + waves - 1) / waves;
  if (a.E > 0) {
    const int chunk = edge_chunk(L, RT, a.n_radial);
    const size_t lds = size_t(edge_smem(RT, d, a.n_radial, chunk).floats) * 4;
    auto k = k_cp_edge<L, RT>;
    hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    k<<<dim3(a.n_range * n_cgrp), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  }
  return hipGetLastError();
}

template <int L>
hipError_t launch_cp_edge_l(const EdgeArgs& a, hipStream_t s) {
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

}  // namespace edge_detail

}  // namespace tdn
