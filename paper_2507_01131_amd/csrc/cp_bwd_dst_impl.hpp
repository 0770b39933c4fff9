// Backward of the CP tensor-product layer with respect to the edge vectors,
// direct form (used for d > 32; d <= 32 takes the factored forms in
// cp_bwd_dst2_impl.hpp and cp_bwd_sg_impl.hpp).
//
// With Gz = grad_out W^T and Gh_t = D^T Gz[t] (per destination node, [R, C]),
// the cotangent of g_e (eq. approximate, Sec. 3.1) is
//   dg_e[r] = sum_c Gh_t[r, c] (A^T x[s_e])[r, c] = sum_k A[k, r] P_e[k, r],
//   P_e = x[s_e] Gh_t^T   ([d, R], contraction over the C channels)
// and then  dv = dg * rho,  drho = dg * v,  dY = B dv,  dphi = Wrad drho,
//   grad r_e = J_Y(r_e)^T dY + (sum_q dphi_q phi'_q(|r_e|)) r_e/|r_e|.
//
// One workgroup per destination segment; each wave takes one 32-row k tile
// and a pair of 32-rank tiles.  Each wave forms its two Gh^T tiles once
// (fp32 MFMA, K = d); in accumulator layout
// lane l holds Gh^T[ct*32 + acc_row(v, l/32)][rt*32 + l%32], so registers
// 8q .. 8q+7 are the B operand of one 32x32x16 step of P_e = x[s_e] Gh^T
// that contracts channels ct*32 + 16q + 8(i/4) + 4h + i%4 (i = 0..7) in
// half-wave h.  The x operand comes in that channel order from the xd layout
// (launch_direct_layout): per edge and channel tile one 16-byte load per
// k tile, K-step and part, one channel tile ahead.
//
// Arithmetic.  fp32 problems: x[n] 2^-e_n and the wave's Gh^T tiles scaled by
// a power of two (largest magnitude to [2^13, 2^14)) are split into two fp16
// parts each (to 2^-22) and P_e sums the three part products with i + j <= 3
// on v_mfma_f32_32x32x16_f16, fp32 accumulation; dg carries both scales back
// (exactly).  bf16 problems: x is bf16 and Gh^T is rounded to bf16, one
// product on v_mfma_f32_32x32x16_bf16.  dg over the wave's k tile is a
// 32-term dot product with A (from LDS, in accumulator order) plus one
// cross-half add; the two k tiles' parts are added in a fixed order.
//
// Per chunk of 16 edges the small products v = Y B, rho = Phi Wrad, dY =
// dV B^T and dphi = dRho Wrad^T run on 16x16x4 fp32 MFMA (the chunk's edges
// are one tile's rows), dY and dphi reading B and Wrad from transposed
// copies that the launch writes (coalesced operand loads).
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace bwd_detail {

constexpr int kChunk = 16;  // edges per chunk: the rows of one 16x16x4 MFMA tile
constexpr int kPy = 80;     // per edge: 64 dY columns (k < d <= 64) and 16 dphi columns (n_radial <= 16)

struct DstSmem {
  int Rp, Rs, off_b, off_v, off_rho, off_dg, off_y, off_phi, off_dy, off_dphi, off_j, off_idx, off_sc, floats;
};

__host__ __device__ inline DstSmem dst_smem(int RT, int MT, int d, int n_radial, int C) {
  DstSmem s{};
  s.Rp = RT * kTile;
  s.Rs = s.Rp + 4;  // row stride of v, rho and dg: the dY products read columns of them
  int o = 0;
  s.off_b = o;  // A in accumulator order: [MT][RT][4][64 lanes] x float4
  o += MT * RT * 4 * kWave * 4;
  s.off_v = o;
  o += kChunk * s.Rs;
  s.off_rho = o;
  o += kChunk * s.Rs;
  s.off_dg = o;
  o += MT * kChunk * s.Rs;
  if (o < s.off_v + d * C) o = s.off_v + d * C;  // the region also holds Gz[seg] while Gh^T is formed
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
  s.off_sc = o;
  o += kChunk;
  s.floats = o;
  return s;
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool BF>
__device__ __forceinline__ f32x16 mfma16(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (BF)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
}

// Waves of the workgroup: MT k tiles x ceil(RT / 2) pairs of rank tiles.
__host__ __device__ constexpr int direct_waves(int MT, int RT) { return MT * ((RT + 1) / 2); }

template <int MT, int RT, int NCT, bool BF>
__global__ __launch_bounds__(direct_waves(MT, RT)* kWave) void k_bwd_dst(BwdDstArgs a) {
  constexpr int P = BF ? 1 : 2;  // 16-bit parts per operand value
  constexpr int NS = 2 * NCT;    // K-steps of 16 channels (xd blocks per part)
  constexpr int NW = direct_waves(MT, RT);
  extern __shared__ float smem[];
  const DstSmem S = dst_smem(RT, MT, a.d, a.n_radial, a.C);
  constexpr int Rp = RT * kTile, Rs = Rp + 4;
  f32x4* sAl = reinterpret_cast<f32x4*>(smem + S.off_b);
  float* sV = smem + S.off_v;
  float* sRho = smem + S.off_rho;
  float* sDG = smem + S.off_dg;  // [MT][kChunk][Rs]: dg over each k tile
  float* sY = smem + S.off_y;
  float* sPhi = smem + S.off_phi;
  float* sDY = smem + S.off_dy;
  float* sDPhi = smem + S.off_dphi;
  float* sJ = smem + S.off_j;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);
  int* sEid = sIdx + kChunk;
  float* sSc = smem + S.off_sc;  // 2^e of the edge's x row (fp32 problems)

  const int seg = xcd_remap(blockIdx.x, a.n_seg);
  const int e_begin = a.offsets[seg], e_end = a.offsets[seg + 1];
  if (e_begin == e_end) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, l32 = lane & 31;
  const int g4 = lane >> 4, l16 = lane & 15;  // 16x16x4 MFMA operand coordinates
  const int d = a.d, C = a.C, nr = a.n_radial, R = a.R;
  // the P_e tiles of this wave: k tile kt, rank tiles 2j and 2j + 1
  const int kt = wave % MT, pj = wave / MT;
  int rtw[2];
  rtw[0] = 2 * pj;
  rtw[1] = 2 * pj + 1 < RT ? 2 * pj + 1 : 2 * pj;  // a lone last tile runs twice; the copy is dropped
  const bool has2 = 2 * pj + 1 < RT;

  // sAl[((kt*RT + rt)*4 + qq)*64 + lane'] = A[kt*32 + acc_row(4 qq + i, h')][rt*32 + l32']:
  // the A values lane' weighs its P accumulators with, one 16-byte read per quarter
  for (int t = tid; t < MT * RT * 4 * kWave; t += blockDim.x) {
    const int ln = t % kWave, q4 = t / kWave;
    const int qq = q4 % 4, krt = q4 / 4, rt = krt % RT, kt2 = krt / RT;
    const int r = rt * kTile + (ln & 31);
    f32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = kt2 * kTile + acc_row(4 * qq + i, ln >> 5);
      v[i] = (k < d && r < R) ? a.A[k * R + r] : 0.f;
    }
    sAl[t] = v;
  }

  // Gz[seg] staged in LDS ([d][C], coalesced float4 loads) in the v/rho/dg
  // region, which the chunk loop uses only after its first barrier
  float* sGzf = sV;
  {
    const f32x4* g4 = reinterpret_cast<const f32x4*>(a.Gz + size_t(seg) * d * C);
    for (int i = tid; i < d * C / 4; i += blockDim.x) reinterpret_cast<f32x4*>(sGzf)[i] = g4[i];
  }
  __syncthreads();
  // Gh^T tiles of the wave's two rank tiles, each scaled by its own power of
  // two (fp32 problems) and split: ghp[t][ct][q][p].  One D value per lane
  // and step feeds all channel tiles.
  u32x4 ghp[2][NCT][2][P];
  float gh_unscale[2] = {1.f, 1.f};
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int r = rtw[t] * kTile + l32;
    f32x16 gh[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) gh[ct] = f32x16{};
#pragma unroll 5
    for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
      const int k = 2 * s2 + h;
      const float bv = (k < d && r < R) ? a.D[k * R + r] : 0.f;
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int cc = ct * kTile + l32;
        const float av = (k < d && cc < C) ? sGzf[k * C + cc] : 0.f;
        gh[ct] = mfma32(av, bv, gh[ct]);
      }
    }
    float sc = 1.f;
    if constexpr (!BF) {
      float mx = 0.f;
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(gh[ct][v]));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const int e = f16_split_exponent(mx);
      sc = ldexpf(1.f, -e);
      gh_unscale[t] = ldexpf(1.f, e);
    }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        uint32_t w[P][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v0 = gh[ct][8 * q + 2 * i] * sc, v1 = gh[ct][8 * q + 2 * i + 1] * sc;
          if constexpr (BF)
            w[0][i] = pack_bf16x2_rne(v0, v1);
          else
            split_f16x2_pair(v0, v1, w[0][i], w[1][i]);
        }
#pragma unroll
        for (int p = 0; p < P; ++p) ghp[t][ct][q][p] = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
      }
  }

  // x operand of channel tile ct for an edge row: xb[q][p] is lane (h, row
  // kt*32 + l32) of block (part p, K-step 2ct + q) of xd.  Rows past d are
  // clamped (their P rows meet A = 0).
  const char* __restrict__ xd = static_cast<const char*>(a.xc);
  const size_t node_bytes = size_t(P) * NS * 2 * d * 16;
  const int kr = kt * kTile + l32 < d ? kt * kTile + l32 : d - 1;
  const uint32_t lane_off = uint32_t((h * d + kr) * 16);
  auto load_step = [&](int row, int ct, u32x4 (&xb)[2][P]) {
    const char* base = xd + size_t(row) * node_bytes;
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int p = 0; p < P; ++p)
        xb[q][p] = *reinterpret_cast<const u32x4*>(base + lane_off + uint32_t((p * NS + 2 * ct + q) * 2 * d * 16));
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
      const int row = a.src[eid];
      sEid[t] = eid;
      sIdx[t] = row;
      sSc[t] = BF ? 1.f : a.x_scale[row];
    }
    __syncthreads();
    // v = Y B and rho = Phi Wrad on 16x16x4 fp32 MFMA (rows: the chunk's 16
    // edges; columns: two 16-rank halves of one 32-rank tile per wave at a
    // time; contraction over k < d, then over the radial functions)
    for (int rt = wave; rt < RT; rt += NW) {
      f32x4 tv[2] = {f32x4{}, f32x4{}}, tr[2] = {f32x4{}, f32x4{}};
#pragma unroll 4
      for (int s4 = 0; s4 < (d + 3) / 4; ++s4) {
        const int k = 4 * s4 + g4;
        const float av = (l16 < n && k < d) ? sY[l16 * d + k] : 0.f;
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const int r = rt * kTile + 16 * c2 + l16;
          const float bv = (k < d && r < R) ? a.Bf[k * R + r] : 0.f;
          tv[c2] = mfma16f32(av, bv, tv[c2]);
        }
      }
      for (int s4 = 0; s4 < (nr + 3) / 4; ++s4) {
        const int q = 4 * s4 + g4;
        const float av = (l16 < n && q < nr) ? sPhi[l16 * nr + q] : 0.f;
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const int r = rt * kTile + 16 * c2 + l16;
          const float bv = (q < nr && r < R) ? a.radial_w[q * R + r] : 0.f;
          tr[c2] = mfma16f32(av, bv, tr[c2]);
        }
      }
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * g4 + i, r = rt * kTile + 16 * c2 + l16;
          if (e < n) {
            sV[e * Rs + r] = tv[c2][i];
            sRho[e * Rs + r] = tr[c2][i];
          }
        }
    }

    // P_e tiles and dg over this wave's k tile, edges in pairs so that the
    // buffer of every (edge, ct) step is a compile-time choice; an odd last
    // edge is paired with a copy of itself whose result is dropped.
    u32x4 xb0[2][P], xb1[2][P];
    f32x16 pacc[2];
    load_step(__builtin_amdgcn_readfirstlane(sIdx[0]), 0, xb0);
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
            const int nrow = __builtin_amdgcn_readfirstlane(last_ct ? sIdx[half_e ? e2 : e1] : sIdx[e]);
            const int nct = last_ct ? 0 : ct + 1;
            if ((s + 1) & 1)
              load_step(nrow, nct, xb1);
            else
              load_step(nrow, nct, xb0);
          }
          __builtin_amdgcn_sched_barrier(0);
          if (ct == 0) {
            pacc[0] = f32x16{};
            pacc[1] = f32x16{};
          }
#pragma unroll
          for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
              const u32x4(&xq)[P] = s & 1 ? xb1[q] : xb0[q];
              const u32x4(&gq)[P] = ghp[t][ct][q];
              if constexpr (!BF) {
                pacc[t] = mfma16<BF>(xq[1], gq[0], pacc[t]);
                pacc[t] = mfma16<BF>(xq[0], gq[1], pacc[t]);
              }
              pacc[t] = mfma16<BF>(xq[0], gq[0], pacc[t]);
            }
          __builtin_amdgcn_sched_barrier(0);
          if (ct + 1 == NCT && (half_e == 0 || e1 != e0)) {
            const float sc = sSc[e];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
              float part = 0.f;
#pragma unroll
              for (int qq = 0; qq < 4; ++qq) {
                const f32x4 av = sAl[((kt * RT + rtw[t]) * 4 + qq) * kWave + lane];
#pragma unroll
                for (int i = 0; i < 4; ++i) part += av[i] * pacc[t][4 * qq + i];
              }
              part += __shfl_xor(part, 32);
              if (h == 0 && (t == 0 || has2))
                sDG[(kt * kChunk + e) * Rs + rtw[t] * kTile + l32] = part * (sc * gh_unscale[t]);
            }
          }
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < n * Rp; i += blockDim.x) {
      const int e = i / Rp, r = i - e * Rp, j = e * Rs + r;
      float dg = sDG[j];
#pragma unroll
      for (int k2 = 1; k2 < MT; ++k2) dg += sDG[k2 * kChunk * Rs + j];
      const float dv = dg * sRho[j], drho = dg * sV[j];
      sV[j] = dv;
      sRho[j] = drho;
      if (a.drho && r < R) a.drho[size_t(sEid[e]) * R + r] = drho;  // for the radial-weight gradient
    }
    __syncthreads();
    // dY = dV B^T (columns k < d <= 64: four 16-column tiles) and dphi =
    // dRho Wrad^T (columns q < n_radial <= 16: one tile) on 16x16x4 fp32
    // MFMA, contraction over one rank tile of 32 per wave (eight steps), B
    // and Wrad read from their transposed copies (a quarter-wave's operands
    // then lie in one row: coalesced loads); the per-tile partials
    // ([RT][kChunk][kPy] floats) go to the v/rho/dg region ((2 + MT) kChunk
    // Rs floats) and are summed over the rank tiles in a fixed order.
    {
      f32x4 py[5] = {f32x4{}, f32x4{}, f32x4{}, f32x4{}, f32x4{}};
      const int rt = wave;  // RT <= NW: one rank tile per wave at most
      const float* __restrict__ BT = a.bt;            // [R][d]
      const float* __restrict__ WT = a.bt + d * R;    // [R][n_radial]
      if (rt < RT) {
#pragma unroll 4
        for (int s4 = 0; s4 < kTile / 4; ++s4) {
          const int rr = rt * kTile + 4 * s4 + g4;
          const bool rok = rr < R;
          const float a_v = l16 < n ? sV[l16 * Rs + rr] : 0.f;
          const float a_r = l16 < n ? sRho[l16 * Rs + rr] : 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (16 * t >= d) break;
            const int k = 16 * t + l16;
            const float bv = (rok && k < d) ? BT[rr * d + k] : 0.f;
            py[t] = mfma16f32(a_v, bv, py[t]);
          }
          const float bw = (rok && l16 < nr) ? WT[rr * nr + l16] : 0.f;
          py[4] = mfma16f32(a_r, bw, py[4]);
        }
      }
      __syncthreads();  // every wave has read dv and drho
      float* sPart = sV;
      if (rt < RT) {
#pragma unroll
        for (int t = 0; t < 5; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int e = 4 * g4 + i;
            if (e < n) sPart[(rt * kChunk + e) * kPy + 16 * t + l16] = py[t][i];
          }
      }
      __syncthreads();
      for (int i = tid; i < n * kPy; i += blockDim.x) {
        const int e = i / kPy, c = i - e * kPy;
        float sum = 0.f;
        for (int w = 0; w < RT; ++w) sum += sPart[(w * kChunk + e) * kPy + c];
        if (c < 64) {
          if (c < d) sDY[e * d + c] = sum;
        } else if (c - 64 < nr) {
          sDPhi[e * nr + c - 64] = sum;
        }
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

namespace {
// out[c][r] = in[r][c] for an [rows, cols] row-major input
__global__ __launch_bounds__(256) void k_transpose(int rows, int cols, const float* __restrict__ in,
                                                   float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int c = i / rows, r = i - c * rows;
  out[i] = in[size_t(r) * cols + c];
}
}  // namespace

template <int MT, int RT, int NCT, bool BF>
hipError_t launch_k(const BwdDstArgs& a, hipStream_t s) {
  const size_t lds = size_t(dst_smem(RT, MT, a.d, a.n_radial, a.C).floats) * 4;
  if (lds > 160 * 1024 || !a.bt) return hipErrorInvalidValue;
  k_transpose<<<dim3((a.d * a.R + 255) / 256), dim3(256), 0, s>>>(a.d, a.R, a.Bf, a.bt);
  k_transpose<<<dim3((a.n_radial * a.R + 255) / 256), dim3(256), 0, s>>>(a.n_radial, a.R, a.radial_w,
                                                                           a.bt + size_t(a.d) * a.R);
  auto k = k_bwd_dst<MT, RT, NCT, BF>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(a.n_seg), dim3(direct_waves(MT, RT) * kWave), lds, s>>>(a);
  return hipGetLastError();
}

template <int MT, bool BF>
hipError_t launch_mt(const BwdDstArgs& a, hipStream_t s) {
  const int rt = (a.R + kTile - 1) / kTile;
  const int NC = bwd_direct_cpad(a.C) / kTile;
#define TDN_BWD_CASE(RTV)                                   \
  case RTV:                                                 \
    if (NC == 2) return launch_k<MT, RTV, 2, BF>(a, s);     \
    if (NC == 4) return launch_k<MT, RTV, 4, BF>(a, s);     \
    return launch_k<MT, RTV, 8, BF>(a, s);
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
