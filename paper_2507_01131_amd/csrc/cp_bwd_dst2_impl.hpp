// Destination-side backward (the edge-vector gradient) for d <= 32 through
// the factored form of dg, on 16-bit MFMA.
//
// With Gz = grad_out W^T and Gh_t = D^T Gz[t], the cotangent of g_e
// (eq. approximate, Sec. 3.1) factors as
//   dg_e[r] = sum_{k,j} S_e[k, j] A[k, r] D[j, r],   S_e = x[s_e] Gz[t]^T
// (d x d, contraction over the C channels): T_e = S_e^T A ([d, R], K = d)
// and dg_e[r] = sum_j D[j, r] T_e[j, r].  Then dv = dg * rho,
// drho = dg * v, dY = B dv, dphi = Wrad drho and
//   grad r_e = J_Y(r_e)^T dY + (sum_q dphi_q phi'_q(|r_e|)) r_e/|r_e|.
//
// Arithmetic.  fp32 problems: S_e and T_e run on v_mfma_f32_32x32x16_f16
// with both operands scaled by powers of two (x per node, Gz per segment,
// S_e per edge tile, A once: each largest magnitude to [2^13, 2^14)) and
// split into two fp16 parts (to 2^-22); the three part products with
// i + j <= 3 are summed in fp32 and dg multiplies the four scales back.
// bf16 problems: x is bf16; Gz, S_e and A are rounded to bf16, one product
// each on v_mfma_f32_32x32x16_bf16.
//
// Work decomposition.  No sum runs over edges here, so the sorted edge list
// is cut into equal ranges anywhere, several per workgroup of eight waves
// (two per SIMD), interleaved so that the workgroups of one XCD work in one
// stretch of destinations at a time.  Per chunk of up to 32 edges: harmonics
// with their Jacobian per (edge, order m) column and the radial basis per
// (edge, function); v = Y B and rho = Phi Wrad as small fp32 MFMA GEMMs; then
// the chunk in segment pieces: the piece's Gz[t] is split into LDS once, and
// each wave takes whole edges: S_e (K-steps of 16 channels; the x operand
// comes straight from global memory, laid out in MFMA operand blocks per
// node, part and K-step, one contiguous 16-byte-per-lane load per part,
// through a per-wave prefetch ring), T_e per rank tile (the accumulator
// registers of S regroup into the A operand of a 32x32x16 step, so the
// factor A is stored with the same row permutation), dg, dv and drho.  Last dY = dV B^T and dphi = dRho Wrad^T
// (fp32 MFMA) and the gradient per edge.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace bwd2_detail {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kMaxChunk = 32;
constexpr int kRing = 4;  // x slots per wave in the S loop
constexpr int kMaxRadial = 16;
constexpr int kBufferWord3 = 0x00020000;  // raw buffer resource, fourth word (gfx9 family)

// K-steps of 16 channels per ring slot: one for the two-part (fp32)
// operands, two for bf16
__host__ __device__ constexpr int dst2_kps(int P) { return P == 2 ? 1 : 2; }
// channels padded to whole ring turns
__host__ __device__ inline int dst2_cpad(int C, int P) {
  const int turn = 16 * dst2_kps(P) * kRing;
  return (C + turn - 1) / turn * turn;
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// 32x32x16 MFMA on fp16 operands (fp32 problems) or bf16 operands
template <bool BF>
__device__ __forceinline__ f32x16 mfma16(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (BF)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
}

// Contraction row of K-step q (0, 1), half h, element i of T = S^T A: the S
// rows that lane half h holds in accumulator registers 8q .. 8q+7.
__host__ __device__ constexpr int t_row(int q, int h, int i) { return 16 * q + 8 * (i / 4) + 4 * h + (i % 4); }

struct Smem {
  int Rp, bs, gzs, off_b, off_wr, off_ap, off_d, off_gz, off_v, off_rho, off_y, off_phi, off_dy, off_dphi, off_w,
      off_j, off_idx, floats;
};

// LDS regions (floats): B and Wrad rows (padded stride bs so row-wise
// operand reads across lanes hit distinct banks), the factor A parts in T
// operand order [q][rank tile][part][64 lanes] x 16 bytes, D in accumulator
// order [rank tile][4][64 lanes] x 16 bytes, the staged Gz parts
// [32 rows][gzs halves] (gzs = P*Cp + 8: rows 16 bytes apart in bank terms),
// and the chunk's v, rho, Y, Phi, dY, dPhi, Jacobian and per-edge records.
__host__ __device__ inline Smem dst2_smem(int RT, int P, int d, int n_radial, int C, int chunk, bool split) {
  Smem s{};
  s.Rp = RT * kTile;
  s.bs = s.Rp + 1;
  s.gzs = P * dst2_cpad(C, P) + 8;
  int o = 0;
  s.off_b = o;
  o += d * s.bs;
  s.off_wr = o;
  o += n_radial * s.bs;
  o = (o + 3) & ~3;
  // A, D and the staged Gz: only where the kernel runs the S/T contraction
  s.off_ap = o;
  o += split ? 0 : 2 * RT * P * kWave * 4;
  s.off_d = o;
  o += split ? 0 : kTile * s.Rp;
  s.off_gz = o;
  o += split ? 0 : kTile * s.gzs / 2;
  s.off_v = o;
  o += chunk * s.bs;
  s.off_rho = o;
  o += chunk * s.bs;
  s.off_y = o;
  o += chunk * d;
  s.off_phi = o;
  o += chunk * n_radial;
  s.off_dy = o;
  o += 2 * chunk * d;  // two rank-half partials
  s.off_dphi = o;
  o += 2 * chunk * n_radial;  // two rank-half partials
  s.off_w = o;  // the workgroup's radial-weight gradient [n_radial][Rp]
  o += n_radial * s.Rp;
  s.off_j = o;
  o += chunk * 3 * d;
  s.off_idx = o;
  o += 7 * chunk;
  s.floats = o;
  return s;
}


// SPLIT: dg of every edge comes from memory (k_bwd_dg below) instead of the
// S/T contraction here; without A, D and Gz in LDS two workgroups share a CU.
template <int L, int RT, bool BF, bool SPLIT>
__global__ __launch_bounds__(kWaves* kWave) __attribute__((amdgpu_waves_per_eu(SPLIT ? 4 : 2))) void k_bwd_dst2(
    BwdDstArgs a, int n_range, int chunk) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int P = BF ? 1 : 2;
  constexpr int KPS = dst2_kps(P);
  constexpr int Rp = RT * kTile;
  extern __shared__ float smem[];
  const Smem S = dst2_smem(RT, P, d, a.n_radial, a.C, chunk, SPLIT);
  const int bs = S.bs, gzs = S.gzs;
  float* sB = smem + S.off_b;
  float* sWr = smem + S.off_wr;
  u32x4* sAp = reinterpret_cast<u32x4*>(smem + S.off_ap);
  f32x4* sDl = reinterpret_cast<f32x4*>(smem + S.off_d);
  uint16_t* sGz = reinterpret_cast<uint16_t*>(smem + S.off_gz);
  float* sV = smem + S.off_v;
  float* sRho = smem + S.off_rho;
  float* sY = smem + S.off_y;
  float* sPhi = smem + S.off_phi;
  float* sDY = smem + S.off_dy;
  float* sDPhi = smem + S.off_dphi;
  float* sW = smem + S.off_w;
  float* sJ = smem + S.off_j;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);  // gathered row
  int* sEid = sIdx + chunk;                             // edge id
  int* sKey = sEid + chunk;                             // destination segment
  float* sVec = reinterpret_cast<float*>(sKey + chunk);  // edge vectors [chunk][3]
  float* sXs = sVec + 3 * chunk;                         // 2^e of the edge's x row (fp32 problems)
  float* sRed = smem + S.off_dy;                         // block maxima (free outside the dY phase)

  // ranges slot, slot + n_blocks, ...: at any time the workgroups of one XCD
  // work in one stretch of the destination-sorted edges, and their gathered
  // source rows overlap in that XCD's L2
  const int n_blocks = gridDim.x, per_block = n_range / n_blocks;
  const int slot = xcd_remap(blockIdx.x, n_blocks);
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform over the wave
  const int h = lane >> 5, l32 = lane & 31;
  const int C = a.C, nr = a.n_radial, R = a.R;

  // ---- factors, once per workgroup; the radial-gradient sum starts at zero
  for (int i = tid; i < (d + nr) * Rp; i += blockDim.x) {
    const int k = i / Rp, r = i - k * Rp;
    const float v = r < R ? (k < d ? a.Bf[k * R + r] : a.radial_w[(k - d) * R + r]) : 0.f;
    (k < d ? sB + k * bs : sWr + (k - d) * bs)[r] = v;
  }
  for (int i = tid; i < nr * Rp; i += blockDim.x) sW[i] = 0.f;
  // fp32 problems: the power of two 2^-e_A that puts A's largest |A| in
  // [2^13, 2^14) for its fp16 parts; dg carries 2^e_A back
  float a_sc = 1.f, a_unscale = 1.f;
  if constexpr (!BF && !SPLIT) {
    float mx = 0.f;
    for (int i = tid; i < d * R; i += blockDim.x) mx = fmaxf(mx, fabsf(a.A[i]));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if (lane == 0) sRed[wave] = mx;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, sRed[w]);
    const int e = f16_split_exponent(mx);
    a_sc = ldexpf(1.f, -e);
    a_unscale = ldexpf(1.f, e);
  }
  // sAp[((q*RT + rt)*P + p)*64 + lane'] = part p of A[t_row(q, h', i)][rt*32 + l32'], i = 0..7
  for (int t = tid; t < (SPLIT ? 0 : 2 * RT * kWave); t += blockDim.x) {
    const int ln = t % kWave, qrt = t / kWave;
    const int q = qrt / RT, rt = qrt - q * RT;
    const int r = rt * kTile + (ln & 31), hh = ln >> 5;
    uint32_t w[P][4];
#pragma unroll
    for (int p2 = 0; p2 < 4; ++p2) {
      const int k0 = t_row(q, hh, 2 * p2), k1 = t_row(q, hh, 2 * p2 + 1);
      const float v0 = (k0 < d && r < R) ? a.A[k0 * R + r] : 0.f;
      const float v1 = (k1 < d && r < R) ? a.A[k1 * R + r] : 0.f;
      if constexpr (P == 2)
        split_f16x2_pair(v0 * a_sc, v1 * a_sc, w[0][p2], w[1][p2]);
      else
        w[0][p2] = pack_bf16x2_rne(v0, v1);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) sAp[(qrt * P + p) * kWave + ln] = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
  }
  // sDl[(rt*4 + qq)*64 + lane'][i] = D[acc_row(4 qq + i, h')][rt*32 + l32']: the D
  // values lane' weighs its T accumulators with, one 16-byte read per quarter
  for (int t = tid; t < (SPLIT ? 0 : RT * 4 * kWave); t += blockDim.x) {
    const int ln = t % kWave, rq = t / kWave;
    const int rt = rq / 4, qq = rq % 4;
    const int r = rt * kTile + (ln & 31);
    f32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = acc_row(4 * qq + i, ln >> 5);
      v[i] = (j < d && r < R) ? a.D[j * R + r] : 0.f;
    }
    sDl[t] = v;
  }

  float gz_unscale = 1.f;  // 2^e_g of the staged Gz (fp32 problems)
  // ---- per edge: S_e, T_e, dg -> dv, drho (in place in sV, sRho)
  // The x operand streams through a ring of kRing slots per wave, kRing - 1
  // slots ahead of the MFMA and on into the wave's next edge of the piece, so
  // that edge's first loads are in flight while this edge's T runs.  A slot
  // is KPS K-steps of 16 channels; the channel count is padded to whole ring
  // turns (zero channels in x and in the staged Gz), so every edge starts on
  // slot 0.  The loads are buffer loads over one node's blocks of xc: lanes of
  // rows k >= d and a missing next edge (a record of no bytes) read zeros
  // through the range check, with no branch that would drain the ring.  The
  // Gz operand is read from LDS one slot ahead.
  const int Cp = dst2_cpad(C, P), nsl = Cp / (16 * KPS);
  const char* __restrict__ xc = static_cast<const char*>(a.xc);
  const int xrow = d * P * Cp * 2;  // bytes per node
  const int xstep = 2 * d * 16;     // bytes per MFMA operand block (part, K-step)
  const uint32_t xoff = l32 < d ? uint32_t((h * d + l32) * 16) : 0x80000000u;
  const uint16_t* gzl = sGz + l32 * gzs + 8 * h;  // lane's Gz row j = l32
  auto row_rsrc = [&](int row, bool valid) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(xc) + size_t(row) * xrow, 0, valid ? xrow : 0,
                                             kBufferWord3);
  };
  auto load_slot = [&](__amdgpu_buffer_rsrc_t rs, int sl, u32x4 (&xb)[KPS][P]) {
#pragma unroll
    for (int kk = 0; kk < KPS; ++kk)
#pragma unroll
      for (int p = 0; p < P; ++p)
        xb[kk][p] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, xoff, (p * (Cp / 16) + sl * KPS + kk) * xstep, 0));
  };
  auto load_g = [&](int sl, u32x4 (&g)[KPS][P]) {
#pragma unroll
    for (int kk = 0; kk < KPS; ++kk)
#pragma unroll
      for (int p = 0; p < P; ++p) g[kk][p] = *reinterpret_cast<const u32x4*>(gzl + p * Cp + 16 * (sl * KPS + kk));
  };
  auto mma_slot = [&](const u32x4 (&xb)[KPS][P], const u32x4 (&g)[KPS][P], f32x16& Sacc) {
#pragma unroll
    for (int kk = 0; kk < KPS; ++kk) {
      const u32x4(&xp)[P] = xb[kk];
      const u32x4(&gp)[P] = g[kk];
      if constexpr (P == 2) {
        Sacc = mfma16<BF>(xp[1], gp[0], Sacc);
        Sacc = mfma16<BF>(xp[0], gp[1], Sacc);
      }
      Sacc = mfma16<BF>(xp[0], gp[0], Sacc);
    }
  };
  auto finish_edge = [&](int e, const f32x16& Sacc) {
    // S in parts, regrouped as the A operand of T's two K-steps; fp32
    // problems scale the tile by the power of two that puts its largest |S|
    // in [2^13, 2^14) first, and dg takes back all four scales
    float s_sc = 1.f, unscale = 1.f;
    if constexpr (P == 2) {
      float mx = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(Sacc[v]));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const int es = f16_split_exponent(mx);
      s_sc = ldexpf(1.f, -es);
      unscale = ldexpf(sXs[e] * gz_unscale * a_unscale, es);
    }
    u32x4 sp[2][P];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      uint32_t w[P][4];
#pragma unroll
      for (int p2 = 0; p2 < 4; ++p2) {
        const float v0 = Sacc[8 * q + 2 * p2], v1 = Sacc[8 * q + 2 * p2 + 1];
        if constexpr (P == 2)
          split_f16x2_pair(v0 * s_sc, v1 * s_sc, w[0][p2], w[1][p2]);
        else
          w[0][p2] = pack_bf16x2_rne(v0, v1);
      }
#pragma unroll
      for (int p = 0; p < P; ++p) sp[q][p] = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
    }
    // the factor operands one rank tile ahead of the MFMA; D values and the
    // edge's v and rho ahead of the tile's MFMA
    u32x4 ap[2][2][P];
    auto load_a = [&](int rt, int b) {
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int p = 0; p < P; ++p) ap[b][q][p] = sAp[((q * RT + rt) * P + p) * kWave + lane];
    };
    load_a(0, 0);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (rt + 1 < RT) load_a(rt + 1, (rt + 1) & 1);
      f32x4 dl[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) dl[qq] = sDl[(rt * 4 + qq) * kWave + lane];
      const float v_e = sV[e * bs + rt * kTile + l32], rho_e = sRho[e * bs + rt * kTile + l32];
      f32x16 T = f32x16{};
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const u32x4(&a_)[P] = ap[rt & 1][q];
        if constexpr (P == 2) {
          T = mfma16<BF>(sp[q][1], a_[0], T);
          T = mfma16<BF>(sp[q][0], a_[1], T);
        }
        T = mfma16<BF>(sp[q][0], a_[0], T);
      }
      // dg[r] = sum_j D[j, r] T[j, r]: this lane's 16 rows, then the other half
      float part = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) part += dl[v / 4][v % 4] * T[v];
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(part), __float_as_uint(part), false, false);
      part = (__uint_as_float(sw[0]) + __uint_as_float(sw[1])) * unscale;
      if (h == 0) {
        const int r = rt * kTile + l32;
        sV[e * bs + r] = part * rho_e;  // dv
        sRho[e * bs + r] = part * v_e;  // drho
      }
    }
  };

  // this wave's edges of the piece [p0, p1): p0 + wave, p0 + wave + kWaves, ...
  auto wave_edges = [&](int p0, int p1) {
    int e = p0 + wave;
    if (e >= p1) return;
    u32x4 ring[kRing][KPS][P];
    u32x4 g2[2][KPS][P];
    __amdgpu_buffer_rsrc_t rs = row_rsrc(__builtin_amdgcn_readfirstlane(sIdx[e]), true);
#pragma unroll
    for (int j = 0; j + 1 < kRing; ++j) load_slot(rs, j, ring[j]);
    load_g(0, g2[0]);
    for (; e < p1; e += kWaves) {
      const bool has_next = e + kWaves < p1;
      const __amdgpu_buffer_rsrc_t nrs =
          row_rsrc(__builtin_amdgcn_readfirstlane(sIdx[has_next ? e + kWaves : e]), has_next);
      f32x16 Sacc = f32x16{};
      for (int u0 = 0; u0 < nsl; u0 += kRing) {
#pragma unroll
        for (int j = 0; j < kRing; ++j) {
          const int fs = u0 + j + kRing - 1;  // slot loaded now, into ring[(j + kRing - 1) % kRing]
          load_slot(fs < nsl ? rs : nrs, fs < nsl ? fs : fs - nsl, ring[(j + kRing - 1) % kRing]);
          const int gs = u0 + j + 1;
          load_g(gs < nsl ? gs : 0, g2[(j + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
          mma_slot(ring[j], g2[j & 1], Sacc);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      finish_edge(e, Sacc);
      rs = nrs;
    }
  };

  // The workgroup's chunks: ranges pc = 0 .. per_block - 1, each in chunks
  // of up to `chunk` edges.  The records (edge id, source, destination,
  // edge vector) of the next chunk are fetched by threads t < chunk while
  // this chunk runs: the edge ids during the geometry, the rest during the
  // edge work, so no chunk starts on a chain of dependent global loads.
  // range pc * n_blocks + slot of this workgroup: [range_lo(pc), range_hi(pc))
  auto range_lo = [&](int pc) { return int(int64_t(pc * n_blocks + slot) * a.E / n_range); };
  auto range_hi = [&](int pc) { return int(int64_t(pc * n_blocks + slot + 1) * a.E / n_range); };
  struct EdgeRec {
    int eid, src, dst;
    float vx, vy, vz, xs;
  };
  auto load_rec = [&](int eid, int cnt, EdgeRec& r) {
    if (tid < cnt) {
      r.eid = eid;
      r.src = a.src[eid];
      r.dst = a.dst[eid];
      r.vx = a.edge_vec[3 * eid];
      r.vy = a.edge_vec[3 * eid + 1];
      r.vz = a.edge_vec[3 * eid + 2];
      r.xs = BF ? 1.f : a.x_scale[r.src];
    }
  };
  int pc = 0, cb = range_lo(0), hi = range_hi(0);
  EdgeRec rec{};
  {
    const int n0 = min(chunk, hi - cb);
    load_rec(tid < n0 ? a.perm[cb + tid] : 0, n0, rec);
  }
  int cur = -1;  // segment whose Gz parts are in sGz
  for (;;) {
    {
      const int n = min(chunk, hi - cb);
      int npc = pc, ncb = cb + chunk, nhi = hi;
      if (ncb >= hi) {
        npc = pc + 1;
        ncb = npc < per_block ? range_lo(npc) : 0;
        nhi = npc < per_block ? range_hi(npc) : 0;
      }
      const int nn = npc < per_block ? min(chunk, nhi - ncb) : 0;
      __syncthreads();  // factors staged / previous chunk consumed
      if (tid < n) {
        sEid[tid] = rec.eid;
        sIdx[tid] = rec.src;
        sKey[tid] = rec.dst;
        sVec[3 * tid] = rec.vx;
        sVec[3 * tid + 1] = rec.vy;
        sVec[3 * tid + 2] = rec.vz;
        sXs[tid] = rec.xs;
      }
      const int next_eid = tid < nn ? a.perm[ncb + tid] : 0;
      __syncthreads();
      // ---- geometry: harmonics and Jacobian per (edge, order m) column,
      // radial basis per (edge, function)
      for (int t = tid; t < n * (L + 1); t += blockDim.x) {
        const int e = t / (L + 1), m = t - e * (L + 1);
        const float vx = sVec[3 * e], vy = sVec[3 * e + 1], vz = sVec[3 * e + 2];
        const float inv = 1.f / sqrtf(vx * vx + vy * vy + vz * vz);
        sh_unit_jacobian_column(L, m, vx * inv, vy * inv, vz * inv, inv, sY + e * d, sJ + e * 3 * d);
      }
      for (int t = tid; t < n * nr; t += blockDim.x) {
        const int e = t / nr, q = t - e * nr;
        const float vx = sVec[3 * e], vy = sVec[3 * e + 1], vz = sVec[3 * e + 2];
        sPhi[t] = radial_phi(sqrtf(vx * vx + vy * vy + vz * vz), q, a.sigma);
      }
      __syncthreads();
      // ---- v = Y B, rho = Phi Wrad (rows: edges, columns: ranks), fp32 MFMA
      // (fully unrolled: every LDS operand read is issued ahead of the chain)
      for (int item = wave; item < 2 * RT; item += kWaves) {
        const int rt = item >> 1;
        const bool is_v = (item & 1) == 0;
        f32x16 T = f32x16{};
        if (is_v) {
#pragma unroll
          for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
            const int k = 2 * s2 + h;
            const float av = (l32 < n && k < d) ? sY[l32 * d + k] : 0.f;
            const float bv = k < d ? sB[k * bs + rt * kTile + l32] : 0.f;
            T = mfma32(av, bv, T);
          }
        } else {
#pragma unroll
          for (int s2 = 0; s2 < kMaxRadial / 2; ++s2) {
            if (2 * s2 < nr) {
              const int q = 2 * s2 + h;
              const float av = (l32 < n && q < nr) ? sPhi[l32 * nr + q] : 0.f;
              const float bv = q < nr ? sWr[q * bs + rt * kTile + l32] : 0.f;
              T = mfma32(av, bv, T);
            }
          }
        }
        float* dstp = is_v ? sV : sRho;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int e = acc_row(v, h);
          if (e < n) dstp[e * bs + rt * kTile + l32] = T[v];
        }
      }
      EdgeRec next{};
      load_rec(next_eid, nn, next);
      if constexpr (SPLIT) {
        // dg of the chunk's edges (sorted positions cb ..): dv, drho in place
        // (the loads issued together, then applied)
        constexpr int kDgPer = kMaxChunk * Rp / (kWaves * kWave);
        float g[kDgPer];
#pragma unroll
        for (int u = 0; u < kDgPer; ++u) {
          const int i = tid + u * kWaves * kWave;
          g[u] = i < n * R ? a.dg[size_t(cb) * R + i] : 0.f;
        }
        __syncthreads();  // v/rho written
#pragma unroll
        for (int u = 0; u < kDgPer; ++u) {
          const int i = tid + u * kWaves * kWave;
          if (i < n * R) {
            const int e = i / R, r = i - e * R;
            const float v = sV[e * bs + r], rho = sRho[e * bs + r];
            sV[e * bs + r] = g[u] * rho;
            sRho[e * bs + r] = g[u] * v;
          }
        }
      }
      // ---- the chunk in segment pieces
      for (int p0 = 0; p0 < (SPLIT ? 0 : n);) {
        __syncthreads();  // v/rho written; the previous piece's edges done with sGz
        const int seg = __builtin_amdgcn_readfirstlane(sKey[p0]);
        int p1 = p0 + 1;
        while (p1 < n && sKey[p1] == seg) ++p1;
        p1 = __builtin_amdgcn_readfirstlane(p1);
        if (seg != cur) {
          // fp32 problems: Gz[seg] scaled by the power of two that puts its
          // largest magnitude in [2^13, 2^14)
          float g_sc = 1.f;
          if constexpr (P == 2) {
            float mx = 0.f;
            for (int i = tid; i < d * C; i += blockDim.x) mx = fmaxf(mx, fabsf(a.Gz[size_t(seg) * d * C + i]));
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
            if (lane == 0) sRed[wave] = mx;
            __syncthreads();
            mx = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, sRed[w]);
            const int eg = f16_split_exponent(mx);
            g_sc = ldexpf(1.f, -eg);
            gz_unscale = ldexpf(1.f, eg);
          }
          // Gz[seg] rows j < 32 in parts, zero from row d and from channel C:
          // one thread per pair of channels
          for (int i = tid; i < kTile * (Cp / 2); i += blockDim.x) {
            const int j = i / (Cp / 2), c2 = 2 * (i - j * (Cp / 2));
            float2 g = make_float2(0.f, 0.f);
            if (j < d && c2 < C) g = *reinterpret_cast<const float2*>(a.Gz + (size_t(seg) * d + j) * C + c2);
            uint32_t w[2];
            if constexpr (P == 2)
              split_f16x2_pair(g.x * g_sc, g.y * g_sc, w[0], w[1]);
            else
              w[0] = pack_bf16x2_rne(g.x, g.y);
#pragma unroll
            for (int p = 0; p < P; ++p) *reinterpret_cast<uint32_t*>(sGz + j * gzs + p * Cp + c2) = w[p];
          }
          cur = seg;
          __syncthreads();
        }
        wave_edges(p0, p1);
        p0 = p1;
      }
      __syncthreads();
      // ---- waves 0-3: dY = dV B^T (k < d) and dphi = dRho Wrad^T (q < nr),
      // K = ranks, one half of the ranks per wave, partial products summed in
      // a fixed order by the gradient below.  Waves 4-7: the radial-weight
      // gradient sum_e phi_e^T drho_e of the chunk (K = its edges) per rank
      // tile, added to the workgroup's sum in LDS.
      {
        static_assert(kWaves == 8, "two products x two rank halves, four radial-gradient waves");
        if (wave < 4) {
          const bool is_y = wave < 2;
          const int hf = wave & 1;
          const int K2 = is_y ? d : nr;
          const float* src = is_y ? sV : sRho;
          const float* fac = is_y ? sB : sWr;
          f32x16 T = f32x16{};
#pragma unroll 8
          for (int s2 = 0; s2 < RT * 8; ++s2) {
            const int r = hf * (RT * 16) + 2 * s2 + h;
            const float av = l32 < n ? src[l32 * bs + r] : 0.f;
            const float bv = l32 < K2 ? fac[l32 * bs + r] : 0.f;
            T = mfma32(av, bv, T);
          }
          float* dstp = is_y ? sDY + hf * chunk * d : sDPhi + hf * chunk * nr;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int ee = acc_row(v, h);
            if (ee < n && l32 < K2) dstp[ee * K2 + l32] = T[v];
          }
        } else {
          for (int rt = wave - 4; rt < RT; rt += 4) {
            f32x16 T = f32x16{};
#pragma unroll 4
            for (int s2 = 0; s2 < kMaxChunk / 2; ++s2) {
              const int e = 2 * s2 + h;
              const float av = (e < n && l32 < nr) ? sPhi[e * nr + l32] : 0.f;
              const float bv = e < n ? sRho[e * bs + rt * kTile + l32] : 0.f;
              T = mfma32(av, bv, T);
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int q = acc_row(v, h);
              if (q < nr) sW[q * Rp + rt * kTile + l32] += T[v];
            }
          }
        }
      }
      __syncthreads();
      // ---- the gradient per edge: sixteen threads per edge, each summing a
      // share of the degree rows and radial functions, then combined across
      // the sixteen lanes in a fixed order
      {
        constexpr int TPE = kWaves * kWave / kMaxChunk;
        const int t = tid / TPE, sub = tid % TPE;
        float gx = 0.f, gy = 0.f, gzv = 0.f, dr = 0.f;
        if (t < n) {
          const float vx = sVec[3 * t], vy = sVec[3 * t + 1], vz = sVec[3 * t + 2];
          const float rn = sqrtf(vx * vx + vy * vy + vz * vz);
          for (int k = sub; k < d; k += TPE) {
            const int i = t * d + k;
            const float dy = sDY[i] + sDY[chunk * d + i];
            gx += dy * sJ[t * 3 * d + 3 * k];
            gy += dy * sJ[t * 3 * d + 3 * k + 1];
            gzv += dy * sJ[t * 3 * d + 3 * k + 2];
          }
          for (int q = sub; q < nr; q += TPE) {
            const float u = (rn - float(q) * a.sigma) / a.sigma;
            const int i = t * nr + q;
            dr += (sDPhi[i] + sDPhi[chunk * nr + i]) * (-u / a.sigma) * sPhi[i];
          }
        }
#pragma unroll
        for (int o = TPE / 2; o > 0; o >>= 1) {
          gx += __shfl_xor(gx, o);
          gy += __shfl_xor(gy, o);
          gzv += __shfl_xor(gzv, o);
          dr += __shfl_xor(dr, o);
        }
        if (t < n && sub == 0) {
          const int eid = sEid[t];
          const float vx = sVec[3 * t], vy = sVec[3 * t + 1], vz = sVec[3 * t + 2];
          const float inv = 1.f / sqrtf(vx * vx + vy * vy + vz * vz);
          a.grad_vec[3 * eid] = gx + dr * vx * inv;
          a.grad_vec[3 * eid + 1] = gy + dr * vy * inv;
          a.grad_vec[3 * eid + 2] = gzv + dr * vz * inv;
        }
      }
      if (npc >= per_block) break;
      pc = npc;
      cb = ncb;
      hi = nhi;
      rec = next;
    }
  }
  // this workgroup's partial of the radial-weight gradient (complete since
  // the last chunk's barrier after the dY phase)
  if (a.wrad_part)
    for (int i = tid; i < nr * R; i += blockDim.x) {
      const int q = i / R, r = i - q * R;
      a.wrad_part[size_t(blockIdx.x) * nr * R + i] = sW[q * Rp + r];
    }
}

// ---- Split form: the S/T contraction alone, for channel counts whose Gz[t]
// operand fits in 64 registers (at most 8 ring slots).  Each wave takes one
// contiguous range of destination-sorted edges, with no workgroup barrier
// after the factors are staged; x[s_e] streams through the ring as in the
// range kernel, across edge boundaries, and Gz[t] comes in the same operand
// blocks (launch_direct_layout of Gz, one power-of-two scale per node for
// fp32 problems), loaded into registers when the destination changes.  The
// edge records are fetched 64 at a time, one batch ahead.  dg is stored per
// sorted edge position, dg[pos][r], for the range kernel's SPLIT mode.
constexpr int kDgWaves = 8;  // one workgroup per CU, two waves per SIMD (measured 4 % faster than two of four)
__host__ __device__ inline int dg_slots(int C, int P) { return dst2_cpad(C, P) / (16 * dst2_kps(P)); }
__host__ __device__ inline int dg_smem_floats(int RT, int P) {
  return 2 * RT * P * kWave * 4 + RT * 4 * kWave * 4 + kDgWaves;
}

constexpr int kDgMaxSlots = 8;
template <int L, int RT, bool BF>
__global__ __launch_bounds__(kDgWaves* kWave) void k_bwd_dg(BwdDstArgs a, int n_wr) {
  constexpr int d = (L + 1) * (L + 1);
  constexpr int P = BF ? 1 : 2;
  constexpr int KPS = dst2_kps(P);
  constexpr int kBatch = kWave;  // edge records per batch, one per lane
  extern __shared__ float smem[];
  u32x4* sAp = reinterpret_cast<u32x4*>(smem);
  f32x4* sDl = reinterpret_cast<f32x4*>(smem + 2 * RT * P * kWave * 4);
  float* sRed = smem + 2 * RT * P * kWave * 4 + RT * 4 * kWave * 4;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int h = lane >> 5, l32 = lane & 31;
  const int R = a.R;

  // ---- A in parts (T operand order) and D (accumulator order), as in the
  // range kernel
  float a_sc = 1.f, a_unscale = 1.f;
  if constexpr (!BF) {
    float mx = 0.f;
    for (int i = tid; i < d * R; i += blockDim.x) mx = fmaxf(mx, fabsf(a.A[i]));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if (lane == 0) sRed[wave] = mx;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kDgWaves; ++w) mx = fmaxf(mx, sRed[w]);
    const int e = f16_split_exponent(mx);
    a_sc = ldexpf(1.f, -e);
    a_unscale = ldexpf(1.f, e);
  }
  for (int t = tid; t < 2 * RT * kWave; t += blockDim.x) {
    const int ln = t % kWave, qrt = t / kWave;
    const int q = qrt / RT, rt = qrt - q * RT;
    const int r = rt * kTile + (ln & 31), hh = ln >> 5;
    uint32_t w[P][4];
#pragma unroll
    for (int p2 = 0; p2 < 4; ++p2) {
      const int k0 = t_row(q, hh, 2 * p2), k1 = t_row(q, hh, 2 * p2 + 1);
      const float v0 = (k0 < d && r < R) ? a.A[k0 * R + r] : 0.f;
      const float v1 = (k1 < d && r < R) ? a.A[k1 * R + r] : 0.f;
      if constexpr (P == 2)
        split_f16x2_pair(v0 * a_sc, v1 * a_sc, w[0][p2], w[1][p2]);
      else
        w[0][p2] = pack_bf16x2_rne(v0, v1);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) sAp[(qrt * P + p) * kWave + ln] = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
  }
  for (int t = tid; t < RT * 4 * kWave; t += blockDim.x) {
    const int ln = t % kWave, rq = t / kWave;
    const int rt = rq / 4, qq = rq % 4;
    const int r = rt * kTile + (ln & 31);
    f32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = acc_row(4 * qq + i, ln >> 5);
      v[i] = (j < d && r < R) ? a.D[j * R + r] : 0.f;
    }
    sDl[t] = v;
  }
  __syncthreads();

  // ---- this wave's range of sorted positions; neighbouring ranges on one XCD
  const int w = xcd_remap(blockIdx.x, gridDim.x) * kDgWaves + wave;
  const int e0 = int(int64_t(w) * a.E / n_wr), e1 = int(int64_t(w + 1) * a.E / n_wr);
  if (e0 >= e1) return;

  const int ns = dg_slots(a.C, P);  // 4 or 8, a multiple of kRing
  const int Cp = ns * 16 * KPS;
  const char* __restrict__ xc = static_cast<const char*>(a.xc);
  const char* __restrict__ gzc = static_cast<const char*>(a.gzc);
  const int xrow = d * P * Cp * 2;  // bytes per node, x and Gz alike
  const int xstep = 2 * d * 16;     // bytes per operand block (part, K-step)
  const uint32_t xoff = l32 < d ? uint32_t((h * d + l32) * 16) : 0x80000000u;
  auto rsrc = [&](const char* base, int row, bool valid) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base) + size_t(row) * xrow, 0, valid ? xrow : 0,
                                             kBufferWord3);
  };
  auto load_slot = [&](__amdgpu_buffer_rsrc_t rs, int sl, u32x4 (&xb)[KPS][P]) {
#pragma unroll
    for (int kk = 0; kk < KPS; ++kk)
#pragma unroll
      for (int p = 0; p < P; ++p)
        xb[kk][p] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, xoff, (p * (Cp / 16) + sl * KPS + kk) * xstep, 0));
  };

  // edge records of positions b0 .. b0 + 63, one per lane
  struct Rec {
    int src, dst;
    float xs, gs;
  };
  auto load_batch = [&](int b0) {
    Rec r{0, -1, 1.f, 1.f};
    const int pos = b0 + lane;
    if (pos < e1) {
      const int eid = a.perm[pos];
      r.src = a.src[eid];
      r.dst = a.dst[eid];
      if constexpr (!BF) {
        r.xs = a.x_scale[r.src];
        r.gs = a.gz_scale[r.dst];
      }
    }
    return r;
  };
  Rec cur = load_batch(e0), nxt = load_batch(e0 + kBatch);
  int b0 = e0;

  u32x4 ring[kRing][KPS][P];
  u32x4 g[kDgMaxSlots][KPS][P];
  int cur_t = -1;
  float g_unscale = 1.f;
  __amdgpu_buffer_rsrc_t rs = rsrc(xc, __builtin_amdgcn_readlane(cur.src, 0), true);
#pragma unroll
  for (int j = 0; j + 1 < kRing; ++j) load_slot(rs, j, ring[j]);

  for (int e = e0; e < e1; ++e) {
    const int j = e - b0;
    const int t = __builtin_amdgcn_readlane(cur.dst, j);
    const float xs = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur.xs), j));
    const bool has_next = e + 1 < e1;
    const int sn = j + 1 < kBatch ? __builtin_amdgcn_readlane(cur.src, j + 1) : __builtin_amdgcn_readlane(nxt.src, 0);
    const __amdgpu_buffer_rsrc_t nrs = rsrc(xc, has_next ? sn : 0, has_next);
    if (t != cur_t) {
      // Gz[t] into registers (rows j >= d read zeros through the range check)
      const __amdgpu_buffer_rsrc_t grs = rsrc(gzc, t, true);
#pragma unroll
      for (int sl = 0; sl < kDgMaxSlots; ++sl)
        if (sl < ns) load_slot(grs, sl, g[sl]);
      g_unscale = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur.gs), j));
      cur_t = t;
    }
    // S_e = x[s_e] Gz[t]^T over the channels, the ring kRing - 1 slots ahead
    f32x16 Sacc = f32x16{};
#pragma unroll
    for (int u = 0; u < kDgMaxSlots; ++u) {
      if (u >= ns) break;
      const int fs = u + kRing - 1;
      load_slot(fs < ns ? rs : nrs, fs < ns ? fs : fs - ns, ring[fs % kRing]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < KPS; ++kk) {
        const u32x4(&xp)[P] = ring[u % kRing][kk];
        const u32x4(&gp)[P] = g[u][kk];
        if constexpr (P == 2) {
          Sacc = mfma16<BF>(xp[1], gp[0], Sacc);
          Sacc = mfma16<BF>(xp[0], gp[1], Sacc);
        }
        Sacc = mfma16<BF>(xp[0], gp[0], Sacc);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // T_e = S_e^T A per rank tile and dg = colsum(D * T), as in the range kernel
    float s_sc = 1.f, unscale = 1.f;
    if constexpr (P == 2) {
      float mx = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(Sacc[v]));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const int es = f16_split_exponent(mx);
      s_sc = ldexpf(1.f, -es);
      unscale = ldexpf(xs * g_unscale * a_unscale, es);
    }
    u32x4 sp[2][P];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      uint32_t wd[P][4];
#pragma unroll
      for (int p2 = 0; p2 < 4; ++p2) {
        const float v0 = Sacc[8 * q + 2 * p2], v1 = Sacc[8 * q + 2 * p2 + 1];
        if constexpr (P == 2)
          split_f16x2_pair(v0 * s_sc, v1 * s_sc, wd[0][p2], wd[1][p2]);
        else
          wd[0][p2] = pack_bf16x2_rne(v0, v1);
      }
#pragma unroll
      for (int p = 0; p < P; ++p) sp[q][p] = u32x4{wd[p][0], wd[p][1], wd[p][2], wd[p][3]};
    }
    u32x4 ap[2][2][P];
    auto load_a = [&](int rt, int b) {
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int p = 0; p < P; ++p) ap[b][q][p] = sAp[((q * RT + rt) * P + p) * kWave + lane];
    };
    load_a(0, 0);
    float* dgrow = a.dg + size_t(e) * R;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (rt + 1 < RT) load_a(rt + 1, (rt + 1) & 1);
      f32x4 dl[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) dl[qq] = sDl[(rt * 4 + qq) * kWave + lane];
      f32x16 T = f32x16{};
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const u32x4(&a_)[P] = ap[rt & 1][q];
        if constexpr (P == 2) {
          T = mfma16<BF>(sp[q][1], a_[0], T);
          T = mfma16<BF>(sp[q][0], a_[1], T);
        }
        T = mfma16<BF>(sp[q][0], a_[0], T);
      }
      float part = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) part += dl[v / 4][v % 4] * T[v];
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(part), __float_as_uint(part), false, false);
      part = (__uint_as_float(sw[0]) + __uint_as_float(sw[1])) * unscale;
      const int r = rt * kTile + l32;
      if (h == 0 && r < R) dgrow[r] = part;
    }
    rs = nrs;
    if (j + 1 == kBatch) {
      cur = nxt;
      b0 += kBatch;
      nxt = load_batch(b0 + kBatch);
    }
  }
}

// Chunk: the largest of 32, 16, 8 edges whose layout fits the 160 KB of LDS.
inline int dst2_chunk(int RT, bool bf, int d, int n_radial, int C, bool split) {
  int chunk = kMaxChunk;
  while (chunk > 8 && dst2_smem(RT, bf ? 1 : 2, d, n_radial, C, chunk, split).floats * 4 > 160 * 1024) chunk >>= 1;
  return chunk;
}

// whether the split form applies: Gz[t] in at most 8 ring slots of registers
inline bool dst2_split(int C, bool bf) { return dg_slots(C, bf ? 1 : 2) <= kDgMaxSlots; }

template <int L, int RT, bool BF>
hipError_t launch_dg(const BwdDstArgs& a, hipStream_t s) {
  const size_t lds = size_t(dg_smem_floats(RT, BF ? 1 : 2)) * 4;
  auto k = k_bwd_dg<L, RT, BF>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  const int nb = device_cus();
  k<<<dim3(nb), dim3(kDgWaves * kWave), lds, s>>>(a, nb * kDgWaves);
  return hipGetLastError();
}

template <int L, int RT, bool BF>
hipError_t launch_l_rt(const BwdDstArgs& a, int n_range, hipStream_t s) {
  if (a.pieces_per_block < 1 || n_range % a.pieces_per_block) return hipErrorInvalidValue;
  constexpr int d = (L + 1) * (L + 1);
  // a Gz layout given: the split form, dg first
  const bool split = a.gzc != nullptr;
  if (split) {
    if (!a.dg || (!BF && !a.gz_scale) || !dst2_split(a.C, BF)) return hipErrorInvalidValue;
    const hipError_t e = launch_dg<L, RT, BF>(a, s);
    if (e != hipSuccess) return e;
  }
  const int chunk = dst2_chunk(RT, BF, d, a.n_radial, a.C, split);
  const size_t lds = size_t(dst2_smem(RT, BF ? 1 : 2, d, a.n_radial, a.C, chunk, split).floats) * 4;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  auto k = split ? k_bwd_dst2<L, RT, BF, true> : k_bwd_dst2<L, RT, BF, false>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(n_range / a.pieces_per_block), dim3(kWaves * kWave), lds, s>>>(a, n_range, chunk);
  return hipGetLastError();
}

template <int L, bool BF>
hipError_t launch_l(const BwdDstArgs& a, int n_range, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt<L, 1, BF>(a, n_range, s);
    case 2: return launch_l_rt<L, 2, BF>(a, n_range, s);
    case 3: return launch_l_rt<L, 3, BF>(a, n_range, s);
    case 4: return launch_l_rt<L, 4, BF>(a, n_range, s);
    case 5: return launch_l_rt<L, 5, BF>(a, n_range, s);
    case 6: return launch_l_rt<L, 6, BF>(a, n_range, s);
    case 7: return launch_l_rt<L, 7, BF>(a, n_range, s);
    case 8: return launch_l_rt<L, 8, BF>(a, n_range, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bwd2_detail

}  // namespace tdn
