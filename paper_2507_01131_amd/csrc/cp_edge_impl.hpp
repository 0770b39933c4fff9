// The CP tensor-product edge pass for fp32 features.
//
// For a destination node t with incoming edges e (eq. approximate of
// Sec. 3.1 per channel, radial weight on the rank index):
//   H_t[r, c] = sum_e g_e[r] U_e[r, c],   U_e = A^T x[s_e]   ([R, C], K = d)
// with g_e = (B^T Y_e) * rho_e.  The output factor is applied once per node,
// Z_t = D H_t, because D commutes with the sum over edges; the shared
// channel mix W (Sec. 3.2) is a separate node GEMM.  The sum over the
// segment stays in registers (no atomics, fixed order).
//
// The same kernel computes grad_x on the source-sorted graph:
//   grad_x[s] = A sum_{e: s_e = s} diag(g_e) D^T Gz[t_e],  Gz = grad_out W^T,
// i.e. the contraction uses D, the epilogue uses A and the gathered rows are
// Gz[t_e].
//
// Arithmetic.  U_e runs on fp16 MFMA (v_mfma_f32_32x32x16_f16) with fp32
// accumulation and fp32-level accuracy: every feature row and the factor are
// scaled by powers of two (exact) that put their largest magnitude in
// [2^13, 2^14), then split into two fp16 parts, a = a1 + a2 and x = x1 + x2,
// each to 2^-22 of the value; the part products are exact in fp32 and the
// three with i + j <= 3 are summed, smallest first (the dropped a2 x2 is
// below 2^-22 of |a x|).  g_e carries the two scales back, exactly.  The
// features arrive pre-split in MFMA operand blocks (launch_feature_layout),
// so one lane's operand for eight consecutive k is one 16-byte load; the
// split factor sits in LDS in MFMA operand order.  Then
// acc[r, c] += g_e[r] U_e[r, c] in fp32 on the VALU, with g read from LDS
// four rows at a time.  bf16 features take the bf16 mode described below.
//
// Work decomposition.  The sorted edge list is cut into n_range equal ranges,
// as many as the device holds workgroups at once (over the channel groups),
// so every workgroup gets the same number of edges and the launch has no
// tail; the factors are staged once per workgroup.  A workgroup covers one
// range for up to four 32-channel tiles: wave w owns channel tile w and all R
// rank rows, so its accumulators are RT = ceil(R/32) MFMA tiles of 32x32.
// Per chunk of edges the block evaluates the harmonics and radial basis, then
// g_e[r] for every rank, into LDS, and marks where in the chunk a new segment
// starts.  The MFMA loop then walks the chunk edge by edge, loading the next
// edge's feature operands one edge ahead.  Where a segment ends the epilogue
// Z = EF H runs on the accumulators and they restart from zero.  A segment
// wholly inside the range is written to its output row; the first segment of
// a range, when it began in an earlier range, and the last one, when it
// continues into a later range, go to two per-range partial slots that a
// small second kernel adds up in range order (fixed order, deterministic);
// that kernel also writes the zero rows of segments without edges.
//
// The degree L is a template parameter so that the K-block count and the
// harmonic recurrences are compile-time constants.
#pragma once

#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace edge_detail {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma_bf16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}
__device__ __forceinline__ f32x16 mfma_f16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0,
                                                0);
}

constexpr int kMaxWavesPerBlock = 4;

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return pack_bf16x2_rne(lo, hi);
}

__host__ __device__ constexpr int edge_dp(int d) { return d <= 32 ? 32 : 64; }

// K-blocks of 16 degree rows per edge
__host__ __device__ constexpr int edge_kb(int d) { return edge_dp(d) / 16; }

// Two modes of the edge contraction:
//  split (fp32 features): U_e = KF^T x from three fp16 part products, then
//    acc += g * U_e; one 32-channel tile per wave;
//  bf16 (bf16 features): the K operand g_e[r] KF[k, r] is formed in fp32 and
//    rounded to bf16, one MFMA per K-block straight into acc; two channel
//    tiles per wave (while R <= 128) so every K operand feeds two MFMAs.
// 16-bit parts per feature value and channel tiles per wave:
__host__ __device__ constexpr int edge_xp(bool bf) { return bf ? 1 : 2; }
__host__ __device__ constexpr int edge_ct(bool bf, int RT) { return bf && RT <= 4 ? 2 : 1; }

// Two waves per SIMD (two workgroups per CU) when the accumulators and the
// operands fit in 256 registers without spilling in the edge loop; one
// otherwise.  Split mode: accumulators 16 RT, two buffers of packed x words
// 2 PN, two rank tiles' factor blocks 8 PB and two U tiles 32 within 168
// (the rest holds addresses, loop state and the epilogue's temporaries).
__host__ __device__ constexpr int edge_waves_per_eu(int L, int RT, bool bf) {
  return bf ? (16 * RT * edge_ct(bf, RT) + 8 * edge_ct(bf, RT) * edge_kb((L + 1) * (L + 1)) <=
                       (edge_kb((L + 1) * (L + 1)) == 2 ? 160 : 128)
                   ? 2
                   : 1)
            : (16 * RT + 2 * pk_rows((L + 1) * (L + 1)) + 8 * pk_blocks((L + 1) * (L + 1)) + 32 <= 168 ? 2 : 1);
}
// Split mode: whether all PB RT packed factor blocks stay in registers
// across the edge loop (no factor reads from LDS per edge): up to 80
// registers at two waves per SIMD, 160 at one.
__host__ __device__ constexpr bool edge_rega(int L, int RT, bool bf) {
  return !bf && 4 * pk_blocks((L + 1) * (L + 1)) * RT <= (edge_waves_per_eu(L, RT, bf) == 2 ? 80 : 160);
}
// Split mode: rank tiles whose factor blocks stay in registers through a run
// of edges.  All of them with edge_rega; otherwise, at one wave per SIMD, as
// many as 80 registers hold (the other tiles' blocks are read from LDS per
// edge): at L = 6, R = 256 two of eight tiles, which took the slab edge pass
// from 3.18-3.21 to 3.04-3.06 ms (three tiles: 3.08; four spilled).  The LDS
// then holds only the other tiles' blocks, which at L = 6, R = 256 leaves
// room for 64-edge chunks instead of 32 (3.10-3.17 -> 2.95-2.96 ms).
__host__ __device__ constexpr int edge_reg_tiles(int L, int RT, bool bf) {
  return bf ? 0
            : edge_rega(L, RT, bf)
                  ? RT
                  : (edge_waves_per_eu(L, RT, bf) == 1
                         ? (RT < 80 / (4 * pk_blocks((L + 1) * (L + 1))) ? RT : 80 / (4 * pk_blocks((L + 1) * (L + 1))))
                         : 0);
}
// Rank tiles whose factor blocks a workgroup stages in LDS: bf16 mode all of
// them (as fp32 K values); split mode those not held in registers (all of
// them for the measurement ablation that reads them from a global copy).
__host__ __device__ constexpr int edge_lds_tiles(int L, int RT, bool bf, bool abl1 = false) {
  return bf || abl1 ? RT : RT - edge_reg_tiles(L, RT, bf);
}
// Split mode: the rank tile at position p of an edge's sequence of NRA
// register tiles (0 .. NRA-1) and RT - NRA LDS tiles (NRA .. RT-1): a
// register tile first, then the two kinds alternate while both last, so
// that the LDS reads of the next LDS tile overlap two MFMA chains instead of
// one; identity when all tiles or none are in registers.
__host__ __device__ constexpr int edge_tile_at(int p, int RT, int NRA) {
  const int NL = RT - NRA, m = NRA < NL ? NRA : NL;
  if (p < 2 * m) return (p & 1) ? NRA + p / 2 : p / 2;
  return NRA > NL ? p - m : p;
}

// Most ranges a workgroup takes: two where two workgroups share a CU (taken
// as ranges b and b + n_blocks, so that at any time an XCD's workgroups
// gather from a window of neighbouring nodes that fits its L2: one range
// per workgroup ran 1-3 % faster at the headline shape, its misses served
// from the MALL, but read five times the bytes past L2), one otherwise (the
// extra loop level costs registers that a one-wave kernel spends on
// accumulators).
__host__ __device__ constexpr int edge_max_ranges(int L, int RT, bool bf) {
  return edge_waves_per_eu(L, RT, bf) == 2 ? 2 : 1;
}

// bf16 mode: whether this lane's K factor values (KB * RT * 8 floats) stay
// in registers instead of LDS.  Never: two waves per SIMD, which the registers
// allow only with the factor in LDS, run faster (1.02 -> 0.93 ms on the bulk
// bf16 workload).
__host__ __device__ constexpr bool edge_reg_kf(int, int) { return false; }

struct EdgeSmem {
  int Rp, off_a, off_g, off_y, off_vec, off_phi, off_idx, off_sc, off_bnd, off_a2, off_al, off_t, floats;
};

// attention (ATT): most heads, and so attention weights per edge, per chunk
constexpr int kMaxHeads = 8;

// Per-wave transpose area of the split-mode segment epilogue: 32 channel rows
// of 32 ranks, row stride 36 floats (16-byte reads of eight ranks by 32
// channels then spread over all banks).
constexpr int kTrStride = 36;
constexpr int kTrFloats = kTile * kTrStride;

// LDS regions (in floats): the factor operands, split mode
// [pk_blocks(d)][a_tiles][64 lanes] x 16 bytes of fp16 (packed slots) for the
// a_tiles rank tiles read from LDS, bf16 mode
// [KB][RT][64 lanes] x 32 bytes of fp32, g for a chunk of edges (rows
// rounded up to a whole 32-row tile), harmonics, normalised edge vectors with
// their lengths, radial basis, gathered rows, the edges' operand scales, and
// the segment starts of the chunk (positions, keys, count and the two
// partial-segment flags); with t3 (the three-input product) the second node
// factor's operands in the layout of the first.  In split mode the
// epilogue's transpose areas (one per wave) share the harmonics' region:
// the harmonics are read only by the chunk's g products, which end at a
// barrier before any epilogue, and written only after the next chunk's
// first barrier.
__host__ __device__ inline EdgeSmem edge_smem(int RT, bool bf, int d, int n_radial, int chunk, bool t3, int a_tiles,
                                              bool att = false) {
  EdgeSmem s{};
  s.Rp = RT * kTile;
  int o = 0;
  s.off_a = o;
  o += bf ? edge_kb(d) * RT * 2 * kWave * 4 : pk_blocks(d) * a_tiles * kWave * 4;
  s.off_g = o;
  o += (chunk + kTile - 1) / kTile * kTile * s.Rp;
  s.off_y = o;
  o += bf ? chunk * d : (chunk * d > kMaxWavesPerBlock * kTrFloats ? chunk * d : kMaxWavesPerBlock * kTrFloats);
  o = (o + 3) & ~3;  // float4 rows
  s.off_vec = o;
  o += chunk * 4;
  s.off_phi = o;
  o += chunk * n_radial;
  s.off_idx = o;
  o += chunk;
  s.off_sc = o;
  o += chunk;
  s.off_bnd = o;
  o += 2 * chunk + 4;
  o = (o + 3) & ~3;
  s.off_a2 = o;
  if (t3) o += pk_blocks(d) * RT * kWave * 4;
  s.off_al = o;  // attention: the chunk's weights [chunk][kMaxHeads]
  if (att) o += chunk * kMaxHeads;
  s.off_t = bf ? o : s.off_y;
  s.floats = o;
  return s;
}

// ATOM (measurement ablation only): every edge is its own segment, so the
// epilogue applies EF per edge, and it adds Z into `out` with float atomics
// instead of storing the segment sums (`out` zeroed beforehand; no partial
// slots, no fix-up) -- the naive scatter-add the segmented sum replaces.
// T3 (fp32 features, forward): the three-input product of the N-input CP
// form (App. A) with the destination node's features as the third input,
//   Z_t = D (V_t * sum_e g_e * U_e),  V_t = KF2^T x[t];
// V_t is the same for every edge of the segment, so it multiplies the
// accumulated sum once, in the epilogue (also for partial segments: the
// epilogue is linear in the sum).
//
// ABL (measurement ablations, launch_cp_edge_ablation): 1 reads the packed
// factor blocks in the edge loop from a per-workgroup copy in global memory
// (written after staging) instead of registers or LDS; 2 reads the harmonics
// from a precomputed per-edge table instead of evaluating them.
// ATT (fp32 features, the attention block): every edge's message is weighted
// per head by a.alpha[sorted position][head] before the segment sum; a head
// owns C / n_heads channels, a multiple of 32, so a wave's channel tile lies
// in one head and the weight is one factor on its g values.
template <int L, int RT, bool BF, bool ATOM = false, bool T3 = false, int ABL = 0, bool ATT = false>
__global__ __launch_bounds__(kMaxWavesPerBlock* kWave)
__attribute__((amdgpu_waves_per_eu(edge_waves_per_eu(L, RT, BF)))) void k_cp_edge(EdgeArgs a, int n_cgrp, int waves,
                                                                                  int chunk) {
  constexpr int XP = edge_xp(BF);
  constexpr int CT = edge_ct(BF, RT);
  constexpr int kMaxRanges = edge_max_ranges(L, RT, BF);
  constexpr int d = (L + 1) * (L + 1);
  constexpr int DP = edge_dp(d);
  constexpr int KB = edge_kb(d);
  constexpr int Rp = RT * kTile;
  constexpr int MT = (d + kTile - 1) / kTile;
  // split mode: packed K slots (pk_rows / pk_blocks in kernels.h), PN words
  // per lane and edge loaded as PQ quads and a PT-word tail
  constexpr int PN = pk_rows(d), PB = pk_blocks(d), PQ = PN / 4, PT = PN % 4;
  extern __shared__ float smem[];
  constexpr bool kRegA = edge_rega(L, RT, BF) && ABL != 1;
  // split mode: rank tiles 0 .. NRA-1 take their factor blocks from registers
  constexpr int NRA = ABL == 1 ? 0 : edge_reg_tiles(L, RT, BF);
  constexpr int NL = edge_lds_tiles(L, RT, BF, ABL == 1);  // split mode: RT - NRA
  const EdgeSmem S = edge_smem(RT, BF, d, a.n_radial, chunk, T3, NL, ATT);
  u32x4* sA = reinterpret_cast<u32x4*>(smem + S.off_a);
  u32x4* sA2 = reinterpret_cast<u32x4*>(smem + S.off_a2);
  float4* sAf = reinterpret_cast<float4*>(smem + S.off_a);
  float* sG = smem + S.off_g;
  float* sY = smem + S.off_y;
  float4* sVec = reinterpret_cast<float4*>(smem + S.off_vec);
  float* sPhi = smem + S.off_phi;
  int* sIdx = reinterpret_cast<int*>(smem + S.off_idx);
  float* sSc = smem + S.off_sc;                          // [chunk] 2^e of the edge's operands (split mode)
  int* sBnd = reinterpret_cast<int*>(smem + S.off_bnd);  // [chunk] chunk positions where a segment starts
  int* sBndKey = sBnd + chunk;                          // [chunk] that segment
  int* sMeta = sBndKey + chunk;                         // start count, first partial, last partial
  float* sAl = smem + S.off_al;                         // ATT: [chunk][kMaxHeads] attention weights


  const int n_blocks = a.n_range / a.pieces_per_block;
  const int logical = xcd_remap(blockIdx.x, n_blocks * n_cgrp);
  const int slot = logical / n_cgrp, cgrp = logical - slot * n_cgrp;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int h = lane >> 5, l32 = lane & 31;
  const int C = a.C, nr = a.n_radial, R = a.R;
  const int c0 = (cgrp * waves + wave) * CT * kTile + l32;  // this lane's channel in tile 0
  // ATT: the head of this wave's channel tile
  const int my_head = ATT ? min((c0 - l32) / (C / a.n_heads), a.n_heads - 1) : 0;

  // Split mode: one thread per (packed K-block b, rank tile rt, lane) writes
  // the factor operand of that block: lane (h, r) slot j = 8b + i holds, for
  // the group j / PN and degree row h PN + j % PN, the fp16 hi part of
  // F 2^-e_F (groups 0 and 1, against x hi and x lo) or its lo part (group 2,
  // against x hi); zero past d, R and the three groups.
  auto stage_packed = [&](const float* __restrict__ F, float fsc, int t, u32x4* dst) {
    const int ln = t % kWave, brt = t / kWave;
    const int b = brt / RT, rt = brt - b * RT;
    const int r = rt * kTile + (ln & 31), hh = ln >> 5;
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t pr = 0;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int j = 8 * b + 2 * q + u, g = j / PN, row = hh * PN + j % PN;
        const float v = (g < 3 && row < d && r < R) ? F[row * R + r] * fsc : 0.f;
        const _Float16 hi = static_cast<_Float16>(v);
        const _Float16 val = g == 2 ? static_cast<_Float16>(v - float(hi)) : hi;
        pr |= uint32_t(__builtin_bit_cast(uint16_t, val)) << (16 * u);
      }
      w[q] = pr;
    }
    dst[brt * kWave + ln] = u32x4{w[0], w[1], w[2], w[3]};
  };

  // Split mode: the power of two 2^-e_K that puts the factor's largest |KF|
  // in [2^13, 2^14) for its fp16 parts (a block maximum through sG, which
  // the chunk loop overwrites only after its first barrier); the edges' g
  // carry 2^e_K back.
  float kf_sc = 1.f, kf_unsc = 1.f;
  if constexpr (!BF && NRA > 0) {
    // the blocks and their scale were written by the launch's block kernel
    kf_unsc = a.ef_scale[1];
  } else if constexpr (!BF) {
    float mx = 0.f;
    for (int i = tid; i < d * R; i += blockDim.x) mx = fmaxf(mx, fabsf(a.KF[i]));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if (lane == 0) sG[wave] = mx;
    __syncthreads();
    for (int w = 0; w < int(blockDim.x / kWave); ++w) mx = fmaxf(mx, sG[w]);
    const int e = f16_split_exponent(mx);
    kf_sc = ldexpf(1.f, -e);
    kf_unsc = ldexpf(1.f, e);
  }
  // T3: the same for the second node factor (its own slots of sG)
  float kf2_sc = 1.f, kf2_unsc = 1.f;
  if constexpr (T3) {
    float mx = 0.f;
    for (int i = tid; i < d * R; i += blockDim.x) mx = fmaxf(mx, fabsf(a.KF2[i]));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    if (lane == 0) sG[kMaxWavesPerBlock + wave] = mx;
    __syncthreads();
    for (int w = 0; w < int(blockDim.x / kWave); ++w) mx = fmaxf(mx, sG[kMaxWavesPerBlock + w]);
    const int e = f16_split_exponent(mx);
    kf2_sc = ldexpf(1.f, -e);
    kf2_unsc = ldexpf(1.f, e);
    for (int t = tid; t < PB * RT * kWave; t += blockDim.x) stage_packed(a.KF2, kf2_sc, t, sA2);
  }
  // Factor operands.  Split mode: the packed blocks above.  bf16 mode: lane
  // (l32, h) of K-block b, rank tile rt holds KF[16b + 8h + i][rt*32 + l32],
  // i = 0..7, zero past d and R, in fp32.  One thread per (b, rt, lane).
  if constexpr (BF) {
    for (int t = tid; t < KB * RT * kWave; t += blockDim.x) {
      const int ln = t % kWave, brt = t / kWave;
      const int b = brt / RT, rt = brt - b * RT;
      const int r = rt * kTile + (ln & 31), k0 = 16 * b + 8 * (ln >> 5);
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = k0 + i < d && r < R ? a.KF[(k0 + i) * R + r] : 0.f;
      sAf[2 * t] = make_float4(v[0], v[1], v[2], v[3]);
      sAf[2 * t + 1] = make_float4(v[4], v[5], v[6], v[7]);
    }
  } else if constexpr (!kRegA && NRA > 0) {
    // the LDS tiles' blocks from the launch's packed copy (its scale above)
    const u32x4* __restrict__ kg =
        reinterpret_cast<const u32x4*>(static_cast<const char*>(a.ef_ops) + edge_ef_blocks_bytes(d, R));
    for (int t = tid; t < PB * NL * kWave; t += blockDim.x) {
      const int ln = t % kWave, bl = t / kWave, b = bl / NL, rt = NRA + (bl - b * NL);
      sA[t] = kg[(b * RT + rt) * kWave + ln];
    }
  } else if constexpr (!kRegA) {
    for (int t = tid; t < PB * RT * kWave; t += blockDim.x) stage_packed(a.KF, kf_sc, t, sA);
  }
  // ABL 1: this workgroup's copy of the staged blocks in global memory
  u32x4* gA = ABL == 1 ? static_cast<u32x4*>(a.fa_global) + size_t(blockIdx.x) * PB * RT * kWave : nullptr;
  if constexpr (ABL == 1) {
    __syncthreads();
    for (int t = tid; t < PB * RT * kWave; t += blockDim.x) gA[t] = sA[t];
  }
  __syncthreads();
  // Split mode with kRegA: every packed factor block is loaded into
  // registers at the start of each run of edges of one segment within a chunk
  // (areg[b * NRA + rt], NRA = RT) from the copy the launch's block kernel
  // wrote in global memory (20 KB at R = 128, cache resident; no LDS for the
  // factor, which leaves room for 64-edge chunks at two workgroups per CU), so
  // the edge loop reads no factor while the geometry phase and the segment
  // epilogue do not hold them.  Otherwise the blocks of rank tiles below NRA
  // are loaded the same way, and only the other tiles' blocks are staged in
  // LDS (copied from the same global copy), read from there where they are
  // used.  Either way their index goes through an opaque copy (zero
  // added in inline asm) so that the compiler does not hoist the reads out of
  // the loops.
  u32x4 areg[NRA > 0 ? PB * NRA : 1];
  // the packed blocks written by the launch (k_ef_blocks), after EF's: the
  // register tiles' source
  const u32x4* __restrict__ kfg = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.ef_ops) +
                                                                edge_ef_blocks_bytes(d, R));
  auto a_op = [&](int base, int b, int rt) -> u32x4 {
    if constexpr (ABL == 1)
      return gA[base + (b * RT + rt) * kWave];
    else
      return sA[base + (b * NL + rt - NRA) * kWave];
  };
  float* sTr = smem + S.off_t + wave * kTrFloats;  // split mode: this wave's transpose area

  // Feature operands of one edge.  Split mode: the lane's PN packed words of
  // the gathered row (launch_feature_layout_packed), PQ 16-byte loads and a
  // PT-word tail, each load of the 64 lanes one contiguous run; the MFMA
  // operand of packed block b is words 4b .. 4b+3 taken modulo PN (slots
  // [2 PN, 3 PN) repeat the hi words, past 3 PN the factor is zero).  bf16
  // mode: channel tile t, K-block b is the lane's 16 bytes of the operand
  // block xs[row][tile][b].  The gathered row is wave-uniform (row base in
  // scalar registers, one 32-bit lane offset per tile).  Channel tiles past
  // the layout's last read that tile; their results are never stored.
  constexpr int XB = BF ? CT : XP;  // bf16 mode: operand rows per edge
  struct XOps {
    u32x4 v[BF ? XB * KB : (PQ > 0 ? PQ : 1)];
    uint32_t t[(!BF && PT > 0) ? PT : 1];
  };
  const char* __restrict__ xs = static_cast<const char*>(a.feat);
  const int n_ct = (C + kTile - 1) / kTile;  // channel tiles of the layout
  const size_t row_bytes = BF ? size_t(n_ct) * XP * KB * 1024 : size_t(n_ct) * 256 * PN;
  uint32_t lane_off[CT];
  uint32_t tail_off = 0;
#pragma unroll
  for (int t = 0; t < CT; ++t) {
    const int ct = min((cgrp * waves + wave) * CT + t, n_ct - 1);
    lane_off[t] = BF ? uint32_t(ct * XP * KB * 1024 + h * 512 + l32 * 16) : uint32_t(ct * 256 * PN + lane * 16);
    if (!BF && t == 0) tail_off = uint32_t(ct * 256 * PN + PQ * 1024 + lane * 4 * PT);
  }
  auto load_x = [&](int row, XOps& xb) {
    const char* p = xs + size_t(row) * row_bytes;
    if constexpr (BF) {
#pragma unroll
      for (int t = 0; t < XB; ++t)
#pragma unroll
        for (int b = 0; b < KB; ++b)
          xb.v[t * KB + b] = *reinterpret_cast<const u32x4*>(p + lane_off[t] + uint32_t(b * 1024));
    } else {
#pragma unroll
      for (int q = 0; q < PQ; ++q) xb.v[q] = *reinterpret_cast<const u32x4*>(p + lane_off[0] + uint32_t(q * 1024));
#pragma unroll
      for (int t = 0; t < PT; ++t) xb.t[t] = *reinterpret_cast<const uint32_t*>(p + tail_off + uint32_t(4 * t));
    }
  };
  auto xw = [&](const XOps& xb, int j) -> uint32_t { return j < 4 * PQ ? xb.v[j / 4][j % 4] : xb.t[j - 4 * PQ]; };
  auto xop = [&](const XOps& xb, int b) -> u32x4 {
    return u32x4{xw(xb, (4 * b) % PN), xw(xb, (4 * b + 1) % PN), xw(xb, (4 * b + 2) % PN),
                 xw(xb, (4 * b + 3) % PN)};
  };

  f32x16 acc[RT][CT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < CT; ++t) acc[rt][t] = f32x16{};

  // Segment epilogue: Z[m][c] = sum_r EF[m][r] H[r][c] on 32x32x16 MFMA.  The
  // accumulators are the K operand as they stand (K-step (rt, q) of lane half
  // h contracts the ranks rt*32 + acc_krow(q, h, i) that its registers
  // 8q .. 8q+7 hold), and EF comes in operand blocks with the same rank order
  // (k_ef_blocks, read from global memory, where they stay cached).  fp32
  // problems: the wave's H scaled by a power of two into [2^13, 2^14) and
  // split into two fp16 parts, three part products, the scales of H and EF
  // multiplied back into Z; bf16 problems: H and EF rounded to bf16, one
  // product.  part < 0 writes the segment's output row, part 0 or 1 the
  // range's partial slot; the accumulators restart from zero.
  const char* __restrict__ efb = static_cast<const char*>(a.ef_ops);
  const float ef_unscale = BF ? 1.f : *a.ef_scale;
  int range = 0;
  auto finish = [&](int seg, int part) {
    float* dst = (ATOM || part < 0) ? a.out + size_t(seg) * d * C : a.partial + (size_t(range) * 2 + part) * d * C;
    constexpr int P16 = BF ? 1 : 2;
    // EF's operand blocks of one rank tile (all mt, both K-steps q and
    // parts), double-buffered: tile 0's loads go out first, before the scale
    // reduction, and tile rt+1's while tile rt computes, so no step waits a
    // full memory latency for its operand
    // (32-bit byte offsets from an opaque lane term: as 64-bit addresses the
    // compiler kept all MT * RT * 2 * P16 of them live across the edge loop,
    // which at L = 4 spilled 18 registers per lane and slowed the edge pass by
    // 3-4 %)
    u32x4 ef[2][MT][2][P16];
    uint32_t ef_lane = uint32_t(lane) * P16 * 16;
    asm volatile("" : "+v"(ef_lane));
    auto load_ef = [&](int rt, int buf) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int p = 0; p < P16; ++p)
            ef[buf][mt][q][p] = *reinterpret_cast<const u32x4*>(
                efb + (ef_lane + uint32_t(((((mt * RT + rt) * 2 + q) * kWave) * P16 + p) * 16)));
    };
    load_ef(0, 0);
    if constexpr (T3) {
      // V^T = x[seg]^T KF2 in the accumulators' layout (channels x ranks),
      // one packed K-reduction per rank tile (the three part products), times
      // the two operands' scales; H *= V
      XOps xv;
      load_x(seg, xv);
      const float vsc = a.row_scale[seg] * kf2_unsc;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        f32x16 u = f32x16{};
#pragma unroll
        for (int b = 0; b < PB; ++b) u = mfma_f16(xop(xv, b), sA2[(b * RT + rt) * kWave + lane], u);
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[rt][0][v] *= u[v] * vsc;
      }
    }
    float hsc = 1.f, zsc = 1.f;
    if constexpr (!BF) {
      float mx = 0.f;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < CT; ++t)
#pragma unroll
          for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fabsf(acc[rt][t][v]));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const int e = f16_split_exponent(mx);
      hsc = ldexpf(1.f, -e);
      zsc = ldexpf(ef_unscale, e);
    }
    f32x16 z[CT][MT];
#pragma unroll
    for (int t = 0; t < CT; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) z[t][mt] = f32x16{};
    if constexpr (BF) {
      // bf16 mode: acc[rt][t] holds H (ranks x channels), so its registers
      // 8q .. 8q+7 are a K operand as they stand (ranks in acc_krow order)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if (rt + 1 < RT) load_ef(rt + 1, (rt + 1) & 1);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          u32x4 hp[CT];
#pragma unroll
          for (int t = 0; t < CT; ++t) {
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2_rne(acc[rt][t][8 * q + 2 * i], acc[rt][t][8 * q + 2 * i + 1]);
            hp[t] = u32x4{w[0], w[1], w[2], w[3]};
          }
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int t = 0; t < CT; ++t) z[t][mt] = mfma_bf16(ef[rt & 1][mt][q][0], hp[t], z[t][mt]);
        }
        __builtin_amdgcn_sched_barrier(0);  // one rank tile's operands live at a time
      }
    } else {
      // split mode: acc[rt][0] holds H^T (channels x ranks, lane column =
      // rank rt*32 + l32, rows = channels 8j + 4h + i); through the wave's
      // LDS area it becomes the K operand of ranks 16q + 8h + i for channel
      // l32, scaled by hsc and split into fp16 hi and lo (three products
      // against EF's parts, ranks in natural order)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if (rt + 1 < RT) load_ef(rt + 1, (rt + 1) & 1);
#pragma unroll
        for (int v = 0; v < 16; ++v)
          sTr[(8 * (v >> 2) + 4 * h + (v & 3)) * kTrStride + l32] = acc[rt][0][v] * hsc;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const float4 f0 = *reinterpret_cast<const float4*>(sTr + l32 * kTrStride + 16 * q + 8 * h);
          const float4 f1 = *reinterpret_cast<const float4*>(sTr + l32 * kTrStride + 16 * q + 8 * h + 4);
          uint32_t w[2][4];
          split_f16x2_pair(f0.x, f0.y, w[0][0], w[1][0]);
          split_f16x2_pair(f0.z, f0.w, w[0][1], w[1][1]);
          split_f16x2_pair(f1.x, f1.y, w[0][2], w[1][2]);
          split_f16x2_pair(f1.z, f1.w, w[0][3], w[1][3]);
          const u32x4 hp0 = u32x4{w[0][0], w[0][1], w[0][2], w[0][3]};
          const u32x4 hp1 = u32x4{w[1][0], w[1][1], w[1][2], w[1][3]};
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const u32x4 e0 = ef[rt & 1][mt][q][0], e1 = ef[rt & 1][mt][q][1];
            z[0][mt] = mfma_f16(e1, hp0, z[0][mt]);
            z[0][mt] = mfma_f16(e0, hp1, z[0][mt]);
            z[0][mt] = mfma_f16(e0, hp0, z[0][mt]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // the next tile's writes after this tile's reads
      }
    }
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = c0 + t * kTile;
      if (c < C) {
        // the lane's base (row 4h, channel c) and wave-uniform row offsets,
        // so no per-row address is kept live across the kernel
        float* dl = dst + (4 * h) * C + c;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int m = mt * kTile + acc_row(v, h);
            const int du = (mt * kTile + 8 * (v >> 2) + (v & 3)) * C;
            if (m < d) {
              if constexpr (ATOM)
                unsafeAtomicAdd(dl + du, z[t][mt][v] * zsc);  // hardware float add
              else
                dl[du] = z[t][mt][v] * zsc;
            }
          }
      }
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int t = 0; t < CT; ++t) acc[rt][t] = f32x16{};
  };

  // Split mode: U_e^T = x[row]^T KF for one rank tile (channels x ranks,
  // the MFMA's A operand the packed x words, its B operand the packed factor
  // blocks) as one packed K-reduction of PB steps holding the three part
  // products (hi hi, hi lo, lo hi), then acc += g_e[r] * U_e^T with this
  // lane's one rank r = rt*32 + l32 (g carries the operands' scales).  The
  // rank tiles are pipelined: step rt runs the MFMA chain of tile rt into one
  // of two U buffers (with the factor blocks of tile rt+1 read from LDS
  // meanwhile unless they are kept in registers) and the VALU multiply-adds
  // of tile rt-1 from the other, so that the MFMA drain does not stall the
  // chain.
  // bf16 mode: per (K-block, rank tile) the K operand bf16(g_e[r] KF[k][r])
  // for this lane's eight k, built once and fed to the CT channel tiles; the
  // K factor values come from registers when they fit, else from LDS.
  constexpr bool kRegKF = BF && edge_reg_kf(d, RT);
  float4 kf[kRegKF ? KB * RT * 2 : 1];
  if constexpr (kRegKF) {
#pragma unroll
    for (int i = 0; i < KB * RT; ++i) {
      kf[2 * i] = sAf[(i * kWave + lane) * 2];
      kf[2 * i + 1] = sAf[(i * kWave + lane) * 2 + 1];
    }
  }
  auto edge_compute_bf = [&](int e, const XOps& xb) {
    int ab = 2 * lane;
    asm volatile("" : "+v"(ab));
    float g[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) g[rt] = sG[e * Rp + rt * kTile + l32];
#pragma unroll
    for (int b = 0; b < KB; ++b)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int i = b * RT + rt;
        const float4 f0 = kRegKF ? kf[2 * i] : sAf[ab + i * 2 * kWave];
        const float4 f1 = kRegKF ? kf[2 * i + 1] : sAf[ab + i * 2 * kWave + 1];
        const u32x4 kop = {pack_bf16x2(g[rt] * f0.x, g[rt] * f0.y), pack_bf16x2(g[rt] * f0.z, g[rt] * f0.w),
                           pack_bf16x2(g[rt] * f1.x, g[rt] * f1.y), pack_bf16x2(g[rt] * f1.z, g[rt] * f1.w)};
#pragma unroll
        for (int t = 0; t < CT; ++t) acc[rt][t] = mfma_bf16(kop, xb.v[t * KB + b], acc[rt][t]);
      }
  };
  auto edge_compute = [&](int e, const XOps& xb) {
    if constexpr (BF) {
      edge_compute_bf(e, xb);
    } else {
      int ab = lane;
      asm volatile("" : "+v"(ab));
      u32x4 am[NRA == RT ? 1 : 2][NRA == RT ? 1 : PB];  // [buffer][packed K-block] of the LDS tiles
      float gl[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) gl[rt] = sG[e * Rp + rt * kTile + l32];
      if constexpr (ATT) {
        const float al = sAl[e * kMaxHeads + my_head];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) gl[rt] *= al;
      }
      f32x16 U[2];
      auto load_a = [&](int rt, int buf) {
        if constexpr (NRA < RT) {
#pragma unroll
          for (int b = 0; b < PB; ++b) am[buf][b] = a_op(ab, b, rt);
        }
      };
      auto chain = [&](int rt, int buf) {
        f32x16 u = f32x16{};
#pragma unroll
        for (int b = 0; b < PB; ++b) {
          if (rt < NRA)
            u = mfma_f16(xop(xb, b), areg[b * NRA + (rt < NRA ? rt : 0)], u);
          else
            u = mfma_f16(xop(xb, b), am[NRA == RT ? 0 : (rt - NRA) & 1][b], u);
        }
        U[buf] = u;
      };
      auto fma_rt = [&](int rt, int buf) {
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[rt][0][v] += gl[rt] * U[buf][v];
      };
      // positions p in the order edge_tile_at gives; an LDS tile's blocks are
      // read while the chains before it run (the first LDS tile's from the
      // edge's start, the next one's from the previous LDS tile's chain on)
      if (NRA < RT) load_a(NRA, 0);
#pragma unroll
      for (int p = 0; p < RT; ++p) {
        const int rt = edge_tile_at(p, RT, NRA);
        if (rt >= NRA && rt + 1 < RT) load_a(rt + 1, (rt + 1 - NRA) & 1);
        __builtin_amdgcn_sched_barrier(0);
        chain(rt, p & 1);
        if (p > 0) fma_rt(edge_tile_at(p - 1, RT, NRA), (p - 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
      }
      fma_rt(edge_tile_at(RT - 1, RT, NRA), (RT - 1) & 1);
    }
  };

  // The workgroup's ranges are slot, slot + n_blocks, ...: at any time the
  // workgroups of one XCD work on neighbouring edges.
  for (int sp = 0; sp < (kMaxRanges == 1 ? 1 : a.pieces_per_block); ++sp) {
    range = sp * n_blocks + slot;
    const int e_lo = int(int64_t(range) * a.E / a.n_range), e_hi = int(int64_t(range + 1) * a.E / a.n_range);
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
          const int row = a.gather[eid];
          sIdx[t] = row;
          if constexpr (!BF) sSc[t] = a.row_scale[row] * kf_unsc;
          key = a.key[eid];
          if constexpr (ATT)
            for (int hh = 0; hh < a.n_heads; ++hh) sAl[t * kMaxHeads + hh] = a.alpha[size_t(cb + t) * a.n_heads + hh];
          const float vx = a.edge_vec[3 * eid], vy = a.edge_vec[3 * eid + 1], vz = a.edge_vec[3 * eid + 2];
          const float len = sqrtf(vx * vx + vy * vy + vz * vz);
          const float inv = 1.f / len;
          sVec[t] = make_float4(vx * inv, vy * inv, vz * inv, len);
        }
        int prev = __shfl_up(key, 1);
        if (t == 0) prev = cb > 0 ? a.key[a.perm[cb - 1]] : -1;
        const int last_key = __shfl(key, n - 1);
        const bool start = t < n && (ATOM || key != prev || (cb == e_lo && t == 0));
        const unsigned long long m = __ballot(start);
        if (start) {
          const int pos = __popcll(m & ((1ull << t) - 1));
          sBnd[pos] = t;
          sBndKey[pos] = key;
        }
        if (t == 0) {
          sMeta[0] = __popcll(m);
          sMeta[1] = !ATOM && cb == e_lo && cb > 0 && key == prev;
          sMeta[2] = !ATOM && cb + n == e_hi && e_hi < a.E && a.key[a.perm[e_hi]] == last_key;
        }
      }
      __syncthreads();
      // harmonics: one thread per edge (all degrees, unrolled); radial basis: one
      // thread per (edge, function)
      if constexpr (ABL == 2) {
        for (int t = tid; t < n; t += blockDim.x) {
          const float* yr = a.y_table + size_t(a.perm[cb + t]) * d;
#pragma unroll
          for (int k = 0; k < d; ++k) sY[t * d + k] = yr[k];
        }
      } else {
        for (int t = tid; t < n; t += blockDim.x) {
          const float4 u = sVec[t];
          sh_unit_all<L>(u.x, u.y, u.z, sY + t * d);
        }
      }
      for (int t = tid; t < n * nr; t += blockDim.x) {
        const int e = t / nr, q = t - e * nr;
        sPhi[t] = radial_phi(sVec[e].w, q, a.sigma);
      }
      __syncthreads();
      // g = (Y B) * (Phi Wrad) for the chunk's edges (rows) and all ranks
      // (columns): two small fp32 MFMA GEMMs per 32x32 tile, one rank tile per
      // wave, with B and Wrad read from global memory (cached; n_radial <= 16,
      // so Wrad's operands are at most 8 steps).  Rows beyond n hold zeros
      // (their A operand is masked) and are never read.
      const int n_et = (n + kTile - 1) / kTile;
      for (int item = wave; item < n_et * RT; item += waves) {
        const int et = item / RT, rt = item - et * RT;
        const int er = et * kTile + l32;  // this lane's edge row
        const bool row_ok = er < n;
        const int r = rt * kTile + l32, rc = r < R ? r : R - 1;
        f32x16 Tr = f32x16{}, Ty = f32x16{};
        if constexpr (edge_waves_per_eu(L, RT, BF) == 1 || L >= 4) {
          // one wave per SIMD, or L >= 4: every B and Wrad operand of the two
          // chains loaded before the first product, one memory latency per
          // item instead of one per radial step (at L = 4 and two waves per
          // SIMD this holds since the epilogue's addresses stopped taking
          // registers: headline edge pass 0.409-0.411 -> 0.398-0.399 ms)
          constexpr int KY = (d + 1) / 2;
          float bq[8], by[KY];
#pragma unroll
          for (int s2 = 0; s2 < 8; ++s2) {
            const int q = 2 * s2 + h, qc = q < nr ? q : nr - 1;
            bq[s2] = 2 * s2 < nr ? a.radial_w[qc * R + rc] : 0.f;
          }
#pragma unroll
          for (int s2 = 0; s2 < KY; ++s2) {
            const int k = 2 * s2 + h, kc = k < d ? k : d - 1;
            by[s2] = a.Bf[kc * R + rc];
          }
#pragma unroll
          for (int s2 = 0; s2 < 8; ++s2) {
            if (2 * s2 >= nr) break;
            const int q = 2 * s2 + h;
            const float av = (row_ok && q < nr) ? sPhi[er * nr + q] : 0.f;
            Tr = mfma32(av, (q < nr && r < R) ? bq[s2] : 0.f, Tr);
          }
#pragma unroll
          for (int s2 = 0; s2 < KY; ++s2) {
            const int k = 2 * s2 + h;
            const float av = (row_ok && k < d) ? sY[er * d + k] : 0.f;
            Ty = mfma32(av, (k < d && r < R) ? by[s2] : 0.f, Ty);
          }
        } else {
          // L <= 3 at two or more waves per SIMD: the loads inside the chains
          // (hoisted, they would cost L = 3 its third wave per SIMD)
#pragma unroll 1
          for (int s2 = 0; s2 < (nr + 1) / 2; ++s2) {
            const int q = 2 * s2 + h, qc = q < nr ? q : nr - 1;
            const float av = (row_ok && q < nr) ? sPhi[er * nr + q] : 0.f;
            const float bw = a.radial_w[qc * R + rc];
            Tr = mfma32(av, (q < nr && r < R) ? bw : 0.f, Tr);
          }
#pragma unroll
          for (int s2 = 0; s2 < (d + 1) / 2; ++s2) {
            const int k = 2 * s2 + h, kc = k < d ? k : d - 1;
            const float av = (row_ok && k < d) ? sY[er * d + k] : 0.f;
            const float bw = a.Bf[kc * R + rc];
            Ty = mfma32(av, (k < d && r < R) ? bw : 0.f, Ty);
          }
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int e = et * kTile + acc_row(v, h);
          sG[e * Rp + rt * kTile + l32] = BF ? Tr[v] * Ty[v] : Tr[v] * Ty[v] * (e < n ? sSc[e] : 0.f);
        }
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
        // kRegA: the factor blocks for this piece (after any epilogue, so
        // they are not held across it or across the chunk's geometry phase)
        if constexpr (kRegA) {
          int ai = lane;
          asm volatile("" : "+v"(ai));
#pragma unroll
          for (int i = 0; i < PB * RT; ++i) areg[i] = kfg[ai + i * kWave];
        } else if constexpr (NRA > 0) {
          int ai = lane;
          asm volatile("" : "+v"(ai));
#pragma unroll
          for (int b = 0; b < PB; ++b)
#pragma unroll
            for (int rt = 0; rt < NRA; ++rt) areg[b * NRA + rt] = kfg[ai + (b * RT + rt) * kWave];
        }
        // Two operand buffers used alternately: the loads of edge f+1 are
        // issued before the MFMAs of edge f, and the scheduling barriers keep
        // the compiler from sinking them next to their use.
        XOps x0, x1;
        load_x(__builtin_amdgcn_readfirstlane(sIdx[e]), x0);
        int f = e;
        for (; f + 1 < pe; f += 2) {
          load_x(__builtin_amdgcn_readfirstlane(sIdx[f + 1]), x1);
          __builtin_amdgcn_sched_barrier(0);
          edge_compute(f, x0);
          __builtin_amdgcn_sched_barrier(0);
          load_x(__builtin_amdgcn_readfirstlane(sIdx[f + 2 < pe ? f + 2 : f + 1]), x0);  // past the end: unused
          __builtin_amdgcn_sched_barrier(0);
          edge_compute(f + 1, x1);
          __builtin_amdgcn_sched_barrier(0);
        }
        if (f < pe) edge_compute(f, x0);
        e = pe;
      }
    }
    if (cur >= 0) finish(cur, first_seg && first_partial ? 0 : (last_partial ? 1 : -1));
  }
}

// Edge chunk of a block: the largest power of two <= 64 (at least 8) whose
// LDS fits the block's share of the CU (160 KB over the blocks per CU).
inline int edge_chunk(int L, int RT, bool bf, int n_radial, bool t3 = false, bool att = false) {
  const int d = (L + 1) * (L + 1);
  const int budget = 160 * 1024 / edge_waves_per_eu(L, RT, bf);
  int chunk = 64;
  while (chunk > 8 && edge_smem(RT, bf, d, n_radial, chunk, t3, edge_lds_tiles(L, RT, bf), att).floats * 4 > budget)
    chunk >>= 1;
  return chunk;
}

// Waves per workgroup and channel groups: a wave takes CT channel tiles, a
// workgroup up to four waves.
struct EdgeGrid {
  int waves, n_cgrp;
};
inline EdgeGrid edge_grid(int C, int RT, bool bf) {
  const int ct = edge_ct(bf, RT);
  const int wave_tiles = (C + ct * kTile - 1) / (ct * kTile);
  const int waves = wave_tiles < kMaxWavesPerBlock ? wave_tiles : kMaxWavesPerBlock;
  return EdgeGrid{waves, (wave_tiles + waves - 1) / waves};
}

template <int L, int RT, bool BF, bool ATOM = false, bool T3 = false, int ABL = 0, bool ATT = false>
hipError_t launch_l_rt_m(const EdgeArgs& a, hipStream_t s) {
  constexpr int d = (L + 1) * (L + 1);
  const EdgeGrid gr = edge_grid(a.C, RT, BF);
  const int waves = gr.waves, n_cgrp = gr.n_cgrp;
  if (a.E > 0) {
    const int chunk = edge_chunk(L, RT, BF, a.n_radial, T3, ATT);
    const size_t lds =
        size_t(edge_smem(RT, BF, d, a.n_radial, chunk, T3, edge_lds_tiles(L, RT, BF, ABL == 1), ATT).floats) * 4;
    auto k = k_cp_edge<L, RT, BF, ATOM, T3, ABL, ATT>;
    hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    k<<<dim3(a.n_range / a.pieces_per_block * n_cgrp), dim3(waves * kWave), lds, s>>>(a, n_cgrp, waves, chunk);
  }
  return hipGetLastError();
}

template <int L, int RT>
hipError_t launch_l_rt(const EdgeArgs& a, hipStream_t s) {
  return a.parts == 1 ? launch_l_rt_m<L, RT, true>(a, s) : launch_l_rt_m<L, RT, false>(a, s);
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

// The ablation's dispatch on the rank tiles (fp32 features only).
template <int L>
hipError_t launch_cp_edge_atomic_l(const EdgeArgs& a, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt_m<L, 1, false, true>(a, s);
    case 2: return launch_l_rt_m<L, 2, false, true>(a, s);
    case 3: return launch_l_rt_m<L, 3, false, true>(a, s);
    case 4: return launch_l_rt_m<L, 4, false, true>(a, s);
    case 5: return launch_l_rt_m<L, 5, false, true>(a, s);
    case 6: return launch_l_rt_m<L, 6, false, true>(a, s);
    case 7: return launch_l_rt_m<L, 7, false, true>(a, s);
    case 8: return launch_l_rt_m<L, 8, false, true>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// The ablations' dispatch on the rank tiles (fp32 features only).
template <int L, int ABL>
hipError_t launch_cp_edge_abl_l(const EdgeArgs& a, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt_m<L, 1, false, false, false, ABL>(a, s);
    case 2: return launch_l_rt_m<L, 2, false, false, false, ABL>(a, s);
    case 3: return launch_l_rt_m<L, 3, false, false, false, ABL>(a, s);
    case 4: return launch_l_rt_m<L, 4, false, false, false, ABL>(a, s);
    case 5: return launch_l_rt_m<L, 5, false, false, false, ABL>(a, s);
    case 6: return launch_l_rt_m<L, 6, false, false, false, ABL>(a, s);
    case 7: return launch_l_rt_m<L, 7, false, false, false, ABL>(a, s);
    case 8: return launch_l_rt_m<L, 8, false, false, false, ABL>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// The attention block's dispatch on the rank tiles (fp32 features only).
template <int L>
hipError_t launch_cp_edge_att_l(const EdgeArgs& a, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt_m<L, 1, false, false, false, 0, true>(a, s);
    case 2: return launch_l_rt_m<L, 2, false, false, false, 0, true>(a, s);
    case 3: return launch_l_rt_m<L, 3, false, false, false, 0, true>(a, s);
    case 4: return launch_l_rt_m<L, 4, false, false, false, 0, true>(a, s);
    case 5: return launch_l_rt_m<L, 5, false, false, false, 0, true>(a, s);
    case 6: return launch_l_rt_m<L, 6, false, false, false, 0, true>(a, s);
    case 7: return launch_l_rt_m<L, 7, false, false, false, 0, true>(a, s);
    case 8: return launch_l_rt_m<L, 8, false, false, false, 0, true>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// The three-input product's dispatch on the rank tiles (fp32 features only).
template <int L>
hipError_t launch_cp_edge_t3_l(const EdgeArgs& a, hipStream_t s) {
  switch ((a.R + kTile - 1) / kTile) {
    case 1: return launch_l_rt_m<L, 1, false, false, true>(a, s);
    case 2: return launch_l_rt_m<L, 2, false, false, true>(a, s);
    case 3: return launch_l_rt_m<L, 3, false, false, true>(a, s);
    case 4: return launch_l_rt_m<L, 4, false, false, true>(a, s);
    case 5: return launch_l_rt_m<L, 5, false, false, true>(a, s);
    case 6: return launch_l_rt_m<L, 6, false, false, true>(a, s);
    case 7: return launch_l_rt_m<L, 7, false, false, true>(a, s);
    case 8: return launch_l_rt_m<L, 8, false, false, true>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace edge_detail

}  // namespace tdn
