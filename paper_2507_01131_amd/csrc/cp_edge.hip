// Dispatch of the edge pass on the maximum degree L (each L is instantiated
// in its own translation unit, cp_edge_l<L>.hip, to keep compile units
// small), the choice of edge ranges, the output factor's operand blocks for
// the segment epilogue, and the kernel that combines the partial slots of
// segments spanning ranges.
#include "cp_edge_impl.hpp"

#include <map>
#include <mutex>

namespace tdn {
namespace edge_detail {
// Instantiated in their own translation units (cp_edge_l<L>.hip,
// cp_edge_ablations.hip, cp_edge_t3.hip); declared here so that this file does
// not compile the kernels again.
extern template hipError_t launch_cp_edge_l<0>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<1>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<2>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<3>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<4>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<5>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_l<6>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_atomic_l<2>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_atomic_l<3>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_atomic_l<4>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_t3_l<2>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_t3_l<3>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_t3_l<4>(const EdgeArgs&, hipStream_t);
#define TDN_ABL_EXTERN(LV)                                                          \
  extern template hipError_t launch_cp_edge_abl_l<LV, 1>(const EdgeArgs&, hipStream_t); \
  extern template hipError_t launch_cp_edge_abl_l<LV, 2>(const EdgeArgs&, hipStream_t);
TDN_ABL_EXTERN(2)
TDN_ABL_EXTERN(3)
TDN_ABL_EXTERN(4)
#undef TDN_ABL_EXTERN
extern template hipError_t launch_cp_edge_att_l<1>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_att_l<2>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_att_l<3>(const EdgeArgs&, hipStream_t);
extern template hipError_t launch_cp_edge_att_l<4>(const EdgeArgs&, hipStream_t);

namespace {

// Adds the partial slots of segments that span ranges, in range order, and
// writes the zero rows of segments without edges.  One block per segment.
__global__ __launch_bounds__(256) void k_range_fixup(int E, int n_range, int dC, const int32_t* __restrict__ offsets,
                                                     const float* __restrict__ partial, float* __restrict__ out) {
  const int seg = blockIdx.x;
  const int a0 = offsets[seg], b0 = offsets[seg + 1];
  float* o = out + size_t(seg) * dC;
  if (a0 == b0) {
    for (int i = threadIdx.x; i < dC; i += blockDim.x) o[i] = 0.f;
    return;
  }
  // range holding sorted slot p: the largest r with floor(r E / n_range) <= p
  const int ra = int((int64_t(a0 + 1) * n_range - 1) / E), rb = int((int64_t(b0) * n_range - 1) / E);
  if (ra == rb) return;
  for (int i = threadIdx.x; i < dC; i += blockDim.x) {
    float s = partial[(size_t(ra) * 2 + 1) * dC + i];
    for (int r = ra + 1; r <= rb; ++r) s += partial[size_t(r) * 2 * dC + i];
    o[i] = s;
  }
}

// The output factor EF [d, R] in the operand blocks of the segment
// epilogue's 32x32x16 MFMA: block (mt, rt, q), lane l holds
// EF[mt*32 + l%32][rt*32 + k(q, l/32, i)], i = 0..7 (zero past d and R).
// P = 2 (fp32 features): ranks in natural order, k = 16q + 8h + i (the
// epilogue transposes its sums through LDS), fp16 hi and lo of EF 2^-e with
// 2^e (EF's largest |EF| to [2^13, 2^14)) to ef_scale; P = 1 (bf16): ranks
// in the order the accumulators hold them, k = acc_krow(q, h, i), bf16.
//
// P = 2 also writes the node factor KF in the edge loop's packed operand
// blocks (fp16 parts of KF 2^-e_K; kf_out [PB][RT][64 lanes], the edge
// kernel keeps them in registers) and 2^e_K into kf_scale.
//
// One thread per 16-byte output entry, KF's entries first; every workgroup
// takes the two largest magnitudes over the whole factors itself (a few KB
// from L2), so the workgroups need no exchange and agree exactly.
__device__ __forceinline__ float block_abs_max(const float* __restrict__ v, int n, float* red) {
  const int tid = threadIdx.x, nt = blockDim.x;
  // eight independent loads in flight per thread
  float m[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int i = tid;
  for (; i + 7 * nt < n; i += 8 * nt)
#pragma unroll
    for (int u = 0; u < 8; ++u) m[u] = fmaxf(m[u], fabsf(v[i + u * nt]));
  for (; i < n; i += nt) m[0] = fmaxf(m[0], fabsf(v[i]));
  float mx = fmaxf(fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3])), fmaxf(fmaxf(m[4], m[5]), fmaxf(m[6], m[7])));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__host__ __device__ inline int ef_kf_entries(int d, int RT, bool kf) { return kf ? pk_blocks(d) * RT * kWave : 0; }

template <int P>
__global__ __launch_bounds__(256) void k_ef_blocks(int d, int R, int RT, int MT, const float* __restrict__ EF,
                                                   u32x4* __restrict__ out, float* __restrict__ ef_scale,
                                                   const float* __restrict__ KF, u32x4* __restrict__ kf_out,
                                                   float* __restrict__ kf_scale) {
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int t = blockIdx.x * blockDim.x + tid;
  const int n_kf = ef_kf_entries(d, RT, P == 2 && KF != nullptr);
  const int n_ef = MT * RT * 2 * kWave;
  if constexpr (P == 2) {
    if (KF) {
      const float mx = block_abs_max(KF, d * R, red + 4);
      const int e = f16_split_exponent(mx);
      const float ksc = ldexpf(1.f, -e);
      if (t == 0) *kf_scale = ldexpf(1.f, e);
      const int PN = pk_rows(d);
      if (t < n_kf) {
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
            const float v = (g < 3 && row < d && r < R) ? KF[row * R + r] * ksc : 0.f;
            const _Float16 hi = static_cast<_Float16>(v);
            const _Float16 val = g == 2 ? static_cast<_Float16>(v - float(hi)) : hi;
            pr |= uint32_t(__builtin_bit_cast(uint16_t, val)) << (16 * u);
          }
          w[q] = pr;
        }
        kf_out[brt * kWave + ln] = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
  }
  float sc = 1.f;
  if constexpr (P == 2) {
    const float mx = block_abs_max(EF, d * R, red);
    const int e = f16_split_exponent(mx);
    sc = ldexpf(1.f, -e);
    if (t == 0) *ef_scale = ldexpf(1.f, e);
  }
  const int te = t - n_kf;
  if (te >= 0 && te < n_ef) {
    const int ln = te % kWave, blk = te / kWave;
    const int q = blk % 2, rt = (blk / 2) % RT, mt = blk / (2 * RT);
    const int m = mt * kTile + (ln & 31), hh = ln >> 5;
    uint32_t w[P][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r0 = rt * kTile + (P == 2 ? 16 * q + 8 * hh + 2 * i : acc_krow(q, hh, 2 * i));
      const int r1 = rt * kTile + (P == 2 ? 16 * q + 8 * hh + 2 * i + 1 : acc_krow(q, hh, 2 * i + 1));
      const float v0 = (m < d && r0 < R) ? EF[m * R + r0] : 0.f;
      const float v1 = (m < d && r1 < R) ? EF[m * R + r1] : 0.f;
      if constexpr (P == 2)
        split_f16x2_pair(v0 * sc, v1 * sc, w[0][i], w[1][i]);
      else
        w[0][i] = pack_bf16x2_rne(v0, v1);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) out[te * P + p] = u32x4{w[p][0], w[p][1], w[p][2], w[p][3]};
  }
}

// the launch of k_ef_blocks: one 256-thread workgroup per 256 output entries
template <int P>
hipError_t launch_ef_blocks(int d, int R, const float* EF, u32x4* out, float* ef_scale, const float* KF,
                            u32x4* kf_out, float* kf_scale, hipStream_t s) {
  const int RT = (R + kTile - 1) / kTile, MT = (d + kTile - 1) / kTile;
  const int n = ef_kf_entries(d, RT, P == 2 && KF != nullptr) + MT * RT * 2 * kWave;
  k_ef_blocks<P><<<dim3((n + 255) / 256), dim3(256), 0, s>>>(d, R, RT, MT, EF, out, ef_scale, KF, kf_out, kf_scale);
  return hipGetLastError();
}

constexpr int kMinRangeEdges = 48;

// the node factor's packed blocks and scale inside ef_ops (after EF's blocks)
u32x4* kf_blocks(const EdgeArgs& a) {
  return reinterpret_cast<u32x4*>(static_cast<char*>(a.ef_ops) + edge_ef_blocks_bytes(a.d, a.R));
}
float* kf_scale(const EdgeArgs& a) { return a.ef_scale + 1; }

}  // namespace
}  // namespace edge_detail

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  static std::mutex mu;
  static std::map<int, int> cus;
  std::lock_guard<std::mutex> lk(mu);
  auto it = cus.find(dev);
  if (it == cus.end()) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    it = cus.emplace(dev, n).first;
  }
  return it->second;
}

size_t edge_ef_bytes(int d, int R) {
  const size_t kf = size_t(pk_blocks(d)) * ((R + kTile - 1) / kTile) * kWave * 16;
  return edge_ef_blocks_bytes(d, R) + kf + 256;
}

EdgePlan edge_plan(int L, int R, int C, int n_radial, bool bf16, int E, bool t3) {
  using namespace edge_detail;
  if (E <= 0) return EdgePlan{0, 0};
  const int RT = (R + kTile - 1) / kTile, d = (L + 1) * (L + 1);
  const EdgeGrid gr = edge_grid(C, RT, bf16);
  // workgroups per CU: as many as the wave slots (four SIMDs) and LDS allow
  const int lds =
      edge_smem(RT, bf16, d, n_radial, edge_chunk(L, RT, bf16, n_radial, t3), t3, edge_lds_tiles(L, RT, bf16)).floats * 4;
  int per_cu = 160 * 1024 / lds;
  const int by_waves = 4 * edge_waves_per_eu(L, RT, bf16) / gr.waves;
  if (per_cu > by_waves) per_cu = by_waves;
  int nb = device_cus() * (per_cu < 1 ? 1 : per_cu) / gr.n_cgrp;
  nb = nb < 1 ? 1 : (nb > E ? E : nb);
  // ranges per workgroup: up to edge_max_ranges while each range keeps at
  // least kMinRangeEdges edges
  const int smax = edge_max_ranges(L, RT, bf16);
  int S = E / (nb * kMinRangeEdges);
  S = S < 1 ? 1 : (S > smax ? smax : S);
  return EdgePlan{nb * S, S};
}

hipError_t launch_cp_edge(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_detail;
  if (a.parts != 1 && a.parts != 2) return hipErrorInvalidValue;
  if (a.parts == 2 && a.E > 0 && !a.row_scale) return hipErrorInvalidValue;
  if (a.E > 0 && (a.n_range < 1 || a.n_range > a.E || a.pieces_per_block < 1 || a.n_range % a.pieces_per_block ||
                  !a.ef_ops || !a.ef_scale))
    return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  if (a.E > 0) {
    u32x4* blocks = static_cast<u32x4*>(a.ef_ops);
    if (a.parts == 2)
      e = launch_ef_blocks<2>(a.d, a.R, a.EF, blocks, a.ef_scale, a.KF, kf_blocks(a), kf_scale(a), s);
    else
      e = launch_ef_blocks<1>(a.d, a.R, a.EF, blocks, a.ef_scale, nullptr, nullptr, nullptr, s);
    if (e != hipSuccess) return e;
  }
  switch (a.L) {
    case 0: e = launch_cp_edge_l<0>(a, s); break;
    case 1: e = launch_cp_edge_l<1>(a, s); break;
    case 2: e = launch_cp_edge_l<2>(a, s); break;
    case 3: e = launch_cp_edge_l<3>(a, s); break;
    case 4: e = launch_cp_edge_l<4>(a, s); break;
    case 5: e = launch_cp_edge_l<5>(a, s); break;
    case 6: e = launch_cp_edge_l<6>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  if (a.n_seg > 0)
    k_range_fixup<<<dim3(a.n_seg), dim3(256), 0, s>>>(a.E, a.n_range, a.d * a.C, a.offsets, a.partial, a.out);
  return hipGetLastError();
}

hipError_t launch_cp_edge_atomic(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_detail;
  if (a.parts != 2 || a.L < 2 || a.L > 4) return hipErrorInvalidValue;
  if (a.E > 0 && (a.n_range < 1 || a.n_range > a.E || a.pieces_per_block < 1 || a.n_range % a.pieces_per_block ||
                  !a.ef_ops || !a.ef_scale || !a.row_scale))
    return hipErrorInvalidValue;
  hipError_t e = launch_zero(a.out, size_t(a.n_seg) * a.d * a.C * 4, s);
  if (e != hipSuccess || a.E == 0) return e;
  e = launch_ef_blocks<2>(a.d, a.R, a.EF, static_cast<u32x4*>(a.ef_ops), a.ef_scale, a.KF, kf_blocks(a),
                          kf_scale(a), s);
  if (e != hipSuccess) return e;
  switch (a.L) {
    case 2: return launch_cp_edge_atomic_l<2>(a, s);
    case 3: return launch_cp_edge_atomic_l<3>(a, s);
    default: return launch_cp_edge_atomic_l<4>(a, s);
  }
}

}  // namespace tdn

namespace tdn {

hipError_t launch_cp_edge_t3(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_detail;
  if (a.parts != 2 || a.L < 2 || a.L > 4 || !a.KF2) return hipErrorInvalidValue;
  if (a.E > 0 && (a.n_range < 1 || a.n_range > a.E || a.pieces_per_block < 1 || a.n_range % a.pieces_per_block ||
                  !a.ef_ops || !a.ef_scale || !a.row_scale))
    return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  if (a.E > 0) {
    e = launch_ef_blocks<2>(a.d, a.R, a.EF, static_cast<u32x4*>(a.ef_ops), a.ef_scale, a.KF, kf_blocks(a),
                            kf_scale(a), s);
    if (e != hipSuccess) return e;
  }
  switch (a.L) {
    case 2: e = launch_cp_edge_t3_l<2>(a, s); break;
    case 3: e = launch_cp_edge_t3_l<3>(a, s); break;
    default: e = launch_cp_edge_t3_l<4>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if (a.n_seg > 0)
    k_range_fixup<<<dim3(a.n_seg), dim3(256), 0, s>>>(a.E, a.n_range, a.d * a.C, a.offsets, a.partial, a.out);
  return hipGetLastError();
}

size_t edge_abl_fa_bytes(int L, int R, int C, int n_range, int pieces_per_block) {
  using namespace edge_detail;
  const int d = (L + 1) * (L + 1), RT = (R + kTile - 1) / kTile;
  if (pieces_per_block < 1) return 0;
  const size_t blocks = size_t(n_range / pieces_per_block) * edge_grid(C, RT, false).n_cgrp;
  return blocks * pk_blocks(d) * RT * kWave * 16;
}

hipError_t launch_cp_edge_ablation(const EdgeArgs& a, int variant, const float* x_f32, hipStream_t s) {
  using namespace edge_detail;
  if (a.L < 2 || a.L > 4) return hipErrorInvalidValue;
  if (variant == kAblValu) return launch_cp_edge_valu(a, x_f32, s);
  if (variant != kAblFactorsGlobal && variant != kAblYTable) return hipErrorInvalidValue;
  if (a.parts != 2) return hipErrorInvalidValue;
  if ((variant == kAblFactorsGlobal && !a.fa_global) || (variant == kAblYTable && a.E > 0 && !a.y_table))
    return hipErrorInvalidValue;
  if (a.E > 0 && (a.n_range < 1 || a.n_range > a.E || a.pieces_per_block < 1 || a.n_range % a.pieces_per_block ||
                  !a.ef_ops || !a.ef_scale || !a.row_scale))
    return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  if (a.E > 0) {
    e = launch_ef_blocks<2>(a.d, a.R, a.EF, static_cast<u32x4*>(a.ef_ops), a.ef_scale, a.KF, kf_blocks(a),
                            kf_scale(a), s);
    if (e != hipSuccess) return e;
  }
  const bool fg = variant == kAblFactorsGlobal;
  switch (a.L) {
    case 2: e = fg ? launch_cp_edge_abl_l<2, 1>(a, s) : launch_cp_edge_abl_l<2, 2>(a, s); break;
    case 3: e = fg ? launch_cp_edge_abl_l<3, 1>(a, s) : launch_cp_edge_abl_l<3, 2>(a, s); break;
    default: e = fg ? launch_cp_edge_abl_l<4, 1>(a, s) : launch_cp_edge_abl_l<4, 2>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if (a.n_seg > 0)
    k_range_fixup<<<dim3(a.n_seg), dim3(256), 0, s>>>(a.E, a.n_range, a.d * a.C, a.offsets, a.partial, a.out);
  return hipGetLastError();
}

hipError_t launch_cp_edge_att(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_detail;
  if (a.parts != 2 || a.L < 1 || a.L > 4 || a.n_heads < 1 || a.n_heads > kMaxHeads ||
      a.C % (kTile * a.n_heads) != 0)
    return hipErrorInvalidValue;
  if (a.E > 0 && (a.n_range < 1 || a.n_range > a.E || a.pieces_per_block < 1 || a.n_range % a.pieces_per_block ||
                  !a.ef_ops || !a.ef_scale || !a.row_scale || !a.alpha))
    return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  if (a.E > 0) {
    e = launch_ef_blocks<2>(a.d, a.R, a.EF, static_cast<u32x4*>(a.ef_ops), a.ef_scale, a.KF, kf_blocks(a),
                            kf_scale(a), s);
    if (e != hipSuccess) return e;
  }
  switch (a.L) {
    case 1: e = launch_cp_edge_att_l<1>(a, s); break;
    case 2: e = launch_cp_edge_att_l<2>(a, s); break;
    case 3: e = launch_cp_edge_att_l<3>(a, s); break;
    default: e = launch_cp_edge_att_l<4>(a, s); break;
  }
  if (e != hipSuccess) return e;
  if (a.n_seg > 0)
    k_range_fixup<<<dim3(a.n_seg), dim3(256), 0, s>>>(a.E, a.n_range, a.d * a.C, a.offsets, a.partial, a.out);
  return hipGetLastError();
}

}  // namespace tdn
