// Dispatch of the edge pass on the maximum degree L (each L is instantiated
// in its own translation unit, cp_edge_l<L>.hip, to keep compile units
// small), the choice of edge ranges, the zero padding of the output factor,
// and the kernel that combines the partial slots of segments spanning
// ranges.
#include "cp_edge_impl.hpp"

#include <map>
#include <mutex>

namespace tdn {
namespace edge_detail {
template <int L>
hipError_t launch_cp_edge_l(const EdgeArgs& a, hipStream_t s);

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

// dst[k][r] = src[k][r] for r < R, 0 for R <= r < Rp
__global__ __launch_bounds__(256) void k_pad_rows(int rows, int R, int Rp, const float* __restrict__ src,
                                                  float* __restrict__ dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * Rp) return;
  const int k = i / Rp, r = i - k * Rp;
  dst[i] = r < R ? src[k * R + r] : 0.f;
}

constexpr int kMinRangeEdges = 48;

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

EdgePlan edge_plan(int L, int R, int C, int n_radial, bool bf16, int E) {
  using namespace edge_detail;
  if (E <= 0) return EdgePlan{0, 0};
  const int RT = (R + kTile - 1) / kTile, d = (L + 1) * (L + 1);
  const EdgeGrid gr = edge_grid(C, RT, bf16);
  // workgroups per CU: as many as the wave slots (four SIMDs) and LDS allow
  const int lds = edge_smem(RT, bf16, d, n_radial, edge_chunk(L, RT, bf16, n_radial)).floats * 4;
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
                  !a.ef_pad))
    return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  if (a.E > 0) {
    const int Rp = (a.R + kTile - 1) / kTile * kTile;
    k_pad_rows<<<dim3((a.d * Rp + 255) / 256), dim3(256), 0, s>>>(a.d, a.R, Rp, a.EF, a.ef_pad);
    e = hipGetLastError();
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

}  // namespace tdn
