// Dispatch of the destination-side backward kernel: for d <= 32 the range
// kernel on bf16 MFMA (cp_bwd_dst2_l<L>.hip), else, or where its LDS layout
// does not fit, the per-segment kernels: the factored form for d <= 32
// (cp_bwd_sg_<dtype>.hip), the direct form on the k-tile count 2 for d <= 64
// (cp_bwd_dst_m2_<dtype>.hip); each in its own translation unit.
#include "cp_bwd_dst2_impl.hpp"

namespace tdn {
namespace bwd_detail {
template <int MT, bool BF>
hipError_t launch_mt(const BwdDstArgs& a, hipStream_t s);
}
namespace bwd_sg_detail {
template <bool BF16>
hipError_t launch_sg_any(const BwdDstArgs& a, hipStream_t s);
}

namespace bwd2_detail {
#define TDN_DST2_EXTERN(LV)                                                              \
  extern template hipError_t launch_l<LV, false>(const BwdDstArgs&, int, hipStream_t); \
  extern template hipError_t launch_l<LV, true>(const BwdDstArgs&, int, hipStream_t);
TDN_DST2_EXTERN(0)
TDN_DST2_EXTERN(1)
TDN_DST2_EXTERN(2)
TDN_DST2_EXTERN(3)
TDN_DST2_EXTERN(4)
#undef TDN_DST2_EXTERN
}  // namespace bwd2_detail

constexpr int kMinPieceEdges = 96, kMaxPieces = 2;

bool bwd_dst_split(int L, int C, bool bf16) {
  return (L + 1) * (L + 1) <= 32 && bwd2_detail::dst2_split(C, bf16);
}

EdgePlan bwd_dst_plan(int L, int R, int C, int n_radial, bool bf16, int E) {
  using namespace bwd2_detail;
  const int d = (L + 1) * (L + 1);
  const int RT = (R + kTile - 1) / kTile;
  if (E <= 0 || d > 32 || RT > 8) return EdgePlan{0, 0};
  const bool split = bwd_dst_split(L, C, bf16);
  const int chunk = dst2_chunk(RT, bf16, d, n_radial, C, split);
  const int lds = dst2_smem(RT, bf16 ? 1 : 2, d, n_radial, C, chunk, split).floats * 4;
  if (lds > 160 * 1024) return EdgePlan{0, 0};
  int per_cu = 160 * 1024 / lds;
  per_cu = per_cu > 2 ? 2 : per_cu;  // eight waves per workgroup, two (four in the split form) per SIMD
  int nb = device_cus() * per_cu;
  nb = nb < E ? nb : E;
  // several ranges per workgroup (there is no sum across ranges here) while
  // each keeps at least kMinPieceEdges edges
  int S = E / (nb * kMinPieceEdges);
  S = S < 1 ? 1 : (S > kMaxPieces ? kMaxPieces : S);
  return EdgePlan{nb * S, S};
}

int bwd_dst_cpad(int C, bool bf16) { return bwd2_detail::dst2_cpad(C, bf16 ? 1 : 2); }

hipError_t launch_bwd_dst(const BwdDstArgs& a, bool x_bf16, hipStream_t s) {
  if (a.n_seg == 0 || a.E == 0) return hipSuccess;
  if (a.n_range > 0) {
    if (a.d > 32 || a.n_range > a.E || !a.xc || !a.dst || (!x_bf16 && !a.x_scale)) return hipErrorInvalidValue;
    switch (a.L) {
#define TDN_DST2_CASE(LV)                                                  \
  case LV:                                                                 \
    return x_bf16 ? bwd2_detail::launch_l<LV, true>(a, a.n_range, s)      \
                  : bwd2_detail::launch_l<LV, false>(a, a.n_range, s);
      TDN_DST2_CASE(0)
      TDN_DST2_CASE(1)
      TDN_DST2_CASE(2)
      TDN_DST2_CASE(3)
      TDN_DST2_CASE(4)
#undef TDN_DST2_CASE
      default: return hipErrorInvalidValue;
    }
  }
  if (a.d <= 32)
    return x_bf16 ? bwd_sg_detail::launch_sg_any<true>(a, s) : bwd_sg_detail::launch_sg_any<false>(a, s);
  if (!a.xc || (!x_bf16 && !a.x_scale)) return hipErrorInvalidValue;
  return x_bf16 ? bwd_detail::launch_mt<2, true>(a, s) : bwd_detail::launch_mt<2, false>(a, s);
}

}  // namespace tdn
