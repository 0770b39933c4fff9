// Dispatch of the destination-side backward kernel: the factored form for
// d <= 32 (cp_bwd_sg_<dtype>.hip), the direct form on the k-tile count 2 for
// d <= 64 (cp_bwd_dst_m2_<dtype>.hip); each in its own translation unit.
#include "kernels.h"

namespace tdn {
namespace bwd_detail {
template <int MT, typename TX>
hipError_t launch_mt(const BwdDstArgs& a, hipStream_t s);
}
namespace bwd_sg_detail {
template <bool BF16>
hipError_t launch_sg_any(const BwdDstArgs& a, hipStream_t s);
}

hipError_t launch_bwd_dst(const BwdDstArgs& a, bool x_bf16, hipStream_t s) {
  if (a.n_seg == 0) return hipSuccess;
  if (a.d <= 32)
    return x_bf16 ? bwd_sg_detail::launch_sg_any<true>(a, s) : bwd_sg_detail::launch_sg_any<false>(a, s);
  return x_bf16 ? bwd_detail::launch_mt<2, uint16_t>(a, s) : bwd_detail::launch_mt<2, float>(a, s);
}

}  // namespace tdn
