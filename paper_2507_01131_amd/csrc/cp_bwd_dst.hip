// Dispatch of the destination-side backward kernel on the k-tile count
// (d <= 32 or d <= 64) and the feature dtype; each combination is
// instantiated in its own translation unit (cp_bwd_dst_m<MT>_<dtype>.hip).
#include "kernels.h"

namespace tdn {
namespace bwd_detail {
template <int MT, typename TX>
hipError_t launch_mt(const BwdDstArgs& a, hipStream_t s);
}

hipError_t launch_bwd_dst(const BwdDstArgs& a, bool x_bf16, hipStream_t s) {
  using namespace bwd_detail;
  if (a.n_seg == 0) return hipSuccess;
  const bool two = a.d > 32;
  if (x_bf16) return two ? launch_mt<2, uint16_t>(a, s) : launch_mt<1, uint16_t>(a, s);
  return two ? launch_mt<2, float>(a, s) : launch_mt<1, float>(a, s);
}

}  // namespace tdn
