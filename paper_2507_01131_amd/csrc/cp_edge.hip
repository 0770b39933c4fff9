// Dispatch of the edge pass on the maximum degree L; each L is instantiated
// in its own translation unit (cp_edge_l<L>.hip) to keep compile units small.
#include "kernels.h"

namespace tdn {
namespace edge_detail {
template <int L>
hipError_t launch_cp_edge_l(const EdgeArgs& a, bool bf16, hipStream_t s);
}

hipError_t launch_cp_edge(const EdgeArgs& a, bool feat_bf16, hipStream_t s) {
  using namespace edge_detail;
  switch (a.L) {
    case 0: return launch_cp_edge_l<0>(a, feat_bf16, s);
    case 1: return launch_cp_edge_l<1>(a, feat_bf16, s);
    case 2: return launch_cp_edge_l<2>(a, feat_bf16, s);
    case 3: return launch_cp_edge_l<3>(a, feat_bf16, s);
    case 4: return launch_cp_edge_l<4>(a, feat_bf16, s);
    case 5: return launch_cp_edge_l<5>(a, feat_bf16, s);
    case 6: return launch_cp_edge_l<6>(a, feat_bf16, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
