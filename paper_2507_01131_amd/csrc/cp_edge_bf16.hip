// bfloat16 edge pass: the dispatch on L; each L is instantiated in its own
// translation unit (cp_edge_bf16_l<L>.hip).
#include "cp_edge_bf16_impl.hpp"

namespace tdn {
namespace edge_bf16_detail {
template <int L>
hipError_t launch_bf16_l(const EdgeArgs& a, hipStream_t s);
}

hipError_t launch_cp_edge_bf16(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_bf16_detail;
  switch (a.L) {
    case 0: return launch_bf16_l<0>(a, s);
    case 1: return launch_bf16_l<1>(a, s);
    case 2: return launch_bf16_l<2>(a, s);
    case 3: return launch_bf16_l<3>(a, s);
    case 4: return launch_bf16_l<4>(a, s);
    case 5: return launch_bf16_l<5>(a, s);
    case 6: return launch_bf16_l<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
