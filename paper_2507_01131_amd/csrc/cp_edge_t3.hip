// The three-input product's edge pass (App. A, N = 3), instantiated for
// L = 2, 3, 4 and fp32 features.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_t3_l<2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_t3_l<3>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_t3_l<4>(const tdn::EdgeArgs&, hipStream_t);
