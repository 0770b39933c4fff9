// The attention block's edge pass (messages weighted per head before the
// segment sum), instantiated for L = 1 .. 4 and fp32 features.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_att_l<1>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_att_l<2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_att_l<3>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_att_l<4>(const tdn::EdgeArgs&, hipStream_t);
