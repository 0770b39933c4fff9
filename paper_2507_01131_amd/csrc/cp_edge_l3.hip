// Edge pass instantiated for maximum degree L = 3.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_l<3>(const tdn::EdgeArgs&, hipStream_t);
