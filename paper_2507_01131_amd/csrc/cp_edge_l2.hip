// Edge pass instantiated for maximum degree L = 2.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_l<2>(const tdn::EdgeArgs&, hipStream_t);
