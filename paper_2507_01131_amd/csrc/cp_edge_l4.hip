// Edge pass instantiated for maximum degree L = 4.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_l<4>(const tdn::EdgeArgs&, hipStream_t);
