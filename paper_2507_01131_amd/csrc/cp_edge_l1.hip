// Edge pass instantiated for maximum degree L = 1.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_l<1>(const tdn::EdgeArgs&, hipStream_t);
