// bfloat16 edge pass instantiated for maximum degree L = 6.
#include "cp_edge_bf16_impl.hpp"

template hipError_t tdn::edge_bf16_detail::launch_bf16_l<6>(const tdn::EdgeArgs&, hipStream_t);
