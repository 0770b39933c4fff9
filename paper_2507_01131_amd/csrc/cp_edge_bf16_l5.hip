// bfloat16 edge pass instantiated for maximum degree L = 5.
#include "cp_edge_bf16_impl.hpp"

template hipError_t tdn::edge_bf16_detail::launch_bf16_l<5>(const tdn::EdgeArgs&, hipStream_t);
