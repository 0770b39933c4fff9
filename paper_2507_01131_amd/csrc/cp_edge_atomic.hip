// The edge pass's atomic scatter-add ablation (per-edge epilogue, float
// atomics into Z), instantiated for L = 2, 3, 4 and fp32 features.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<3>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<4>(const tdn::EdgeArgs&, hipStream_t);
