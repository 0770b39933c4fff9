// The edge pass's measurement ablations, instantiated for L = 2, 3, 4 and
// fp32 features: the atomic scatter-add (per-edge epilogue, float atomics
// into Z), the factor blocks read from global memory, and the harmonics read
// from a precomputed table.
#include "cp_edge_impl.hpp"

template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<3>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_atomic_l<4>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<2, 1>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<3, 1>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<4, 1>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<2, 2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<3, 2>(const tdn::EdgeArgs&, hipStream_t);
template hipError_t tdn::edge_detail::launch_cp_edge_abl_l<4, 2>(const tdn::EdgeArgs&, hipStream_t);
