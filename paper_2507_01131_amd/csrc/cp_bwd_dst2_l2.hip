// Destination-side backward on bf16 MFMA (d <= 32) instantiated for L = 2.
#include "cp_bwd_dst2_impl.hpp"

template hipError_t tdn::bwd2_detail::launch_l<2, false>(const tdn::BwdDstArgs&, int, hipStream_t);
template hipError_t tdn::bwd2_detail::launch_l<2, true>(const tdn::BwdDstArgs&, int, hipStream_t);
