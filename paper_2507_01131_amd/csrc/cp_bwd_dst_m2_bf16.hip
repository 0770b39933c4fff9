// Destination-side backward kernel instantiated for MT = 2 k tiles, bf16 features.
#include "cp_bwd_dst_impl.hpp"

template hipError_t tdn::bwd_detail::launch_mt<2, true>(const tdn::BwdDstArgs&, hipStream_t);
