// Destination-side backward kernel instantiated for MT = 2 k tiles, f32 features.
#include "cp_bwd_dst_impl.hpp"

template hipError_t tdn::bwd_detail::launch_mt<2, false>(const tdn::BwdDstArgs&, hipStream_t);
