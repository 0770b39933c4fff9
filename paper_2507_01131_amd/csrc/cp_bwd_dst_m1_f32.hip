// Destination-side backward kernel instantiated for MT = 1 k tiles, f32 features.
#include "cp_bwd_dst_impl.hpp"

template hipError_t tdn::bwd_detail::launch_mt<1, float>(const tdn::BwdDstArgs&, hipStream_t);
