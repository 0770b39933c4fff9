// Factored destination-side backward (d <= 32) instantiated for f32 features.
#include "cp_bwd_sg_impl.hpp"

template hipError_t tdn::bwd_sg_detail::launch_sg_any<false>(const tdn::BwdDstArgs&, hipStream_t);
