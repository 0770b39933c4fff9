// Split-form destination-side backward (d <= 32: dg per edge, then geometry and gradients per edge), instantiated for L = 2; fp32 features run on fp16 MFMA with two-part splits, bf16 features on bf16 MFMA.
#include "cp_bwd_dst2_impl.hpp"

template hipError_t tdn::bwd2_detail::launch_l<2, false>(const tdn::BwdDstArgs&, int, hipStream_t);
template hipError_t tdn::bwd2_detail::launch_l<2, true>(const tdn::BwdDstArgs&, int, hipStream_t);
