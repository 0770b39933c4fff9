// bfloat16 edge pass: the feature transpose and the dispatch on L; each L is
// instantiated in its own translation unit (cp_edge_bf16_l<L>.hip).
#include "cp_edge_bf16_impl.hpp"

namespace tdn {
namespace edge_bf16_detail {
template <int L>
hipError_t launch_bf16_l(const EdgeArgs& a, hipStream_t s);
}

int bf16_kpad(int d) { return d <= 32 ? 32 : 64; }

hipError_t launch_transpose_bf16(int N, int d, int C, const void* x, void* xT, hipStream_t s) {
  using namespace edge_bf16_detail;
  if (N == 0) return hipSuccess;
  const size_t lds = size_t(d) * C * 2;
  const uint16_t* xs = static_cast<const uint16_t*>(x);
  uint16_t* xd = static_cast<uint16_t*>(xT);
  if (bf16_kpad(d) == 32) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_transpose_bf16<32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    k_transpose_bf16<32><<<dim3(N), dim3(256), lds, s>>>(d, C, xs, xd);
  } else {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_transpose_bf16<64>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    k_transpose_bf16<64><<<dim3(N), dim3(256), lds, s>>>(d, C, xs, xd);
  }
  return hipGetLastError();
}

hipError_t launch_cp_edge_bf16(const EdgeArgs& a, hipStream_t s) {
  using namespace edge_bf16_detail;
  switch (a.L) {
    case 0: return launch_bf16_l<0>(a, s);
    case 1: return launch_bf16_l<1>(a, s);
    case 2: return launch_bf16_l<2>(a, s);
    case 3: return launch_bf16_l<3>(a, s);
    case 4: return launch_bf16_l<4>(a, s);
    case 5: return launch_bf16_l<5>(a, s);
    case 6: return launch_bf16_l<6>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tdn
