// bfloat16 edge pass: the feature transpose and the dispatch on L; each L is
// instantiated in its own translation unit (cp_edge_bf16_l<L>.hip).
#include "cp_edge_bf16_impl.hpp"

namespace tdn {
namespace edge_bf16_detail {
template <int L>
hipError_t launch_bf16_l(const EdgeArgs& a, hipStream_t s);
}

int bf16_kpad(int d) { return d <= 32 ? 32 : 64; }

template <int DP, typename TI>
hipError_t transpose_dp(int N, int d, int C, const TI* x, uint16_t* xT, hipStream_t s) {
  using namespace edge_bf16_detail;
  const size_t lds = size_t(d) * C * 2;
  auto k = k_transpose_bf16<DP, TI>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(lds));
  if (e != hipSuccess) return e;
  k<<<dim3(N), dim3(256), lds, s>>>(d, C, x, xT);
  return hipGetLastError();
}

hipError_t launch_transpose_bf16(int N, int d, int C, const void* x, bool x_is_f32, void* xT, hipStream_t s) {
  if (N == 0) return hipSuccess;
  uint16_t* xd = static_cast<uint16_t*>(xT);
  const bool k32 = bf16_kpad(d) == 32;
  if (x_is_f32) {
    const float* xs = static_cast<const float*>(x);
    return k32 ? transpose_dp<32>(N, d, C, xs, xd, s) : transpose_dp<64>(N, d, C, xs, xd, s);
  }
  const uint16_t* xs = static_cast<const uint16_t*>(x);
  return k32 ? transpose_dp<32>(N, d, C, xs, xd, s) : transpose_dp<64>(N, d, C, xs, xd, s);
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
