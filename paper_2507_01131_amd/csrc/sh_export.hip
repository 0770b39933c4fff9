// Stand-alone evaluation of the edge harmonics (and their Jacobian), the same
// device routines the layer kernels use, exported for stage-by-stage checks.
#include "common.hpp"
#include "kernels.h"
#include "sh_device.hpp"

namespace tdn {

namespace {

__global__ void k_sh(int L, int E, const float* __restrict__ vec, float* __restrict__ Y, float* __restrict__ J) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int d = (L + 1) * (L + 1);
  const float vx = vec[3 * e], vy = vec[3 * e + 1], vz = vec[3 * e + 2];
  const float inv = 1.f / sqrtf(vx * vx + vy * vy + vz * vz);
  if (J)
    sh_unit_jacobian(L, vx * inv, vy * inv, vz * inv, inv, Y + size_t(e) * d, J + size_t(e) * d * 3);
  else
    sh_unit(L, vx * inv, vy * inv, vz * inv, Y + size_t(e) * d);
}

}  // namespace

hipError_t launch_sh(int L, int E, const float* edge_vec, float* Y, float* dY, hipStream_t s) {
  if (E == 0) return hipSuccess;
  k_sh<<<dim3((E + 127) / 128), dim3(128), 0, s>>>(L, E, edge_vec, Y, dY);
  return hipGetLastError();
}

}  // namespace tdn
