// The forward pass for callers that cannot allocate device memory: the same
// launches as tdn_cp_tp_forward, with the workspace taken from a fixed
// scratch area that the library holds on every device it runs on.
//
// The area is a file-scope device array.  Its name in host code is not a
// device address, so on the first call on a device (with that device
// current) its address is looked up once with hipGetSymbolAddress and kept
// per device; only that address reaches kernels.  Each device holds its own
// copy until the process ends.  Nothing in the area has to start at zero:
// the forward writes every scratch region before reading it, as it does for
// a caller's uninitialised workspace.  Calls that overlap on one device
// share the area and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "api_internal.h"
#include "tdn.h"

namespace {

__device__ __align__(256) unsigned char scratch[TDN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// The current device's address of the scratch area (looked up on its first
// use on that device).
tdn_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return tdn::record_hip_error(e);
  if (dev < 0 || dev >= kMaxDevices) return TDN_ERR_UNSUPPORTED_DEVICE;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return tdn::record_hip_error(e);
    if (!p) return tdn::record_hip_error(hipErrorInvalidSymbol);
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return TDN_OK;
}

}  // namespace

extern "C" tdn_status tdn_cp_tp_forward_noalloc(const tdn_problem* p, const void* x, const float* edge_vec,
                                                const int32_t* edge_index, const float* A, const float* B,
                                                const float* D, const void* W, const float* radial_w, float* out,
                                                float* z_save, int32_t* perm, int32_t* offsets,
                                                hipStream_t stream) {
  size_t need = 0;
  tdn_status st = tdn_workspace_size(p, &need, nullptr);
  if (st != TDN_OK) return st;
  if (need > size_t(TDN_NOALLOC_SCRATCH_BYTES)) return TDN_ERR_SCRATCH_LIMIT;
  st = tdn::require_gfx950();
  if (st != TDN_OK) return st;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != TDN_OK) return st;
  return tdn::forward_untimed(p, x, edge_vec, edge_index, A, B, D, W, radial_w, out, z_save, perm, offsets, ws,
                              size_t(TDN_NOALLOC_SCRATCH_BYTES), stream);
}
