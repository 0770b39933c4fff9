// Library-internal entry points shared between the C ABI's source files.
#pragma once

#include <hip/hip_runtime.h>

#include "tdn.h"

namespace tdn {

// Records a failed HIP call for tdn_last_hip_error and returns TDN_ERR_HIP.
tdn_status record_hip_error(hipError_t e);

// TDN_OK when the current device is gfx950.
tdn_status require_gfx950();

// tdn_cp_tp_forward on a given workspace, recording no timing events.
tdn_status forward_untimed(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                           const float* A, const float* B, const float* D, const void* W, const float* radial_w,
                           float* out, float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

}  // namespace tdn
