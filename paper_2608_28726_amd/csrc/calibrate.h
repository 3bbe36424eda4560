// Launch interface of the threshold calibration kernel (internal).
#pragma once

#include "device_util.h"

namespace pr {

// Workspace bytes for a pool of n scores (0: none needed).
size_t calibrate_workspace_bytes(int32_t n);

// tau[0] = the k-th largest non-NaN score, k = max(1, ceil(q * n_valid));
// n_ship[0] (may be NULL) = #{scores >= tau}. q == 0 or no valid score:
// tau = +inf, n_ship = 0. workspace: calibrate_workspace_bytes(n) bytes.
hipError_t launch_calibrate(const float* scores, int32_t n, double q, float* tau, int32_t* n_ship, void* workspace,
                            hipStream_t stream);

}  // namespace pr
