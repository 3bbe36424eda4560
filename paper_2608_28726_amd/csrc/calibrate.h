// Launch interface of the threshold calibration kernel (internal).
#pragma once

#include "device_util.h"

namespace pr {

// tau[0] = the k-th largest non-NaN score, k = max(1, ceil(q * n_valid));
// n_ship[0] (may be NULL) = #{scores >= tau}. q == 0 or no valid score:
// tau = +inf, n_ship = 0. One workgroup.
hipError_t launch_calibrate(const float* scores, int32_t n, double q, float* tau, int32_t* n_ship,
                            hipStream_t stream);

}  // namespace pr
