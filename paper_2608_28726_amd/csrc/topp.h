// Launch interface of the top-p (nucleus) feature kernels (internal).
#pragma once

#include "row_features.h"

namespace pr {

size_t topp_workspace(pr_dtype dtype, int64_t n_rows, int32_t V);
hipError_t launch_topp(const RowArgs& a, pr_dtype dtype, void* workspace, hipStream_t stream);

}  // namespace pr
