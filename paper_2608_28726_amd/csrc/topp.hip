// Top-p (nucleus) features. Not built yet: reports "not supported".
#include "topp.h"

namespace pr {

size_t topp_workspace(pr_dtype, int64_t, int32_t) { return 0; }

hipError_t launch_topp(const RowArgs&, pr_dtype, void*, hipStream_t) { return hipErrorNotSupported; }

}  // namespace pr
