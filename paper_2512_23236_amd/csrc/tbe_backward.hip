// Sparse-gradient backward (sort + segmented reduce).  Placeholder until the
// kernels land: reports that the operation is not available.
#include "tbe_internal.h"

namespace tbe {

size_t backward_workspace_bytes(const Plan &, int64_t) { return 0; }

hipError_t launch_backward(const Plan &, const float *, const int64_t *, const int64_t *, int64_t,
                           const float *, void *, size_t, float *, int64_t, int64_t *, int64_t *,
                           int64_t *, int64_t *, int32_t *, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace tbe
