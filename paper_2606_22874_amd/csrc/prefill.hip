// Block-sparse causal prefill attention (placeholder until the MFMA tile
// kernel is in place): reports SPOT_ERR_UNSUPPORTED through a launch error.
#include "spot_internal.h"

namespace spot {

hipError_t launch_sparse_prefill(const void*, const void*, const void*, int, const int32_t*,
                                 const int32_t*, int, int, int, int, float, void*, float*,
                                 hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace spot
