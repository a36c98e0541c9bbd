// Backward entry points; the bf16 backward kernels are not built in this revision,
// so the ABI reports COWA_ERR_UNSUPPORTED for cowa_bwd.
#include "internal.h"
namespace cowa {
bool bwd_bf16_supported(int, int, int) { return false; }
hipError_t launch_bwd_bf16(const cowa_params&, const SchedView&, const void*, const void*, const void*, const void*,
                           const float*, const void*, void*, void*, void*, float*, float*, hipStream_t) {
  return hipErrorNotSupported;
}
}
