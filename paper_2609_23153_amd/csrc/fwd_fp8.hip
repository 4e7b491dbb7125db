// Fused block-sparse attention forward on fp8 (e4m3) operands for gfx950.
#include "common.h"
#include "launch.h"

namespace sa {

hipError_t launch_fwd_fp8(const Shape&, const FwdArgs&, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace sa
