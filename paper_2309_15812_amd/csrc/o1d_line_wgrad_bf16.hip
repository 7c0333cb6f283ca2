// Weight-gradient line kernels, bfloat16 storage.
#include "o1d_line_kernels.h"

namespace o1d {

hipError_t launch_wgrad_line_bf16(const line::LinePlan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial, hipStream_t stream) {
  return line::wgrad_t<uint16_t>(pl, x, dy, theta, dw, partial, stream);
}

}  // namespace o1d
