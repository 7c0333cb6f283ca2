// Weight-gradient strip kernels, bfloat16 storage (float32 arithmetic), walks of up to 32 cells.
#include "o1d_strip_kernels.h"

namespace o1d {

hipError_t launch_wgrad_strip_bf16_k32(const strip::Plan& pl, const void* x, const void* dy, const float* theta,
                                    void* dw, float* partial, hipStream_t stream) {
  return strip::wgrad_t<uint16_t, 32>(pl, x, dy, theta, dw, partial, stream);
}

}  // namespace o1d
