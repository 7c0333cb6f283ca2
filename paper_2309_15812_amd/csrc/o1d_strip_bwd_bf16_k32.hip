// Fused backward strip kernels, bfloat16 storage (float32 arithmetic), walks of up to 32 cells.
#include "o1d_strip_kernels.h"

namespace o1d {

hipError_t launch_bwd_strip_bf16_k32(const strip::Plan& pl, const void* x, const void* dy, const void* w,
                                  const float* theta, void* dx, void* dw, float* partial, hipStream_t stream) {
  return strip::bwd_t<uint16_t, 32>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace o1d
