// Forward / input-gradient strip kernels, bfloat16 storage (float32 arithmetic), walks of up to 32 cells.
#include "o1d_strip_kernels.h"

namespace o1d {

hipError_t launch_gather_strip_bf16_k32(const strip::Plan& pl, const void* in, const void* w, const float* theta,
                                     void* out, hipStream_t stream) {
  return strip::gather_t<uint16_t, 32>(pl, in, w, theta, out, stream);
}

}  // namespace o1d
