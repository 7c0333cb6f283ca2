// Forward / input-gradient strip kernels, float32 storage, walks of up to 32 cells.
#include "o1d_strip_kernels.h"

namespace o1d {

hipError_t launch_gather_strip_f32_k32(const strip::Plan& pl, const void* in, const void* w, const float* theta,
                                     void* out, hipStream_t stream) {
  return strip::gather_t<float, 32>(pl, in, w, theta, out, stream);
}

}  // namespace o1d
