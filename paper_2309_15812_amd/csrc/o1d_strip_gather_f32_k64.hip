// Forward / input-gradient strip kernels, float32 storage, walks of up to 64 cells.
#include "o1d_strip_kernels.h"

namespace o1d {

hipError_t launch_gather_strip_f32_k64(const strip::Plan& pl, const void* in, const void* w, const float* theta,
                                     void* out, hipStream_t stream) {
  return strip::gather_t<float, 64>(pl, in, w, theta, out, stream);
}

}  // namespace o1d
