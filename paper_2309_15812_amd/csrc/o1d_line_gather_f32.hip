// Forward / input-gradient line kernels, float32 storage.
#include "o1d_line_kernels.h"

namespace o1d {

hipError_t launch_gather_line_f32(const line::LinePlan& pl, const void* in, const void* w, const float* theta, void* out, hipStream_t stream) {
  return line::gather_t<float>(pl, in, w, theta, out, stream);
}

}  // namespace o1d
