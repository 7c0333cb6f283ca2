// Plane kernels (small planes, lanes over images), bfloat16 storage.
#include "o1d_plane_kernels.h"

namespace o1d {

hipError_t launch_plane_gather_bf16(const plane::Plan& pl, const void* in, const void* w, const float* theta, void* out,
                                 hipStream_t stream) {
  return plane::gather_t<uint16_t>(pl, in, w, theta, out, stream);
}

hipError_t launch_plane_wgrad_bf16(const plane::Plan& pl, const void* x, const void* dy, const float* theta, void* dw,
                                float* partial, hipStream_t stream) {
  return plane::wgrad_t<uint16_t>(pl, x, dy, theta, dw, partial, stream);
}

hipError_t launch_plane_bwd_bf16(const plane::Plan& pl, const void* x, const void* dy, const void* w, const float* theta,
                              void* dx, void* dw, float* partial, hipStream_t stream) {
  return plane::bwd_t<uint16_t>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace o1d
