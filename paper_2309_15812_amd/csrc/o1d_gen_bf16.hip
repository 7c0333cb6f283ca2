// General kernels (any plane, alignment, stride, layout, discretisation),
// bfloat16 storage, float32 arithmetic.
#include "o1d_gen_kernels.h"

namespace o1d {

hipError_t launch_gen_gather_bf16(const gen::Plan& pl, int layout, const void* in, const void* w, const float* theta,
                                void* out, hipStream_t stream) {
  return gen::gather_t<uint16_t>(pl, layout, in, w, theta, out, stream);
}

hipError_t launch_gen_wgrad_bf16(const gen::Plan& pl, int layout, const void* x, const void* dy, const float* theta,
                               void* dw, float* partial, hipStream_t stream) {
  return gen::wgrad_t<uint16_t>(pl, layout, x, dy, theta, dw, partial, stream);
}

hipError_t launch_gen_bwd_bf16(const gen::Plan& pl, const void* x, const void* dy, const void* w, const float* theta,
                             void* dx, void* dw, float* partial, hipStream_t stream) {
  return gen::bwd_t<uint16_t>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace o1d
