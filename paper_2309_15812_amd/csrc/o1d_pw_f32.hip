// Pointwise convolution matrix products on the matrix cores, float32 storage.
#include "o1d_pw_kernels.h"

namespace o1d {

hipError_t launch_pw_gemm_f32(const pw::Params& p, const void* A, const void* B, void* out, hipStream_t stream) {
  return pw::gemm_t<float>(p, A, B, out, stream);
}

}  // namespace o1d
