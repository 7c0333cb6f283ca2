// Small helper kernels of the library.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_launch.h"

namespace o1d {
namespace {

template <typename T>
__global__ __launch_bounds__(kThreads) void fill_zero(T* __restrict__ dst, size_t count) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) dst[i] = from_f32<T>(0.f);
}

}  // namespace

hipError_t launch_zero(Dtype dt, void* dst, size_t count, hipStream_t stream) {
  if (count == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((count + kThreads - 1) / kThreads);
  if (dt == Dtype::F32)
    hipLaunchKernelGGL(fill_zero<float>, dim3(blocks), dim3(kThreads), 0, stream, static_cast<float*>(dst), count);
  else
    hipLaunchKernelGGL(fill_zero<uint16_t>, dim3(blocks), dim3(kThreads), 0, stream, static_cast<uint16_t*>(dst),
                       count);
  return hipGetLastError();
}

}  // namespace o1d
