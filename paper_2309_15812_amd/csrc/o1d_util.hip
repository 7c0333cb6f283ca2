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

// dw[i] = sum over j < parts of partial[j CK + i], added in the order of j.
// The loads are issued sixteen at a time ahead of their additions, so that a
// thread waits for memory once per sixteen rows instead of once per row.
template <typename T>
__global__ __launch_bounds__(kThreads) void partial_sum(const float* __restrict__ partial, T* __restrict__ dw, int CK,
                                                        int parts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CK) return;
  constexpr int kBatch = 16;
  float s = 0.f;
  for (int j0 = 0; j0 < parts; j0 += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) v[u] = j0 + u < parts ? partial[(size_t)(j0 + u) * CK + i] : 0.f;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (j0 + u < parts) s += v[u];
  }
  dw[i] = from_f32<T>(s);
}

}  // namespace

hipError_t launch_partial_sum(Dtype dt, const float* partial, void* dw, int CK, int parts, hipStream_t stream) {
  if (CK <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((CK + kThreads - 1) / kThreads);
  if (dt == Dtype::F32)
    hipLaunchKernelGGL(partial_sum<float>, dim3(blocks), dim3(kThreads), 0, stream, partial, static_cast<float*>(dw),
                       CK, parts);
  else
    hipLaunchKernelGGL(partial_sum<uint16_t>, dim3(blocks), dim3(kThreads), 0, stream, partial,
                       static_cast<uint16_t*>(dw), CK, parts);
  return hipGetLastError();
}

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
