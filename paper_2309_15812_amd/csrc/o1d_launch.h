// Internal launcher interface between the C ABI (argument checks, planning)
// and the kernel translation units.  Launchers enqueue on `stream` and
// return the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>

#include "o1d_plan.h"

namespace o1d {

enum class Dtype { F32 = 0, BF16 = 1 };

// Gather form of Eq. (1): out[n,c,p,q] = sum_k w[c,k] in[n,c, p + s dh_k, q + s dw_k],
// s = +1 for the forward pass and -1 for the input gradient.
hipError_t launch_gather(Dtype dt, const void* in, const void* w, const float* theta, void* out, int N, int C,
                         int H, int W, int K, int sign, hipStream_t stream);

// Weight gradient: per-(tile, batch chunk) partial sums into `partial`
// ([parts][C][K] float32), then a fixed-order reduction into dw.
hipError_t launch_wgrad(Dtype dt, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                        int N, int C, int H, int W, int K, hipStream_t stream);

// dw[c,k] = 0 (empty batch or plane).
hipError_t launch_zero(Dtype dt, void* dst, size_t count, hipStream_t stream);

}  // namespace o1d
