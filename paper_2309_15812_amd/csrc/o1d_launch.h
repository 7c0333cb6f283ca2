// Internal launcher interface between the C ABI (argument checks, planning)
// and the kernel translation units.  Launchers enqueue on `stream` and
// return the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>

#include "o1d_plan.h"

namespace o1d {

enum class Dtype { F32 = 0, BF16 = 1 };

// dst[i] = 0 for i < count (the weight gradient of an empty batch or plane).
hipError_t launch_zero(Dtype dt, void* dst, size_t count, hipStream_t stream);

// dw[i] = sum over j < parts of partial[j CK + i] (float32 partial rows of the
// weight gradient), summed in a fixed order, stored in dw's type.
hipError_t launch_partial_sum(Dtype dt, const float* partial, void* dw, int CK, int parts, hipStream_t stream);

}  // namespace o1d
