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

}  // namespace o1d
