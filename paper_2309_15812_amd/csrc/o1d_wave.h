// Wave-level helpers shared by the general and plane kernels: compile-time
// unrolled loops (per-cell sums must stay in registers, so their index must
// be a constant) and the sum over a wave's 64 lanes of 32 values at once.
#pragma once

#include <hip/hip_runtime.h>

#include <utility>

namespace o1d {
namespace wave {

// Calls f(integral_constant<int, I>) for I = 0 .. N - 1, unrolled whatever
// the loop body's size.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Sum over the 64 lanes of each of the 32 values acc[O .. O + 31]: five
// halving exchanges leave lane L with the sum over its lane pair of value
// O + ((L >> 1) & 31); the last exchange adds the pair.  Returns the total of
// that value.  acc[O .. O + 31] is consumed.
template <int O, int KB>
__device__ __forceinline__ float sum32(float (&acc)[KB]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 32, half = 16; m >= 2; m >>= 1, half >>= 1) {
    // select with bit masks on the loaded values, so that no select of two
    // array addresses (a run-time index, which would put acc in scratch) appears
    const int up = (lane & m) ? -1 : 0;
#pragma unroll
    for (int i = 0; i < half; ++i) {
      const int lo = __float_as_int(acc[O + i]), hi = __float_as_int(acc[O + i + half]);
      const float give = __int_as_float((lo & up) | (hi & ~up));
      const float keep = __int_as_float((hi & up) | (lo & ~up));
      acc[O + i] = keep + __shfl_xor(give, m, 64);
    }
  }
  return acc[O] + __shfl_xor(acc[O], 1, 64);
}

// red[wave * KB + j] = sum over the wave's lanes of acc[j], j < KB (a
// multiple of 32).  acc is consumed.
template <int KB, int H = 0>
__device__ __forceinline__ void sums(float (&acc)[KB], float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const float s = sum32<32 * H>(acc);
  if ((lane & 1) == 0) red[w * KB + 32 * H + ((lane >> 1) & 31)] = s;
  if constexpr (32 * (H + 1) < KB) sums<KB, H + 1>(acc, red);
}

}  // namespace wave
}  // namespace o1d
