// Device-side helpers shared by the oriented 1D convolution kernels:
// element conversion (float32 / bfloat16 storage) and the per-tap filter
// offsets of Eq. (2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace o1d {

// ---------------------------------------------------------------- storage

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);

template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }

// float32 -> bfloat16, IEEE round to nearest, ties to even (gfx950 converts
// in hardware: v_cvt_pk_bf16_f32).  NaN stays a quiet NaN; overflow rounds
// to infinity.
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) {
  return __builtin_bit_cast(uint16_t, (__bf16)v);
}

// ---------------------------------------------------------------- offsets

// Products closer than this to an integer are taken to be that integer
// before the floor; exact-integer products (0, 30, 90 ... degrees) would
// otherwise round to the wrong side in double precision.
constexpr double kSnapEps = 1e-9;
constexpr double kDegToRad = 3.141592653589793238462643383279502884 / 180.0;

__device__ __forceinline__ int floor_snapped(double v) {
  const double r = rint(v);
  return (fabs(v - r) <= kSnapEps) ? (int)r : (int)floor(v);
}

// Filter offsets of tap k (Eq. 2 with pad = K/2):
//   dh = floor(-(k - pad) sin theta),  dw = floor((k - pad) cos theta).
// Returns false for a non-finite angle; the offsets are then 0.
// For finite angles |dh|, |dw| <= pad always holds (|j sin| <= |j| <= pad
// in double precision as well), which the staging tiles rely on.
__device__ __forceinline__ bool tap_offset(float theta_deg, int K, int k, int* dh, int* dw) {
  const int pad = K >> 1;
  if (!isfinite(theta_deg)) {
    *dh = 0;
    *dw = 0;
    return false;
  }
  double s, c;
  sincos((double)theta_deg * kDegToRad, &s, &c);
  const double j = (double)(k - pad);
  int h = floor_snapped(-j * s);
  int w = floor_snapped(j * c);
  *dh = h < -pad ? -pad : (h > pad ? pad : h);
  *dw = w < -pad ? -pad : (w > pad ? pad : w);
  return true;
}

// Unrounded offsets of tap k (the rotation of (0, k - pad) by theta, before
// the floor of Eq. 2): rh = -(k - pad) sin theta, rw = (k - pad) cos theta.
// Returns false for a non-finite angle (the offsets are then 0).
__device__ __forceinline__ bool tap_real(float theta_deg, int K, int k, double* rh, double* rw) {
  if (!isfinite(theta_deg)) {
    *rh = 0.0;
    *rw = 0.0;
    return false;
  }
  double s, c;
  sincos((double)theta_deg * kDegToRad, &s, &c);
  const double j = (double)(k - (K >> 1));
  *rh = -j * s;
  *rw = j * c;
  return true;
}

// Fraction of v above floor_snapped(v): zero for a snapped (near-integer) v.
__device__ __forceinline__ double frac_snapped(double v, int fl) {
  const double f = v - (double)fl;
  return fabs(f) <= kSnapEps ? 0.0 : f;
}

}  // namespace o1d
