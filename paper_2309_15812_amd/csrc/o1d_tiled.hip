// General tiled kernels for depthwise convolution with oriented 1D kernels.
//
// Each workgroup owns one BH x BW output tile of one (n, c) plane and stages
// the (BH + 2 pad) x (BW + 2 pad) input window it reads, zero-filled outside
// the plane, in LDS.  With the halo in LDS the tap loop needs no bounds
// checks, every global load is coalesced and every input pixel of the tile is
// read from HBM once (plus the halo shared with neighbouring tiles).  This is
// the data-reuse idea of the paper's "CUDA from scratch" kernel (appendix
// "Implementation Notes": stage the input in shared memory, cut large images
// into bands) in a form that works for any H, W and K up to O1D_MAX_K; the
// per-angle register-blocked kernels take over the shapes they cover.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_launch.h"

namespace o1d {
namespace {

// Builds the flat LDS offsets of the K taps for channel c into s_off and the
// weights into s_w.  A non-finite angle makes the channel's weights NaN, so
// its outputs are NaN rather than silently wrong.
template <typename T>
__device__ __forceinline__ void load_taps(const T* __restrict__ wgt, const float* __restrict__ theta, int c, int K,
                                          int sign, int S, int* s_off, float* s_w) {
  const int pad = K >> 1;
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    int dh, dw;
    const bool ok = tap_offset(theta[c], K, k, &dh, &dw);
    s_off[k] = (pad + sign * dh) * S + (pad + sign * dw);
    if (s_w) s_w[k] = ok ? to_f32(wgt[(size_t)c * K + k]) : __builtin_nanf("");
  }
}

// Stages rows [p0 - pad, p0 + BH + pad) x cols [q0 - pad, q0 + BW + pad) of
// one plane into tile (row stride S), zero outside the plane.
template <typename T>
__device__ __forceinline__ void stage_tile(const T* __restrict__ src, int H, int W, int p0, int q0, int pad, int TR,
                                           int S, float* tile) {
  const int total = TR * S;
  for (int i = threadIdx.x; i < total; i += blockDim.x) {
    const int r = i / S;
    const int s = i - r * S;
    const int h = p0 - pad + r;
    const int w = q0 - pad + s;
    float v = 0.f;
    if (h >= 0 && h < H && w >= 0 && w < W) v = to_f32(src[(size_t)h * W + w]);
    tile[i] = v;
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void gather_tiled(const T* __restrict__ in, const T* __restrict__ wgt,
                                                         const float* __restrict__ theta, T* __restrict__ out,
                                                         int C, int H, int W, int K, int sign, int BH, int BW,
                                                         int tiles_x) {
  extern __shared__ float smem[];
  const int c = blockIdx.y;
  const int n = blockIdx.z;
  const int ty = blockIdx.x / tiles_x;
  const int tx = blockIdx.x - ty * tiles_x;
  const int p0 = ty * BH, q0 = tx * BW;
  const int pad = K >> 1;
  const int S = BW + 2 * pad, TR = BH + 2 * pad;
  int* s_off = reinterpret_cast<int*>(smem);
  float* s_w = smem + K;
  float* tile = smem + 2 * K;

  load_taps(wgt, theta, c, K, sign, S, s_off, s_w);
  const size_t plane = ((size_t)n * C + c) * (size_t)H * (size_t)W;
  stage_tile(in + plane, H, W, p0, q0, pad, TR, S, tile);
  __syncthreads();

  T* dst = out + plane;
  for (int i = threadIdx.x; i < BH * BW; i += blockDim.x) {
    const int r = i / BW;
    const int s = i - r * BW;
    const int p = p0 + r, q = q0 + s;
    if (p < H && q < W) {
      const float* t = tile + r * S + s;
      float acc = 0.f;
      for (int k = 0; k < K; ++k) acc = fmaf(s_w[k], t[s_off[k]], acc);
      dst[(size_t)p * W + q] = from_f32<T>(acc);
    }
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Weight gradient, one (tile, channel, batch chunk) per workgroup:
//   partial[part][c][k] = sum over the chunk's images and the tile's outputs of
//                         dy[n,c,p,q] * x[n,c,p+dh_k,q+dw_k].
// KB taps are accumulated in registers per pass; K > KB takes several passes.
template <typename T, int KB>
__global__ __launch_bounds__(kThreads) void wgrad_tiled(const T* __restrict__ x, const T* __restrict__ dy,
                                                        const float* __restrict__ theta, float* __restrict__ partial,
                                                        int N, int C, int H, int W, int K, int BH, int BW,
                                                        int tiles_x, int npc) {
  extern __shared__ float smem[];
  const int c = blockIdx.y;
  const int chunk = blockIdx.z;
  const int tile_id = blockIdx.x;
  const int ty = tile_id / tiles_x;
  const int tx = tile_id - ty * tiles_x;
  const int p0 = ty * BH, q0 = tx * BW;
  const int pad = K >> 1;
  const int S = BW + 2 * pad, TR = BH + 2 * pad;
  int* s_off = reinterpret_cast<int*>(smem);
  float* s_red = smem + 2 * K;           // [waves][KB]
  float* tile = s_red + (kThreads / 64) * KB;
  const int n_begin = chunk * npc;
  const int n_end = min(N, n_begin + npc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool finite = isfinite(theta[c]);

  load_taps<T>(nullptr, theta, c, K, 1, S, s_off, nullptr);
  const size_t parts = (size_t)gridDim.z * (size_t)gridDim.x;
  const size_t part = (size_t)chunk * gridDim.x + tile_id;

  for (int kb = 0; kb < K; kb += KB) {
    float acc[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) acc[j] = 0.f;
    for (int n = n_begin; n < n_end; ++n) {
      const size_t plane = ((size_t)n * C + c) * (size_t)H * (size_t)W;
      __syncthreads();  // previous image's tile fully consumed
      stage_tile(x + plane, H, W, p0, q0, pad, TR, S, tile);
      __syncthreads();
      const T* g = dy + plane;
      for (int i = threadIdx.x; i < BH * BW; i += blockDim.x) {
        const int r = i / BW;
        const int s = i - r * BW;
        const int p = p0 + r, q = q0 + s;
        if (p < H && q < W) {
          const float gv = to_f32(g[(size_t)p * W + q]);
          const float* t = tile + r * S + s;
#pragma unroll
          for (int j = 0; j < KB; ++j)
            if (kb + j < K) acc[j] = fmaf(gv, t[s_off[kb + j]], acc[j]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const float v = wave_sum(acc[j]);
      if (lane == 0) s_red[wave * KB + j] = v;
    }
    __syncthreads();
    if (threadIdx.x < KB && kb + (int)threadIdx.x < K) {
      float v = 0.f;
      for (int wv = 0; wv < kThreads / 64; ++wv) v += s_red[wv * KB + threadIdx.x];
      partial[(part * C + c) * (size_t)K + kb + threadIdx.x] = finite ? v : __builtin_nanf("");
    }
    __syncthreads();
  }
  (void)parts;
}

// dw[c,k] = sum over parts of partial[part][c][k], in part order.
template <typename T>
__global__ __launch_bounds__(kThreads) void wgrad_finish(const float* __restrict__ partial, T* __restrict__ dw,
                                                         int CK, int parts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CK) return;
  float s = 0.f;
  for (int j = 0; j < parts; ++j) s += partial[(size_t)j * CK + i];
  dw[i] = from_f32<T>(s);
}

template <typename T>
__global__ __launch_bounds__(kThreads) void fill_zero(T* __restrict__ dst, size_t count) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) dst[i] = from_f32<T>(0.f);
}

template <typename K_>
hipError_t set_lds_limit(K_ kernel, size_t bytes) {
  if (bytes <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)kMaxLdsBytes);
}

template <typename T>
hipError_t gather_t(const void* in, const void* w, const float* theta, void* out, int N, int C, int H, int W, int K,
                    int sign, hipStream_t stream) {
  const TilePlan p = plan_tiles(H, W, K, 0);
  hipError_t e = set_lds_limit(gather_tiled<T>, p.lds_bytes);
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)p.tiles(), (unsigned)C, (unsigned)N);
  hipLaunchKernelGGL(gather_tiled<T>, grid, dim3(kThreads), p.lds_bytes, stream, static_cast<const T*>(in),
                     static_cast<const T*>(w), theta, static_cast<T*>(out), C, H, W, K, sign, p.BH, p.BW,
                     p.tiles_x);
  return hipGetLastError();
}

template <typename T, int KB>
hipError_t wgrad_kb(const void* x, const void* dy, const float* theta, void* dw, float* partial, int N, int C, int H,
                    int W, int K, hipStream_t stream) {
  const WgradPlan p = plan_wgrad(N, C, H, W, K);
  hipError_t e = set_lds_limit(wgrad_tiled<T, KB>, p.tile.lds_bytes);
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)p.tile.tiles(), (unsigned)C, (unsigned)p.nchunk);
  hipLaunchKernelGGL((wgrad_tiled<T, KB>), grid, dim3(kThreads), p.tile.lds_bytes, stream, static_cast<const T*>(x),
                     static_cast<const T*>(dy), theta, partial, N, C, H, W, K, p.tile.BH, p.tile.BW,
                     p.tile.tiles_x, p.npc);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int CK = C * K;
  hipLaunchKernelGGL(wgrad_finish<T>, dim3((unsigned)((CK + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     partial, static_cast<T*>(dw), CK, (int)p.parts());
  return hipGetLastError();
}

template <typename T>
hipError_t wgrad_t(const void* x, const void* dy, const float* theta, void* dw, float* partial, int N, int C, int H,
                   int W, int K, hipStream_t stream) {
  switch (wgrad_tap_block(K)) {
    case 16: return wgrad_kb<T, 16>(x, dy, theta, dw, partial, N, C, H, W, K, stream);
    case 32: return wgrad_kb<T, 32>(x, dy, theta, dw, partial, N, C, H, W, K, stream);
    default: return wgrad_kb<T, 64>(x, dy, theta, dw, partial, N, C, H, W, K, stream);
  }
}

}  // namespace

hipError_t launch_gather(Dtype dt, const void* in, const void* w, const float* theta, void* out, int N, int C, int H,
                         int W, int K, int sign, hipStream_t stream) {
  if (dt == Dtype::F32) return gather_t<float>(in, w, theta, out, N, C, H, W, K, sign, stream);
  return gather_t<uint16_t>(in, w, theta, out, N, C, H, W, K, sign, stream);
}

hipError_t launch_wgrad(Dtype dt, const void* x, const void* dy, const float* theta, void* dw, float* partial, int N,
                        int C, int H, int W, int K, hipStream_t stream) {
  if (dt == Dtype::F32) return wgrad_t<float>(x, dy, theta, dw, partial, N, C, H, W, K, stream);
  return wgrad_t<uint16_t>(x, dy, theta, dw, partial, N, C, H, W, K, stream);
}

hipError_t launch_zero(Dtype dt, void* dst, size_t count, hipStream_t stream) {
  const unsigned blocks = (unsigned)((count + kThreads - 1) / kThreads);
  if (dt == Dtype::F32)
    hipLaunchKernelGGL(fill_zero<float>, dim3(blocks), dim3(kThreads), 0, stream, static_cast<float*>(dst), count);
  else
    hipLaunchKernelGGL(fill_zero<uint16_t>, dim3(blocks), dim3(kThreads), 0, stream, static_cast<uint16_t*>(dst),
                       count);
  return hipGetLastError();
}

}  // namespace o1d
