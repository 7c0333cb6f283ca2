// Device code of the pointwise convolution's matrix products (included by
// o1d_pw_f32.hip and o1d_pw_bf16.hip); the host plan is in o1d_pw.h.
//
// A workgroup computes a 128 x 128 tile of C_b with four waves (2 x 2, each
// a 64 x 64 block of four 32 x 32 matrix-core tiles).  Per step of 32 along
// k the A and B tiles are staged in LDS with k contiguous (As[m][k],
// Bs[n][k]); the next step's global loads are in flight while the matrix
// cores work on the current one.  float32 storage multiplies on
// v_mfma_f32_32x32x2_f32 (float32 products), bfloat16 storage on
// v_mfma_f32_32x32x16_bf16; both accumulate in float32.
//
// Operand layout of a 32 x 32 tile (lane l of the wave): A row l % 32 and B
// column l % 32, the k values split between the two half-waves (l / 32);
// accumulator element e of lane l is row 8 (e / 4) + 4 (l / 32) + e % 4,
// column l % 32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_pw.h"

namespace o1d {
namespace pw {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Per storage type: elements per vector access (16 bytes) and the LDS row
// pitch (k contiguous): an odd number of words for float32, so that 32 lanes
// reading one k of 32 rows hit 32 banks; 80-byte rows for bfloat16, so that
// every lane's 8 consecutive k are one aligned 16-byte read.
template <typename T>
struct Fmt;
template <>
struct Fmt<float> {
  static constexpr int V = 4, LP = kBK + 1;
};
template <>
struct Fmt<uint16_t> {
  static constexpr int V = 8, LP = kBK + 8;
};

template <typename T>
struct Vec {
  T v[Fmt<T>::V];
};

// V consecutive elements from p (`n` of them in range, the rest zero); one
// vector access where all are in range and p is aligned.
template <typename T>
__device__ __forceinline__ Vec<T> load_run(const T* p, int n, bool aligned) {
  constexpr int V = Fmt<T>::V;
  Vec<T> r;
  if (n >= V && aligned) {
    __builtin_memcpy(&r, p, sizeof(r));  // one 16-byte load
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) r.v[e] = e < n ? p[e] : T(0);
  }
  return r;
}

// A lane's share of one k-step's tiles: kLoads vector loads of A and of B.
template <typename T>
struct Stage {
  static constexpr int V = Fmt<T>::V;
  static constexpr int kLoads = kBM * kBK / V / kThreads;  // the same for B (kBN = kBM)
  Vec<T> a[kLoads], b[kLoads];
};

// Loads the A and B tiles of batch b at (m0, n0, k0).  Contiguous runs go to
// consecutive lanes in groups that the LDS writes spread over all banks
// (see store_stage).
template <typename T>
__device__ __forceinline__ void load_stage(const Params& P, const T* __restrict__ A, const T* __restrict__ B, int b,
                                           int m0, int n0, int k0, Stage<T>& s) {
  constexpr int V = Fmt<T>::V;
  const T* Ab = A + b * P.sA;
  const T* Bb = B + b * P.sB;
#pragma unroll
  for (int i = 0; i < Stage<T>::kLoads; ++i) {
    const int idx = threadIdx.x + i * kThreads;
    if (P.a_kc) {
      // runs along k: idx -> (m, kq), kBK / V runs per row
      const int kq = idx % (kBK / V), m = idx / (kBK / V);
      const int gm = m0 + m, gk = k0 + kq * V;
      const T* p = Ab + (long long)gm * P.am + gk;
      s.a[i] = load_run<T>(p, gm < P.M ? P.K - gk : 0, ((uintptr_t)p & 15) == 0);
    } else {
      // runs along m
      const int mq = idx % 8 + 8 * (idx / (8 * kBK)), k = (idx / 8) % kBK;
      const int gm = m0 + mq * V, gk = k0 + k;
      const T* p = Ab + (long long)gk * P.ak + gm;
      s.a[i] = load_run<T>(p, gk < P.K ? P.M - gm : 0, ((uintptr_t)p & 15) == 0);
    }
    if (P.b_nc) {
      // runs along n
      const int nq = idx % 8 + 8 * (idx / (8 * kBK)), k = (idx / 8) % kBK;
      const int gn = n0 + nq * V, gk = k0 + k;
      const T* p = Bb + (long long)gk * P.bk + gn;
      s.b[i] = load_run<T>(p, gk < P.K ? P.N - gn : 0, ((uintptr_t)p & 15) == 0);
    } else {
      // runs along k
      const int kq = idx % (kBK / V), n = idx / (kBK / V);
      const int gn = n0 + n, gk = k0 + kq * V;
      const T* p = Bb + (long long)gn * P.bn + gk;
      s.b[i] = load_run<T>(p, gn < P.N ? P.K - gk : 0, ((uintptr_t)p & 15) == 0);
    }
  }
}

template <typename T>
__device__ __forceinline__ void store_stage(const Params& P, const Stage<T>& s, T* As, T* Bs) {
  constexpr int V = Fmt<T>::V, LP = Fmt<T>::LP;
#pragma unroll
  for (int i = 0; i < Stage<T>::kLoads; ++i) {
    const int idx = threadIdx.x + i * kThreads;
    if (P.a_kc) {
      const int kq = idx % (kBK / V), m = idx / (kBK / V);
#pragma unroll
      for (int e = 0; e < V; ++e) As[m * LP + kq * V + e] = s.a[i].v[e];
    } else {
      const int mq = idx % 8 + 8 * (idx / (8 * kBK)), k = (idx / 8) % kBK;
#pragma unroll
      for (int e = 0; e < V; ++e) As[(mq * V + e) * LP + k] = s.a[i].v[e];
    }
    if (P.b_nc) {
      const int nq = idx % 8 + 8 * (idx / (8 * kBK)), k = (idx / 8) % kBK;
#pragma unroll
      for (int e = 0; e < V; ++e) Bs[(nq * V + e) * LP + k] = s.b[i].v[e];
    } else {
      const int kq = idx % (kBK / V), n = idx / (kBK / V);
#pragma unroll
      for (int e = 0; e < V; ++e) Bs[n * LP + kq * V + e] = s.b[i].v[e];
    }
  }
}

// The wave's 64 x 64 block at (wm, wn) of the tile: acc[i][j] += A rows
// wm + 32 i .. times B columns wn + 32 j .. over the k-step.
__device__ __forceinline__ void mma_step(const float* As, const float* Bs, int wm, int wn, f32x16 (&acc)[2][2]) {
  constexpr int LP = Fmt<float>::LP;
  const int l = threadIdx.x & 63, r = l & 31, h = l >> 5;
#pragma unroll
  for (int kk = 0; kk < kBK; kk += 2) {
    float a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) a[i] = As[(wm + 32 * i + r) * LP + kk + h];
#pragma unroll
    for (int j = 0; j < 2; ++j) b[j] = Bs[(wn + 32 * j + r) * LP + kk + h];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
  }
}

__device__ __forceinline__ void mma_step(const uint16_t* As, const uint16_t* Bs, int wm, int wn,
                                         f32x16 (&acc)[2][2]) {
  constexpr int LP = Fmt<uint16_t>::LP;
  const int l = threadIdx.x & 63, r = l & 31, h = l >> 5;
#pragma unroll
  for (int kk = 0; kk < kBK; kk += 16) {
    bf16x8 a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) a[i] = *reinterpret_cast<const bf16x8*>(As + (wm + 32 * i + r) * LP + kk + 8 * h);
#pragma unroll
    for (int j = 0; j < 2; ++j) b[j] = *reinterpret_cast<const bf16x8*>(Bs + (wn + 32 * j + r) * LP + kk + 8 * h);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
}

// sum == 0: C_b (the output, type T) for batch blockIdx.z; sum == 1: the
// float32 partial tile of batch group blockIdx.z (batches summed).
template <typename T>
__global__ __launch_bounds__(kThreads) void pw_gemm(Params P, const T* __restrict__ A, const T* __restrict__ B,
                                                    void* __restrict__ out) {
  constexpr int LP = Fmt<T>::LP;
  __shared__ __align__(16) T As[kBM * LP];
  __shared__ __align__(16) T Bs[kBN * LP];
  const int n0 = blockIdx.x * kBN, m0 = blockIdx.y * kBM;
  const int w = threadIdx.x >> 6, wm = (w & 1) * 64, wn = (w >> 1) * 64;
  const int b0 = P.sum ? blockIdx.z * P.per_split : blockIdx.z;
  const int b1 = P.sum ? min(P.nbatch, b0 + P.per_split) : b0 + 1;
  const int nk = (P.K + kBK - 1) / kBK;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  Stage<T> s;
  load_stage<T>(P, A, B, b0, m0, n0, 0, s);
  for (int b = b0, t = 0; b < b1;) {
    __syncthreads();  // the previous step's reads of the tiles are done
    store_stage<T>(P, s, As, Bs);
    __syncthreads();
    // the next step: its loads are in flight during this step's products
    int nb = b, nt = t + 1;
    if (nt == nk) {
      nt = 0;
      ++nb;
    }
    if (nb < b1) load_stage<T>(P, A, B, nb, m0, n0, nt * kBK, s);
    mma_step(As, Bs, wm, wn, acc);
    b = nb;
    t = nt;
  }
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + 32 * j + (l & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm + 32 * i + 8 * (e >> 2) + 4 * (l >> 5) + (e & 3);
        if (m < P.M && n < P.N) {
          if (P.sum)
            static_cast<float*>(out)[((long long)blockIdx.z * P.M + m) * P.N + n] = acc[i][j][e];
          else
            static_cast<T*>(out)[b0 * P.sC + (long long)m * P.cm + (long long)n * P.cn] = from_f32<T>(acc[i][j][e]);
        }
      }
    }
}

template <typename T>
hipError_t gemm_t(const Params& p, const void* A, const void* B, void* out, hipStream_t stream) {
  const dim3 grid((unsigned)p.tn, (unsigned)p.tm, (unsigned)(p.sum ? p.nsplit : p.nbatch));
  hipLaunchKernelGGL(pw_gemm<T>, grid, dim3(kThreads), 0, stream, p, static_cast<const T*>(A),
                     static_cast<const T*>(B), out);
  return hipGetLastError();
}

}  // namespace
}  // namespace pw
}  // namespace o1d
