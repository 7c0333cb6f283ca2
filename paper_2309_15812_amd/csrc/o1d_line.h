// Host-side plan of the line kernels (o1d_line.hip): depthwise convolution
// with oriented 1D kernels for K <= 63 and planes whose haloed tile fits in
// LDS.  The plan depends only on (N, C, H, W, K): the angles stay on the
// device and every workgroup derives its channel's geometry itself, so the
// plan reserves room for both staging frames (the plane and its transpose)
// and both strip shapes (vertical strips of kRv outputs, diagonal strips of
// kRd outputs).
#pragma once

#include <stddef.h>
#include <stdlib.h>

#include "o1d_launch.h"
#include "o1d_plan.h"
#include "o1d_strip.h"

namespace o1d {
namespace line {

constexpr int kThreads = 256;  // 4 waves per workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kMaxTaps = 63;   // wave 0 builds the program with one tap per lane
constexpr int kMaxSlots = 16;  // staged elements per thread per plane group
constexpr int kMaxIt = 4;      // strip tasks per lane per plane group
constexpr int kRv = 14;        // outputs per vertical strip
constexpr int kRd = 7;         // outputs per diagonal strip
constexpr int kGuard = 8;      // zero floats before and after every tile slot
constexpr int kProgFloats = 208;  // sizeof the per-channel program in LDS (floats)
constexpr size_t kLdsBudget = 80 * 1024;

// Odd tile row strides compiled into the kernels (an odd stride keeps the
// transposed staging writes of a half-wave on 32 distinct banks).
#define O1D_LINE_STRIDES(X) X(23) X(31) X(47) X(63) X(71) X(87) X(103) X(119) X(143)
constexpr int kStrides[] = {23, 31, 47, 63, 71, 87, 103, 119, 143};

__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Strip tiling of one staging frame (Hs rows x Ws columns) for strips of R
// outputs along u = (1, s): bands of R rows; within a band one strip per
// column j in [jlo, jlo + nj) (diagonal strips start up to R - 1 columns
// outside the plane so that their outputs cover every column).  A task is
// a segment of up to segw strips of one band of one plane; tpw tasks share
// a wave.
struct Tiling {
  int nb, nj, jlo, segw, nseg, tpw;
};

__host__ __device__ inline Tiling tiling(int Hs, int Ws, int R, int s) {
  Tiling t;
  t.nb = cdiv(Hs, R);
  t.nj = Ws + (s != 0 ? R - 1 : 0);
  t.jlo = s > 0 ? -(R - 1) : 0;
  t.segw = t.nj <= 16 ? 16 : (t.nj <= 32 ? 32 : 64);
  t.nseg = cdiv(t.nj, t.segw);
  t.tpw = 64 / t.segw;
  return t;
}

struct LineParams {
  int N, C, H, W, K, sign;
  int G;      // planes staged in LDS at once
  int npw;    // images per workgroup
  int halo;   // zero rows/columns around the plane in the tile (>= every kept cell offset)
  int TR;     // tile rows per slot
  int PS;     // floats per tile slot (including the guards)
  int OS;     // row stride of the output bounce tile (= S)
  int OPS;    // floats per output bounce slot
  int GS;     // row stride of the weight-gradient dy tile (= S)
  int GPS;    // floats per dy slot
  int aux;    // float offset of the bounce / dy area in dynamic LDS
  int red;    // float offset of the per-wave reduction area (weight gradient)
  int trash;  // float offset of the trash area (staging writes of slots outside the plane)
  int ks;     // staging: row steps per plane (32 rows each)
  int ms;     // staging: column segments per plane (32 columns each)
};

struct LinePlan {
  LineParams p{};
  int S = 0;
  int KB = 0;  // cell bound compiled into the kernel: 32 or 64
  int blocks_n = 0;
  size_t lds_bytes = 0;
  bool ok = false;
};

inline size_t round4(size_t v) { return (v + 3) & ~(size_t)3; }

// kind: 0 = gather (forward / input gradient), 1 = weight gradient.
// vec_ok: the tensors are aligned for vector accesses (16 bytes for float32,
// 8 bytes for bfloat16).  Staging moves 4 elements of a row per access, so
// the plan needs W % 4 == 0 and aligned tensors (else the tiled kernels run).
inline LinePlan plan_line(int N, int C, int H, int W, int K, int sign, int kind, bool vec_ok = true) {
  LinePlan pl;
  if (K < 1 || K > kMaxTaps || N < 1 || C < 1 || H < 1 || W < 1) return pl;
  if (W % 4 != 0 || !vec_ok) return pl;
  const int M = H > W ? H : W;
  const int halo = (K / 2) < (M - 1) ? (K / 2) : (M - 1);
  // rows covered by whole bands, worst case over both frames and strip shapes
  int cover = 0;
  for (int f = 0; f < 2; ++f)
    for (int v = 0; v < 2; ++v) {
      const int R = v ? kRd : kRv;
      const Tiling t = tiling(f ? W : H, f ? H : W, R, v);
      if (t.nb * R > cover) cover = t.nb * R;
    }
  // one compile-time row stride serves the input tile (M + 2 halo columns),
  // the dy tile (M + 12: six zero columns either side) and the output bounce
  // tile (band rows up to `cover`)
  int need = M + 2 * halo;
  if (M + 12 > need) need = M + 12;
  if (cover > need) need = cover;
  int S = 0;
  for (int s : kStrides)
    if (s >= need) {
      S = s;
      break;
    }
  if (S == 0) return pl;
  LineParams& p = pl.p;
  p.N = N; p.C = C; p.H = H; p.W = W; p.K = K; p.sign = sign;
  p.halo = halo;
  p.TR = cover + 2 * halo;
  p.PS = (int)round4((size_t)p.TR * S + 2 * kGuard);
  p.OS = S;
  p.OPS = (int)round4((size_t)H * S);
  p.GS = S;
  p.GPS = (int)round4((size_t)cover * S);
  const long long HW = (long long)H * W;
  // staging (see o1d_line_kernels.h): kMaxSlots / 4 vector slots per thread,
  // each a step of 32 rows and a segment of 32 columns of one plane
  if (W > 64) return pl;
  const int ks = cdiv(H, 32), ms = cdiv(W, 32);
  const int gmax_slots = (kMaxSlots / 4) / (ks * ms);
  if (gmax_slots < 1) return pl;
  p.ks = ks;
  p.ms = ms;
  // trash area: a word per lane plus the reach of a transposed vector write
  const int trash = (int)round4((size_t)(64 + 3 * S + 4));
  auto lds_for = [&](int g) -> size_t {
    size_t f = (size_t)kProgFloats + (size_t)g * p.PS;
    f += (size_t)g * (kind == 0 ? p.OPS : p.GPS);
    if (kind == 1) f += (size_t)kWaves * 64;
    f += (size_t)trash;
    return f * 4;
  };
  // lane iterations per plane group, worst case over frames and strip shapes
  auto iters = [&](int g) {
    int m = 0;
    for (int f = 0; f < 2; ++f)
      for (int v = 0; v < 2; ++v) {
        const Tiling t = tiling(f ? W : H, f ? H : W, v ? kRd : kRv, v);
        const int it = cdiv(g * t.nb * t.nseg, kWaves * t.tpw);
        if (it > m) m = it;
      }
    return m;
  };
  // planes per group: enough vertical-strip tasks to occupy the four waves,
  // bounded by the batch, the staging registers, the lane task slots and LDS
  int G = 1;
  for (int f = 0; f < 2; ++f) {
    const Tiling t = tiling(f ? W : H, f ? H : W, kRv, 0);
    const int need = cdiv(kWaves * t.tpw, t.nb * t.nseg);
    if (need > G) G = need;
  }
  if (G > N) G = N;
  if (G > gmax_slots) G = gmax_slots;
  while (G > 1 && (lds_for(G) > kLdsBudget || iters(G) > kMaxIt)) --G;
  if (iters(G) > kMaxIt) return pl;
  if (lds_for(G) > kMaxLdsBytes) return pl;
  // buffer resources cover a group in bytes (float32 at most), below 2^31
  if ((long long)(G + 1) * C * HW * 4 >= (1ll << 31)) return pl;
  p.G = G;
  p.aux = kProgFloats + G * p.PS;
  p.red = p.aux + G * (kind == 0 ? p.OPS : p.GPS);
  p.trash = p.red + (kind == 1 ? kWaves * 64 : 0);
  // Images per workgroup for about three resident workgroups per CU (at
  // most three by VGPRs, fewer when LDS runs out), fitted like the strip
  // kernels' grids.  The choice depends on the sizes only, so the
  // weight-gradient workspace size is a function of (N, C, H, W, K).
  const size_t lds = lds_for(G);
  int per_cu = strip::lds_resident(lds);
  if (per_cu > 3) per_cu = 3;
  if (per_cu < 1) per_cu = 1;
  const int npw = strip::fit_npw(N, C, G, 256LL * per_cu);
  p.npw = npw;
  pl.S = S;
  pl.KB = K <= 32 ? 32 : 64;
  pl.blocks_n = cdiv(N, npw);
  pl.lds_bytes = lds;
  pl.ok = true;
  return pl;
}

}  // namespace line

// One translation unit per (kind, storage type); see o1d_line_kernels.h.
hipError_t launch_gather_line_f32(const line::LinePlan& pl, const void* in, const void* w, const float* theta,
                                  void* out, hipStream_t stream);
hipError_t launch_gather_line_bf16(const line::LinePlan& pl, const void* in, const void* w, const float* theta,
                                   void* out, hipStream_t stream);
hipError_t launch_wgrad_line_f32(const line::LinePlan& pl, const void* x, const void* dy, const float* theta,
                                 void* dw, float* partial, hipStream_t stream);
hipError_t launch_wgrad_line_bf16(const line::LinePlan& pl, const void* x, const void* dy, const float* theta,
                                  void* dw, float* partial, hipStream_t stream);

inline hipError_t launch_gather_line(Dtype dt, const line::LinePlan& pl, const void* in, const void* w,
                                     const float* theta, void* out, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_gather_line_f32(pl, in, w, theta, out, stream)
                          : launch_gather_line_bf16(pl, in, w, theta, out, stream);
}

inline hipError_t launch_wgrad_line(Dtype dt, const line::LinePlan& pl, const void* x, const void* dy,
                                    const float* theta, void* dw, float* partial, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_wgrad_line_f32(pl, x, dy, theta, dw, partial, stream)
                          : launch_wgrad_line_bf16(pl, x, dy, theta, dw, partial, stream);
}

}  // namespace o1d
