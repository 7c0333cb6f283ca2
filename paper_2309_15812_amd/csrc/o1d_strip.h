// Host-side plan of the strip kernels: forward pass, input gradient and
// weight gradient of the oriented 1D depthwise convolution for K <= 63 and planes
// whose haloed tile fits in LDS.  The plan depends only on (N, C, H, W, K):
// angles stay on the device and every workgroup derives its channel's line
// itself, so the plan covers both staging frames (the plane and its
// transpose) and both strip shapes (vertical and diagonal).
#pragma once

#include <stddef.h>

#include "o1d_launch.h"
#include "o1d_plan.h"

namespace o1d {
namespace strip {

constexpr int kWaves = 2;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxTaps = 63;  // wave 0 builds the program with one tap per lane
// Strip shapes: a lane computes NC adjacent strips of R outputs.  Vertical
// strips step u = (1, 0) in the staging frame, diagonal ones u = (1, +-1).
// The lanes of a half-wave read 32 distinct LDS banks: vertical strips sit
// on consecutive columns; diagonal blocks (4 columns apart) are laid out as
// 8 blocks x 4 bands per half-wave, the bands being 7 S (odd) rows apart.
constexpr int kRv = 28, kNv = 1;
constexpr int kRd = 7, kNd = 4;
constexpr int kGuard = 16;       // floats before and after every tile slot
constexpr int kProgWords = 208;  // the per-channel program in LDS
constexpr int kMaxSlots = 8;     // staging slots (4 elements each) per lane and group
constexpr size_t kLdsBudget = 64 * 1024;

// Odd tile row strides compiled into the kernels: for an odd stride the
// transposed staging accesses of a half-wave hit 32 distinct banks.
#define O1D_STRIP_STRIDES(X) X(47) X(51) X(63) X(77) X(87) X(103) X(119) X(143)
constexpr int kStrides[] = {47, 51, 63, 77, 87, 103, 119, 143};

__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Workgroups of `lds_bytes` dynamic LDS that stay resident on one CU: LDS is
// granted in 1 KB steps and a little of the 160 KB is not available, so five
// workgroups of 32 KB do not fit (measured: four are resident).
inline int lds_resident(size_t lds_bytes) {
  const size_t granted = (lds_bytes + 1023) / 1024 * 1024;
  return granted ? (int)((kMaxLdsBytes - 512) / granted) : 1;
}

// Images per workgroup (a multiple of G) for `slots` resident workgroups:
// the grid of C * ceil(N / npw) workgroups runs in ceil(grid / slots)
// rounds, each costing npw planes plus about 1.5 planes of workgroup set-up
// (program, zeroed tile, the first group's exposed load); npw minimises
// that, the most planes per workgroup among equals.
inline int fit_npw(int N, int C, int G, long long slots) {
  if (slots < 1) slots = 1;
  double best = -1.0;
  int npw = cdiv(N, G) * G;
  for (int n = G; n <= cdiv(N, G) * G; n += G) {
    const long long grid = (long long)C * cdiv(N, n);
    const double span = (double)((grid + slots - 1) / slots) * (n + 1.5);
    if (best < 0 || span <= best) {
      best = span;
      npw = n;
    }
  }
  return npw;
}

// Task grid of one staging frame (Hs rows x Ws columns) for the strip shape
// of step s: nb bands of R rows; strip columns j in [jlo, jlo + nj) (a
// diagonal strip's R outputs cover columns j .. j + s (R - 1), so strips
// start up to R - 1 columns outside the plane); ncg groups of NC adjacent
// strips per band.  A task = one group of one band of one plane.
// Lanes per plane (ppt): vertical tasks one per lane, band after band;
// diagonal tasks in half-wave blocks of 8 column groups x 4 bands, unless
// the plane is so small that the blocks leave enough lanes idle to cost a
// plane per group: then one per lane, band after band (dense).  In the
// band-after-band layouts a band takes lpb >= ncg lanes: rounded up to a
// whole wave (else half-wave) where that costs no plane per group, so that
// the lanes of one wave read one band's consecutive columns (two bands in a
// wave map their columns onto overlapping LDS banks).
// A dense diagonal layout whose bands come in fours and whose bands hold
// more than 8 column groups is split instead: the first 8 q column groups
// (q = ncg / 8) of every plane of the group in half-wave blocks as above,
// plane after plane, then the remaining column groups of all the planes,
// band after band.  A band of 9 or more groups 4 columns apart spans more
// than 32 banks, so band after band its first and ninth lanes would share a
// bank in every read; split, every half-wave of blocks is conflict-free.
struct Shape {
  int R, NC, nb, nj, jlo, ncg, ppt;
  int bq, bb;  // diagonal: half-wave blocks along the column groups and along the bands
  int dense;   // tasks one per lane, band after band
  int lpb;     // band-after-band layouts: lanes per band
  int split;   // dense diagonal layout split into blocks and a remainder
};

__host__ __device__ inline Shape shape_of(int Hs, int Ws, int s) {
  Shape t;
  t.R = s ? kRd : kRv;
  t.NC = s ? kNd : kNv;
  t.nb = cdiv(Hs, t.R);
  t.nj = Ws + (s ? t.R - 1 : 0);
  t.jlo = s > 0 ? -(t.R - 1) : 0;
  t.ncg = cdiv(t.nj, t.NC);
  t.bq = cdiv(t.ncg, 8);
  t.bb = cdiv(t.nb, 4);
  const int blocked = 32 * t.bq * t.bb, dense = t.nb * t.ncg;
  t.dense = !s || kThreads / dense > kThreads / blocked;
  t.lpb = t.ncg;
  if (t.dense) {
    const int planes = kThreads / dense;
    for (int a = 64; a >= 32; a /= 2) {
      const int l = cdiv(t.ncg, a) * a;
      if (t.nb * l <= kThreads && kThreads / (t.nb * l) == planes) {
        t.lpb = l;
        break;
      }
    }
  }
  t.ppt = t.dense ? t.nb * t.lpb : blocked;
  t.split = s && t.dense && t.nb % 4 == 0 && t.ncg > 8 && t.lpb == t.ncg;
  return t;
}

struct Params {
  int N, C, H, W, K, sign;
  int G;      // planes staged at once (one task per lane for all of them)
  int npw;    // images per workgroup
  int halo;   // zero rows above and below the plane in the tile
  int mc;     // columns a walk reads past either side of the plane; the zero gap between
              // consecutive tile rows (S - max(H, W) >= mc) serves as the right margin of one
              // row and the left margin of the next
  int TR;     // tile rows
  int PS;     // floats per tile slot, guards included
  int ks, ms; // staging grid per plane: steps of 8 kWaves rows, segments of 32 columns
  int nq;     // staging slots per group = G ks ms
  int trash;  // float offset of the trash area (writes of slots outside the plane)
};

struct Plan {
  Params p{};
  int S = 0;
  int KB = 0;  // cell bound compiled into the walk: 32 or 64
  int blocks_n = 0;
  size_t lds_bytes = 0;
  bool ok = false;
};

// kind: 0 = gather (forward / input gradient), 1 = weight gradient, 2 =
// fused backward (the weight gradient's layout).
// vec_ok: tensors aligned for 4-element vector accesses.
inline Plan plan_strip(int N, int C, int H, int W, int K, int sign, int kind, bool vec_ok) {
  Plan pl;
  if (K < 1 || K > kMaxTaps || N < 1 || C < 1 || H < 1 || W < 1 || kind < 0 || kind > 2) return pl;
  if (kind >= 1 && K > 32) return pl;  // see launch_wgrad_strip
  if (W % 4 != 0 || !vec_ok) return pl;
  const int M = H > W ? H : W;
  const int halo = (K / 2) < (M - 1) ? (K / 2) : (M - 1);
  // Column reach: the staging frame puts the line's longer extent along its
  // rows, so a cell's column offset is at most floor((K / 2) sin 45 deg) + 1
  // in magnitude (checked by enumeration of the offsets of Eq. 2 over
  // angles, K <= 63; one more here for margin); a diagonal block adds the
  // R - 1 columns its strips start left of the plane, or its NC - 1 + R - 1
  // columns past its first strip on the right.
  const int bmax = (int)((K / 2) * 0.70711) + 2;
  const int mc = kRd - 1 + kNd - 1 + bmax;
  int cover = 0, ppt = 0;
  for (int f = 0; f < 2; ++f)
    for (int s = 0; s < 2; ++s) {
      const Shape t = shape_of(f ? W : H, f ? H : W, s);
      if (t.nb * t.R > cover) cover = t.nb * t.R;
      if (t.ppt > ppt) ppt = t.ppt;
    }
  // rows share their margins: the gap of S - M >= mc zero columns after a
  // row's data is also the left margin of the next row
  int S = 0;
  for (int s : kStrides)
    if (s >= M + mc) {
      S = s;
      break;
    }
  if (S == 0) return pl;
  Params& p = pl.p;
  p.N = N; p.C = C; p.H = H; p.W = W; p.K = K; p.sign = sign;
  p.halo = halo;
  p.mc = mc;
  p.TR = cover + 2 * halo;
  // the last row's right-hand reads run up to mc + M + mc - S columns past
  // the tile; slots are a whole number of 16-byte chunks
  const int tail = mc + M + mc - S > kGuard ? mc + M + mc - S : kGuard;
  p.PS = (p.TR * S + kGuard + tail + 3) & ~3;
  p.ks = cdiv(H, 8 * kWaves);
  p.ms = cdiv(W, 32);
  const int per_plane_slots = p.ks * p.ms;
  const int max_slots = kMaxSlots;
  // planes per group: every task of the group on its own lane
  int G = kThreads / ppt;
  if (G < 1) return pl;
  if (G > N) G = N;
  if (G * per_plane_slots > max_slots) G = max_slots / per_plane_slots;
  if (G < 1) return pl;
  const int trash = 64 + 3 * S + 4;  // a word per lane plus the reach of a transposed vector write
  const int red = kind >= 1 ? kWaves * 64 : 0;  // weight gradients: per-wave cell sums
  auto lds_for = [&](int g) { return ((size_t)kProgWords + (size_t)g * p.PS + (size_t)red + (size_t)trash) * 4; };
  while (G > 1 && lds_for(G) > kLdsBudget) --G;
  if (lds_for(G) > kMaxLdsBytes) return pl;
  // buffer resources cover a group in bytes (float32 at most), below 2^31
  const long long HW = (long long)H * W;
  if ((long long)(G + 1) * C * HW * 4 >= (1ll << 31)) return pl;
  p.G = G;
  p.nq = G * per_plane_slots;
  p.trash = kProgWords + G * p.PS + red;
  // images per workgroup: from the LDS rule and the kernel's registers
  // (waves per SIMD: the weight gradient's walk keeps 32 cell sums and the
  // window, two; the fused backward, below 168 registers, three); the
  // gather launcher refits it to the kernel's residency, the weight
  // gradients keep it (their workspace size depends on it)
  const size_t lds = lds_for(G);
  int per_cu = lds_resident(lds);
  const int by_regs = kind == 2 ? 3 * 4 / kWaves : 2 * 4 / kWaves;
  if (per_cu > by_regs) per_cu = by_regs;
  const int npw = fit_npw(N, C, G, 256LL * (per_cu < 1 ? 1 : per_cu));
  p.npw = npw;
  pl.S = S;
  pl.KB = K <= 32 ? 32 : 64;
  pl.blocks_n = cdiv(N, npw);
  pl.lds_bytes = lds;
  pl.ok = true;
  return pl;
}

}  // namespace strip

// One translation unit per storage type and cell bound; see o1d_strip_kernels.h.
#define O1D_STRIP_DECL(NAME)                                                                                   \
  hipError_t NAME(const strip::Plan& pl, const void* in, const void* w, const float* theta, void* out, \
                  hipStream_t stream);
O1D_STRIP_DECL(launch_gather_strip_f32_k32)
O1D_STRIP_DECL(launch_gather_strip_f32_k64)
O1D_STRIP_DECL(launch_gather_strip_bf16_k32)
O1D_STRIP_DECL(launch_gather_strip_bf16_k64)
#undef O1D_STRIP_DECL

#define O1D_STRIP_WDECL(NAME)                                                                                    \
  hipError_t NAME(const strip::Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial, \
                  hipStream_t stream);
O1D_STRIP_WDECL(launch_wgrad_strip_f32_k32)
O1D_STRIP_WDECL(launch_wgrad_strip_bf16_k32)
#undef O1D_STRIP_WDECL

#define O1D_STRIP_BDECL(NAME)                                                                                   \
  hipError_t NAME(const strip::Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx, \
                  void* dw, float* partial, hipStream_t stream);
O1D_STRIP_BDECL(launch_bwd_strip_f32_k32)
O1D_STRIP_BDECL(launch_bwd_strip_bf16_k32)
#undef O1D_STRIP_BDECL

// Fused backward (input and weight gradients in one pass): the weight
// gradient's plan with mirrored offsets (sign -1), walks of up to 31 cells.
inline hipError_t launch_bwd_strip(Dtype dt, const strip::Plan& pl, const void* x, const void* dy, const void* w,
                                   const float* theta, void* dx, void* dw, float* partial, hipStream_t stream) {
  if (pl.KB != 32 || pl.p.sign != -1) return hipErrorInvalidValue;
  return dt == Dtype::F32 ? launch_bwd_strip_f32_k32(pl, x, dy, w, theta, dx, dw, partial, stream)
                          : launch_bwd_strip_bf16_k32(pl, x, dy, w, theta, dx, dw, partial, stream);
}

// Weight gradient: walks of up to 32 cells (the per-cell accumulators of
// longer walks do not fit in registers next to the window; the general
// kernels take K > 31).
inline hipError_t launch_wgrad_strip(Dtype dt, const strip::Plan& pl, const void* x, const void* dy,
                                     const float* theta, void* dw, float* partial, hipStream_t stream) {
  if (pl.KB != 32) return hipErrorInvalidValue;
  return dt == Dtype::F32 ? launch_wgrad_strip_f32_k32(pl, x, dy, theta, dw, partial, stream)
                          : launch_wgrad_strip_bf16_k32(pl, x, dy, theta, dw, partial, stream);
}

inline hipError_t launch_gather_strip(Dtype dt, const strip::Plan& pl, const void* in, const void* w,
                                      const float* theta, void* out, hipStream_t stream) {
  if (dt == Dtype::F32)
    return pl.KB == 32 ? launch_gather_strip_f32_k32(pl, in, w, theta, out, stream)
                       : launch_gather_strip_f32_k64(pl, in, w, theta, out, stream);
  return pl.KB == 32 ? launch_gather_strip_bf16_k32(pl, in, w, theta, out, stream)
                     : launch_gather_strip_bf16_k64(pl, in, w, theta, out, stream);
}

}  // namespace o1d
