// Host-side plan of the general ("gen") kernels: forward pass, input
// gradient, weight gradient and both gradients in one pass of the oriented
// 1D depthwise convolution for any plane size, any element alignment,
// stride >= 1, K <= 127, both discretisations of Eq. (2) (offsets rounded
// down, or bilinear interpolation at the unrounded offsets) and both memory
// layouts (NCHW, NHWC).  The plan depends only on sizes, never on device
// data.
//
// A workgroup owns one band of output rows and columns of CB channels and a
// run of images.  Per pass it stages G images' bands of the source plane
// (x for the forward pass and the weight gradient; for the input gradient dy
// spread onto the stride-`str` lattice, zeros between, so that the input
// gradient is a plain gather with mirrored offsets) in LDS with a zero
// margin, then every lane computes RP outputs of one column.
#pragma once

#include <stddef.h>

#include "o1d_launch.h"
#include "o1d_plan.h"

namespace o1d {
namespace gen {

constexpr int kThreads = 256;
constexpr int kMaxK = 127;
constexpr int kMaxCells = 4 * kMaxK;    // bilinear: four corners per tap
// Staged tiles per workgroup.  Gathers: up to 78 KB, the largest that keeps
// two workgroups per CU (LDS is granted in 1 KB steps out of slightly less
// than 160 KB): taller bands re-stage fewer margin rows.  The NCHW weight
// gradient and fused backward keep 64 KB: their per-cell sums hold more
// registers, and the smaller tiles keep more of them resident (measured
// faster; NHWC, whose bands are shorter, gains from the taller bands).
constexpr size_t kTileBudget = 78 * 1024;
constexpr size_t kTileBudgetSums = 64 * 1024;
constexpr int kXcds = 8;                // blocks are dealt round-robin to the eight XCDs

enum Op { kFwd = 0, kDgrad = 1, kWgrad = 2, kBwd = 3 };
enum Layout { kNCHW = 0, kNHWC = 1 };

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

struct Params {
  int N, C, H, W, K;  // input plane H x W
  int P, Q;           // forward output plane: P = (H - 1) / str + 1
  int str, mode, op, sign;
  int OH, OW;         // this op's output plane (forward and weight gradient: P x Q; input gradient: H x W)
  int SH, SW;         // staged plane (forward and weight gradient: x, H x W; input gradient: dy, P x Q)
  int sig;            // tile rows / columns per output step (forward: str; input gradient: 1)
  int dil;            // lattice step of the staged plane in the tile (input gradient: str; else 1)
  int hp;             // zero margin: K / 2, plus one for bilinear interpolation
  int RP;             // outputs per lane (consecutive rows of one column)
  int BP, BQ;         // output band
  int nbp, nbq;       // bands along rows and columns
  int NRG;            // row groups per band = BP / RP
  int TR, TC;         // tile rows and row stride (floats)
  int TW;             // floats per tile (odd)
  int OS;             // floats per output-band tile (BP BQ, odd)
  int G;              // images per pass
  int CB, lcb;        // channels per workgroup (a power of two; NCHW: 1) and its log2
  int ncb;            // channel blocks = ceil(C / CB)
  int npw;            // images per workgroup
  int nchunk;         // image runs = ceil(N / npw)
  int nblocks;        // workgroups = nbp nbq nchunk ncb
  int xcd_per;        // workgroups per XCD in the XCD-aware order (0: plain order)
  int ncap;           // cell slots per channel
  int KB, nck;        // weight gradients: per-cell sums held per lane (32, 64 or 128) and cell groups of KB
  int cell_off, tile_off, band_off, red_off;  // LDS word offsets
};

struct Plan {
  Params p{};
  size_t lds_bytes = 0;
  size_t parts = 0;  // weight gradient: partial rows per channel
  bool ok = false;
};

// Output size along one axis for a centred odd kernel (the reading of Eq. 2's
// P and Q taken here): floor((n - 1) / str) + 1.
inline int out_size(int n, int str) { return (n - 1) / str + 1; }

inline Plan plan_gen(int op, int layout, int N, int C, int H, int W, int K, int str, int mode, int esize) {
  Plan pl;
  Params& p = pl.p;
  if (N < 1 || C < 1 || H < 1 || W < 1 || K < 1 || K > kMaxK || str < 1 || (mode != 0 && mode != 1)) return pl;
  if (op == kBwd && (layout != kNCHW || str != 1 || mode != 0)) return pl;
  p.N = N; p.C = C; p.H = H; p.W = W; p.K = K;
  p.str = str; p.mode = mode; p.op = op; p.sign = (op == kDgrad || op == kBwd) ? -1 : 1;
  p.P = out_size(H, str);
  p.Q = out_size(W, str);
  p.hp = K / 2 + (mode == 1 ? 1 : 0);
  if (op == kDgrad || op == kBwd) {
    p.OH = H; p.OW = W; p.SH = p.P; p.SW = p.Q; p.sig = 1; p.dil = str;
  } else {
    p.OH = p.P; p.OW = p.Q; p.SH = H; p.SW = W; p.sig = str; p.dil = 1;
  }
  const size_t budget = layout == kNCHW && (op == kWgrad || op == kBwd) ? kTileBudgetSums : kTileBudget;
  p.ncap = (K * (mode == 1 ? 4 : 1) + 7) & ~7;  // whole groups of eight cells
  p.KB = p.ncap <= 32 ? 32 : (p.ncap <= 64 ? 64 : 128);
  // outputs per lane: four for short planes, and where the weight gradients
  // hold more than 32 per-cell sums per lane (registers)
  p.RP = (p.OH <= 16 || ((op == kWgrad || op == kBwd) && p.KB > 32)) ? 4 : 8;
  p.nck = cdiv(p.ncap, p.KB);
  auto tc_of = [&](int bq) { return (bq - 1) * p.sig + 2 * p.hp + 1; };
  auto tr_of = [&](int bp) { return (bp - 1) * p.sig + 2 * p.hp + 1; };
  // the band's output tile (dy of the weight gradient and the fused
  // backward, x of the fused backward, the NHWC output) is staged too
  const bool band_tile = op == kWgrad || op == kBwd || layout == kNHWC;
  const int band_tiles = op == kBwd ? 2 : (band_tile ? 1 : 0);
  auto bytes_of = [&](int bp, int bq) {
    const size_t tw = (size_t)tr_of(bp) * tc_of(bq) | 1;
    const size_t os = (size_t)bp * bq | 1;
    return (tw + band_tiles * os) * 4 * p.CB;
  };
  // NHWC stages 16-byte channel runs per pixel (no more channels than
  // exist), fewer where the channels' tiles do not fit
  p.CB = 1;
  if (layout == kNHWC) {
    p.CB = esize == 2 ? 8 : 4;
    while (p.CB > 1 && p.CB / 2 >= C) p.CB /= 2;
  }
  for (;; p.CB /= 2) {
    // columns: the whole output width while a band of RP rows fits
    p.BQ = p.OW;
    while (p.BQ > 8 && bytes_of(p.RP, p.BQ) > budget) p.BQ = cdiv(p.BQ, 2);
    // rows: as many as fit, in row groups of RP
    p.BP = cdiv(p.OH, p.RP) * p.RP;
    while (p.BP > p.RP && bytes_of(p.BP, p.BQ) > budget) p.BP -= p.RP;
    if (bytes_of(p.BP, p.BQ) <= budget || p.CB == 1) break;
  }
  if (bytes_of(p.BP, p.BQ) > kMaxLdsBytes / 2) return pl;
  p.lcb = 0;
  while ((1 << p.lcb) < p.CB) ++p.lcb;
  p.NRG = p.BP / p.RP;
  p.nbp = cdiv(p.OH, p.BP);
  p.nbq = cdiv(p.OW, p.BQ);
  p.TC = tc_of(p.BQ);
  p.TR = tr_of(p.BP);
  p.TW = p.TR * p.TC | 1;  // odd: channel tiles start on different banks
  p.OS = p.BP * p.BQ | 1;
  // images per pass: lanes for every task, within the tile budget
  const int tasks = p.CB * p.NRG * p.BQ;
  p.G = 1;
  if (tasks < kThreads) p.G = kThreads / tasks;
  if (p.G > N) p.G = N;
  const size_t per_img = ((size_t)p.TW + (size_t)band_tiles * p.OS) * 4 * p.CB;
  while (p.G > 1 && (size_t)p.G * per_img > budget) --p.G;
  p.ncb = cdiv(C, p.CB);
  // LDS: cell tables (offset and weight, tap, coefficient per cell and
  // channel, the cell count per channel), tiles, band tiles, the
  // weight-gradient reduction area
  p.cell_off = 0;
  p.tile_off = 4 * p.ncap * p.CB + p.CB;
  p.band_off = p.tile_off + p.G * p.CB * p.TW;
  p.red_off = p.band_off + p.G * p.CB * band_tiles * p.OS;
  size_t words = (size_t)p.red_off;
  if (op == kWgrad || op == kBwd) words += (size_t)(kThreads / 64) * p.KB + (size_t)p.CB * K;
  pl.lds_bytes = words * 4;
  if (pl.lds_bytes > kMaxLdsBytes) return pl;
  // images per workgroup: a multiple of G, enough workgroups to fill 256 CUs
  // four times over
  const long long bands = (long long)p.nbp * p.nbq * p.ncb;
  int npw = cdiv(N, p.G) * p.G;
  while (npw > p.G && bands * cdiv(N, npw) < 1024) npw -= p.G;
  p.npw = npw;
  p.nchunk = cdiv(N, npw);
  // 32-bit element offsets within one tensor
  const long long elems = (long long)N * C * (long long)H * W;
  const long long oelems = (long long)N * C * (long long)p.P * p.Q;
  if (elems >= (1ll << 31) || oelems >= (1ll << 31)) return pl;
  const long long nblocks = bands * p.nchunk;
  if (nblocks > 0x7fffffffll) return pl;
  p.nblocks = (int)nblocks;
  p.xcd_per = p.nblocks % kXcds == 0 ? p.nblocks / kXcds : 0;
  pl.parts = (size_t)p.nbp * p.nbq * p.nchunk;
  pl.ok = true;
  return pl;
}

}  // namespace gen

// One translation unit per storage type; see o1d_gen_kernels.h.
#define O1D_GEN_DECL(T)                                                                                          \
  hipError_t launch_gen_gather_##T(const gen::Plan& pl, int layout, const void* in, const void* w,             \
                                   const float* theta, void* out, hipStream_t stream);                         \
  hipError_t launch_gen_wgrad_##T(const gen::Plan& pl, int layout, const void* x, const void* dy,              \
                                  const float* theta, void* dw, float* partial, hipStream_t stream);          \
  hipError_t launch_gen_bwd_##T(const gen::Plan& pl, const void* x, const void* dy, const void* w,             \
                                const float* theta, void* dx, void* dw, float* partial, hipStream_t stream);
O1D_GEN_DECL(f32)
O1D_GEN_DECL(bf16)
#undef O1D_GEN_DECL

inline hipError_t launch_gen_gather(Dtype dt, const gen::Plan& pl, int layout, const void* in, const void* w,
                                    const float* theta, void* out, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_gen_gather_f32(pl, layout, in, w, theta, out, stream)
                          : launch_gen_gather_bf16(pl, layout, in, w, theta, out, stream);
}

inline hipError_t launch_gen_wgrad(Dtype dt, const gen::Plan& pl, int layout, const void* x, const void* dy,
                                   const float* theta, void* dw, float* partial, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_gen_wgrad_f32(pl, layout, x, dy, theta, dw, partial, stream)
                          : launch_gen_wgrad_bf16(pl, layout, x, dy, theta, dw, partial, stream);
}

inline hipError_t launch_gen_bwd(Dtype dt, const gen::Plan& pl, const void* x, const void* dy, const void* w,
                                 const float* theta, void* dx, void* dw, float* partial, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_gen_bwd_f32(pl, x, dy, w, theta, dx, dw, partial, stream)
                          : launch_gen_bwd_bf16(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace o1d
