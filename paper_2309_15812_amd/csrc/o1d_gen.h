// Host-side plan of the general ("gen") kernels: forward pass, input
// gradient and weight gradient of the oriented 1D depthwise convolution for
// any plane size, any element alignment, stride >= 1, K <= 127, both
// discretisations of Eq. (2) (offsets rounded down, or bilinear
// interpolation at the unrounded offsets) and both memory layouts (NCHW,
// NHWC).  The plan depends only on sizes, never on device data.
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
constexpr int kMaxCells = 4 * kMaxK;  // bilinear: four corners per tap
constexpr int kChunk = 32;            // weight gradient: cells per register pass
constexpr size_t kLdsBudget = 48 * 1024;

enum Op { kFwd = 0, kDgrad = 1, kWgrad = 2 };
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
  int NRG;            // row groups per band = ceil(BP / RP)
  int TR, TC;         // tile rows and row stride (floats)
  int TW;             // floats per tile (odd)
  int G;              // images per pass
  int CB;             // channels per workgroup (NCHW: 1)
  int ncb;            // channel blocks = ceil(C / CB)
  int npw;            // images per workgroup
  int nchunk;         // image runs = ceil(N / npw)
  int cell_words;     // LDS words of the cell tables
  int tile_off;       // LDS word offset of the tiles
  int out_off;        // LDS word offset of the NHWC output / dy tile (0 if none)
  int red_off;        // LDS word offset of the weight-gradient reduction area (0 if none)
};

struct Plan {
  Params p{};
  size_t lds_bytes = 0;
  int grid_x = 0, grid_y = 0;
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
  p.N = N; p.C = C; p.H = H; p.W = W; p.K = K;
  p.str = str; p.mode = mode; p.op = op; p.sign = op == kDgrad ? -1 : 1;
  p.P = out_size(H, str);
  p.Q = out_size(W, str);
  p.hp = K / 2 + (mode == 1 ? 1 : 0);
  if (op == kDgrad) {
    p.OH = H; p.OW = W; p.SH = p.P; p.SW = p.Q; p.sig = 1; p.dil = str;
  } else {
    p.OH = p.P; p.OW = p.Q; p.SH = H; p.SW = W; p.sig = str; p.dil = 1;
  }
  p.RP = p.OH <= 16 ? 4 : 8;
  const int ncell = K * (mode == 1 ? 4 : 1);
  // columns: the whole output width when a band of RP rows fits, else bands
  auto tc_of = [&](int bq) { return (bq - 1) * p.sig + 2 * p.hp + 1; };
  auto tr_of = [&](int bp) { return (bp - 1) * p.sig + 2 * p.hp + 1; };
  p.BQ = p.OW;
  while (p.BQ > 16 && (size_t)tc_of(p.BQ) * tr_of(p.RP) * 4 > kLdsBudget / 2) p.BQ = cdiv(p.BQ, 2);
  // rows: up to one lane per (column, row group)
  const int rg_max = p.BQ >= kThreads ? 1 : kThreads / p.BQ;
  p.BP = p.RP * rg_max;
  if (p.BP > cdiv(p.OH, p.RP) * p.RP) p.BP = cdiv(p.OH, p.RP) * p.RP;
  while (p.BP > p.RP && (size_t)tc_of(p.BQ) * tr_of(p.BP) * 4 > kLdsBudget / 2) p.BP -= p.RP;
  p.NRG = cdiv(p.BP, p.RP);
  p.nbp = cdiv(p.OH, p.BP);
  p.nbq = cdiv(p.OW, p.BQ);
  p.TC = tc_of(p.BQ);
  p.TR = tr_of(p.BP);
  p.TW = p.TR * p.TC;
  if ((p.TW & 1) == 0) p.TW += 1;  // odd: channel tiles start on different banks
  const size_t tile_bytes = (size_t)p.TW * 4;
  if (tile_bytes > kMaxLdsBytes / 2) return pl;
  const int tasks = p.BQ * p.NRG;  // per image and channel
  // channels per workgroup: NHWC stages a block of channels with coalesced loads
  p.CB = 1;
  if (layout == kNHWC) {
    p.CB = esize == 2 ? 16 : 8;
    if (p.CB > C) p.CB = C;
    while (p.CB > 1 && (size_t)p.CB * tile_bytes > kLdsBudget) p.CB /= 2;
  }
  // images per pass: enough tasks for the workgroup's lanes
  p.G = 1;
  const int per_pass = p.CB * tasks;
  if (per_pass < kThreads) p.G = kThreads / per_pass;
  if (p.G > N) p.G = N;
  while (p.G > 1 && (size_t)p.G * p.CB * tile_bytes > kLdsBudget) --p.G;
  p.ncb = cdiv(C, p.CB);
  // LDS: cell tables (offset and weight, tap, coefficient per cell and
  // channel, and the cell count per channel), tiles, the NHWC output / dy
  // tile, the weight-gradient reduction area
  p.cell_words = 4 * ncell * p.CB + p.CB;
  p.tile_off = p.cell_words;
  size_t words = (size_t)p.tile_off + (size_t)p.G * p.CB * p.TW;
  p.out_off = 0;
  if (layout == kNHWC) {
    p.out_off = (int)words;
    words += (size_t)p.G * p.CB * (p.BP * p.BQ | 1);
  }
  p.red_off = 0;
  if (op == kWgrad) {
    p.red_off = (int)words;
    words += (size_t)(kThreads / 64) * kChunk + (size_t)p.CB * K;
  }
  pl.lds_bytes = words * 4;
  if (pl.lds_bytes > kMaxLdsBytes) return pl;
  // images per workgroup: a multiple of G, enough workgroups to fill 256 CUs
  // about four times over
  const long long bands = (long long)p.nbp * p.nbq * p.ncb;
  const long long want = 1024;
  int npw = cdiv(N, p.G) * p.G;
  while (npw > p.G && bands * cdiv(N, npw) < want) npw -= p.G;
  p.npw = npw;
  p.nchunk = cdiv(N, npw);
  // 32-bit element offsets within one tensor
  const long long elems = (long long)N * C * (long long)H * W;
  const long long oelems = (long long)N * C * (long long)p.P * p.Q;
  if (elems >= (1ll << 31) || oelems >= (1ll << 31)) return pl;
  if ((long long)p.nbp * p.nbq * p.nchunk > 0x7fffffffll || p.ncb > 65535) return pl;
  pl.grid_x = p.nbp * p.nbq * p.nchunk;
  pl.grid_y = p.ncb;
  pl.parts = (size_t)p.nbp * p.nbq * p.nchunk;
  pl.ok = true;
  return pl;
}

}  // namespace gen

// One translation unit per storage type; see o1d_gen_kernels.h.
#define O1D_GEN_DECL(T)                                                                                        \
  hipError_t launch_gen_gather_##T(const gen::Plan& pl, int layout, const void* in, const void* w,           \
                                   const float* theta, void* out, hipStream_t stream);                       \
  hipError_t launch_gen_wgrad_##T(const gen::Plan& pl, int layout, const void* x, const void* dy,            \
                                  const float* theta, void* dw, float* partial, hipStream_t stream);
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

}  // namespace o1d
