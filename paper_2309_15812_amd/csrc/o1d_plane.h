// Host-side plan of the plane kernels: the oriented 1D depthwise convolution
// (forward pass, input gradient, weight gradient, both gradients in one
// pass) of planes small enough that a whole plane of one channel, for a
// group of images, fits in LDS.  NCHW only; any stride, both discretisations
// of Eq. (2), K <= 127.
//
// A workgroup owns one channel and NI images.  A wave's 64 lanes are NI / 2
// image pairs times R = 128 / NI neighbouring output columns, and each lane
// computes RP outputs down its column for its two images, so every lane of a
// wave applies the same cells (tap offsets) at the same time.  The plane is
// staged in LDS as [row][column][image] (one 32-bit word per image: a lane
// reads its pair with one 64-bit access, and a wave's reads of one cell touch
// consecutive words), with a margin of only (RP - 1) rows and
// (R - 1) columns (times the stride, plus one for bilinear corners): cells
// that fall outside the plane for a whole group of RP x R outputs are not
// visited at all, instead of reading zeros from a margin of K / 2.  The
// column margin is one gap per row, shared by a row's right-hand and the
// next row's left-hand reads.
#pragma once

#include <stddef.h>

#include <algorithm>

#include "o1d_launch.h"
#include "o1d_plan.h"

namespace o1d {
namespace plane {

constexpr int kThreads = 512;  // eight waves: twice the waves per SIMD of four at the same LDS
constexpr int kWaves = kThreads / 64;
constexpr int kMaxK = 127;
constexpr size_t kLdsBudget = 80 * 1024;  // at least two workgroups per CU

enum Op { kFwd = 0, kDgrad = 1, kWgrad = 2, kBwd = 3 };

inline int cdiv(int a, int b) { return (a + b - 1) / b; }
inline size_t align16(size_t b) { return (b + 15) & ~(size_t)15; }

struct Params {
  int N, C, H, W, K;
  int str, mode, op, sign;
  int OH, OW;       // this op's output plane (forward, weight gradient: P x Q; input gradient: H x W)
  int SH, SW, dil;  // staged plane (x, or dy for the input gradients) and its lattice step in the H x W frame
  int sig;          // frame rows (columns) per output row (column): forward and weight gradient str, else 1
  int NI, lni, R;   // lanes: NI / 2 image pairs (NI a power of two, lni its log2) x R output columns
  int RP;           // output rows per lane
  int mr, mc;       // tile margins (rows, columns)
  int TRm, TCm;     // tile rows H + 2 mr; tile row stride W + mc (consecutive rows share one gap of mc
                    // zero columns as their right and left margins; mc more columns end the tile)
  int nrg, ncg;     // row groups (of RP rows) and column groups (of R columns) of the output plane
  int nitems;       // nrg ncg
  int OSz;          // elements per image of the output-shaped tile (an odd number of 32-bit words)
  int ncells;       // cell slots per channel in use at most (K, or 4 K bilinear)
  int ncap;         // table slots (room for reads past the last cell)
  int KB, nck;      // weight gradients: per-cell sums per lane, and groups of KB cells
  int vt, va;       // elements per global access: staged plane (dividing its width); output-shaped planes
  int nslot;        // cell tables in LDS
  int table_bytes;  // bytes per cell table (cells, then their runs at ival_off)
  int nchunk;       // image groups = ceil(N / NI); work items = C nchunk (channel, image group)
  int per;          // items per workgroup
  int nblocks;      // workgroups = ceil(C nchunk / per)
  int ival_off;                       // byte offset of the cell runs in a table
  int tile_off, aux_off, red_off;     // LDS byte offsets (tables start at 0)
};

struct Plan {
  Params p{};
  size_t lds_bytes = 0;
  size_t parts = 0;  // weight gradients: partial rows per channel (= nchunk)
  bool ok = false;
};

inline int out_size(int n, int str) { return (n - 1) / str + 1; }

// esize: bytes per element; aligned: the tensors' base addresses allow 16-byte
// (float32) or 8-byte (bfloat16) accesses.
inline Plan plan_plane(int op, int N, int C, int H, int W, int K, int str, int mode, int esize, bool aligned) {
  Plan best;
  if (N < 8 || C < 1 || H < 1 || W < 1 || K < 1 || K > kMaxK || str < 1 || (mode != 0 && mode != 1)) return best;
  if (op == kBwd && (str != 1 || mode != 0)) return best;
  Params q{};
  q.N = N; q.C = C; q.H = H; q.W = W; q.K = K;
  q.str = str; q.mode = mode; q.op = op; q.sign = (op == kDgrad || op == kBwd) ? -1 : 1;
  const int P = out_size(H, str), Q = out_size(W, str);
  if (op == kFwd || op == kWgrad) {
    q.OH = P; q.OW = Q; q.SH = H; q.SW = W; q.dil = 1; q.sig = str;
  } else if (op == kDgrad) {
    q.OH = H; q.OW = W; q.SH = P; q.SW = Q; q.dil = str; q.sig = 1;
  } else {
    q.OH = H; q.OW = W; q.SH = H; q.SW = W; q.dil = 1; q.sig = 1;
  }
  q.ncells = K * (mode == 1 ? 4 : 1);
  q.ncap = (q.ncells + 8 + 1) & ~1;
  q.KB = q.ncells <= 32 ? 32 : (q.ncells <= 64 ? 64 : 128);
  q.nck = cdiv(q.ncells, q.KB);
  const bool reduce = op == kWgrad || op == kBwd;
  // vector accesses of 4, 2 or 1 elements: a staged chunk stays within one
  // row; output-shaped planes are copied as flat runs
  auto vec_of = [&](long long e) {
    for (int v = aligned ? 4 : 1; v > 1; v /= 2)
      if (e % v == 0) return v;
    return 1;
  };
  q.vt = vec_of(q.SW);
  q.va = vec_of((long long)q.OH * q.OW);
  double best_score = 0.0;
  for (int NI = 64; NI >= 8; NI /= 2) {
    for (int RP : {4, 2}) {
      // the fused backward keeps 128 per-cell sums per lane only with two rows
      // (registers)
      if (op == kBwd && q.KB == 128 && RP == 4) continue;
      Params p = q;
      p.NI = NI;
      p.lni = 0;
      while ((1 << p.lni) < NI) ++p.lni;
      p.R = 128 / NI;
      p.RP = RP;
      p.mr = (RP - 1) * p.sig + mode;
      p.mc = (p.R - 1) * p.sig + mode;
      p.TRm = H + 2 * p.mr;
      p.TCm = W + p.mc;
      p.nrg = cdiv(p.OH, RP);
      p.ncg = cdiv(p.OW, p.R);
      p.nitems = p.nrg * p.ncg;
      const int oe = p.OH * p.OW;
      if (esize == 4) {
        p.OSz = oe | 1;
      } else {
        p.OSz = (oe + 1) & ~1;
        if ((p.OSz / 2) % 2 == 0) p.OSz += 2;
      }
      // LDS: nslot cell tables, the tile, the output-shaped tile, the weight
      // gradients' reduction area
      p.ival_off = (int)align16((size_t)p.ncap * 24 + (size_t)(2 * K + 1) * 4);  // cells (offset and weight,
      // row and column, tap, coefficient), first cell per tap, per-tap counts
      p.table_bytes = (int)align16((size_t)p.ival_off + (size_t)(p.nrg + p.ncg) * 8);  // then the runs
      const size_t tile = align16(((size_t)p.TRm * p.TCm + p.mc) * NI * 4);
      size_t rest = tile + align16((size_t)NI * p.OSz * esize);
      if (reduce) rest += align16((size_t)(kWaves * p.KB + K) * 4);
      p.nchunk = cdiv(N, NI);
      const long long nitem = (long long)C * p.nchunk;
      if (nitem > 0x7fffffffll) continue;
      // one work item per workgroup, one cell table
      p.per = 1;
      p.nslot = 1;
      const size_t off = (size_t)p.table_bytes + rest;
      if (off > kLdsBudget) continue;
      p.tile_off = p.nslot * p.table_bytes;
      p.aux_off = p.tile_off + (int)tile;
      p.red_off = p.aux_off + (int)align16((size_t)NI * p.OSz * esize);
      const long long blocks = (nitem + p.per - 1) / p.per;
      p.nblocks = (int)blocks;
      // idle lanes (images past N, rows and columns past the plane), one
      // table read per cell and RP tile reads, the cells a group's run adds
      // for its extent (R - 1 columns, RP - 1 rows), too few workgroups for
      // 256 CUs, a single workgroup per CU, and the idle share of the last
      // round of workgroups (resident per CU by LDS, granted in 1 KB steps,
      // at most four of eight waves)
      double score = (double)p.nchunk * NI / N * ((double)p.nrg * RP / p.OH) * ((double)p.ncg * p.R / p.OW) *
                     (1.0 + 0.5 / RP) * (1.0 + (double)(p.R - 1) / p.OW) * (1.0 + (double)(RP - 1) / p.OH);
      if (blocks < 640) score *= 640.0 / (double)blocks;
      if (kMaxLdsBytes / off < 2) score *= 1.5;
      {
        const size_t granted = (off + 1023) / 1024 * 1024;
        long long resident = (long long)((kMaxLdsBytes - 512) / granted);
        if (resident > 4) resident = 4;
        if (resident < 1) resident = 1;
        const long long slots = 256 * resident, rounds = (blocks + slots - 1) / slots;
        score *= (double)(rounds * slots) / (double)blocks;
      }
      if (!best.ok || score < best_score - 1e-9) {
        best_score = score;
        best.p = p;
        best.lds_bytes = off;
        best.parts = (size_t)p.nchunk;
        best.ok = true;
      }
    }
  }
  return best;
}

}  // namespace plane

// One translation unit per storage type; see o1d_plane_kernels.h.
#define O1D_PLANE_DECL(T)                                                                                        \
  hipError_t launch_plane_gather_##T(const plane::Plan& pl, const void* in, const void* w, const float* theta, \
                                     void* out, hipStream_t stream);                                           \
  hipError_t launch_plane_wgrad_##T(const plane::Plan& pl, const void* x, const void* dy, const float* theta,  \
                                    void* dw, float* partial, hipStream_t stream);                            \
  hipError_t launch_plane_bwd_##T(const plane::Plan& pl, const void* x, const void* dy, const void* w,         \
                                  const float* theta, void* dx, void* dw, float* partial, hipStream_t stream);
O1D_PLANE_DECL(f32)
O1D_PLANE_DECL(bf16)
#undef O1D_PLANE_DECL

inline hipError_t launch_plane_gather(Dtype dt, const plane::Plan& pl, const void* in, const void* w,
                                      const float* theta, void* out, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_plane_gather_f32(pl, in, w, theta, out, stream)
                          : launch_plane_gather_bf16(pl, in, w, theta, out, stream);
}

inline hipError_t launch_plane_wgrad(Dtype dt, const plane::Plan& pl, const void* x, const void* dy,
                                     const float* theta, void* dw, float* partial, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_plane_wgrad_f32(pl, x, dy, theta, dw, partial, stream)
                          : launch_plane_wgrad_bf16(pl, x, dy, theta, dw, partial, stream);
}

inline hipError_t launch_plane_bwd(Dtype dt, const plane::Plan& pl, const void* x, const void* dy, const void* w,
                                   const float* theta, void* dx, void* dw, float* partial, hipStream_t stream) {
  return dt == Dtype::F32 ? launch_plane_bwd_f32(pl, x, dy, w, theta, dx, dw, partial, stream)
                          : launch_plane_bwd_bf16(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace o1d
