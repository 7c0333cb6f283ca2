// Host-side plan of the run-decomposed kernels (o1d_runs.hip).  The plan
// depends only on (N, C, H, W, K): the angles live on the device and each
// workgroup derives its channel's program itself, so the plan must hold for
// every staging frame (plane or transposed plane) and strip direction.
#pragma once

#include <stddef.h>
#include <stdlib.h>

#include "o1d_launch.h"
#include "o1d_plan.h"

namespace o1d {
namespace runs {

constexpr int kR = 7;           // outputs per strip (a lane's register block)
constexpr int kLmax = 7;        // cells per run piece
constexpr int kMaxTaps = 64;    // K <= 63: one tap per lane of wave 0
constexpr int kMaxRuns = 64;
constexpr int kThreads2 = 512;  // 8 waves per workgroup
constexpr int kMaxStage = 8;    // staged elements per thread per plane group
constexpr int kProgBytes = 4 * (16 + 4 * 64) + 4 * 64 * 8;  // matches sizeof(Prog) in o1d_runs.hip

// Row strides compiled into the kernels.  A wave-tile is RB bands x CB
// columns of strips (RB * CB = 64 lanes); its lanes hit distinct LDS banks
// when 7 * S = CB * (odd) mod 64, so each S serves the layouts it satisfies.
constexpr int kStrides[] = {32, 48, 72, 80, 88, 104, 112, 120, 136};

struct RunsParams {
  int N, C, H, W, K, sign;
  int G;    // planes resident in LDS at once
  int NPW;  // planes per workgroup
  int RB, CB;
  int RT;   // tile row holding image row 0
  int TR;   // tile rows per plane
  int PS;   // plane stride in the tile area (dwords)
  int gather_lds_floats;
};

struct RunsPlan {
  RunsParams p;
  int S = 0;
  int threads = kThreads2;
  int blocks_n = 0;  // workgroups along the batch
  size_t lds_bytes = 0;
  bool ok = false;
};

inline bool bank_ok(int S, int CB) {
  if (CB >= 64) return true;
  const int v = (7 * S) & 63;
  return v % CB == 0 && ((v / CB) & 1) == 1;
}

// kind: 0 = gather (forward / input gradient), 1 = weight gradient.
inline RunsPlan plan_runs(int N, int C, int H, int W, int K, int sign, int kind) {
  RunsPlan pl;
  if (K > kMaxTaps - 1 || N < 1 || C < 1 || H < 1 || W < 1) return pl;
  const int pad = K / 2;
  const int M = H > W ? H : W;  // either staging frame
  const int nb = (M + kR - 1) / kR;
  int RB = 1;
  while (RB * 2 <= nb && RB * 2 <= 8) RB *= 2;
  const int CB = 64 / RB;
  int S = 0;
  for (int s : kStrides)
    if (s >= M + pad && bank_ok(s, CB)) {
      S = s;
      break;
    }
  if (S == 0) return pl;
  RunsParams& p = pl.p;
  p.N = N; p.C = C; p.H = H; p.W = W; p.K = K; p.sign = sign;
  p.RB = RB; p.CB = CB;
  p.RT = pad + 1;
  p.TR = p.RT + M + pad + kR + 1;
  p.PS = ((p.TR * S) + 3) & ~3;
  const long long HW = (long long)H * W;
  // planes per group: bounded by the per-thread staging registers and LDS
  int G = (int)((long long)kMaxStage * kThreads2 / HW);
  if (G < 1) return pl;
  if (G > 16) G = 16;
  const size_t budget = 56 * 1024;
  auto lds_for = [&](int g) -> size_t {
    size_t f = (size_t)kProgBytes / 4 + (size_t)g * p.PS;
    if (kind == 1) f += 8 * 64 + (((size_t)g * HW + 3) & ~(size_t)3);
    return f * 4;
  };
  while (G > 1 && lds_for(G) > budget) --G;
  if (lds_for(G) > kMaxLdsBytes) return pl;
  if ((long long)G * C * HW >= (1ll << 31)) return pl;
  p.G = G;
  // planes per workgroup: about two rounds of four resident workgroups per CU
  long long planes = (long long)N * C;
  int npw = (int)((planes + 2047) / 2048);
  if (const char* e = getenv("O1D_TUNE_NPW")) npw = atoi(e);
  if (npw < 1) npw = 1;
  npw = ((npw + G - 1) / G) * G;
  if (npw > ((N + G - 1) / G) * G) npw = ((N + G - 1) / G) * G;
  p.NPW = npw;
  pl.S = S;
  pl.blocks_n = (N + npw - 1) / npw;
  pl.lds_bytes = lds_for(G);
  pl.ok = true;
  return pl;
}

}  // namespace runs

hipError_t launch_gather_runs(Dtype dt, const runs::RunsPlan& pl, const void* in, const void* w, const float* theta,
                              void* out, hipStream_t stream);
hipError_t launch_wgrad_runs(Dtype dt, const runs::RunsPlan& pl, const void* x, const void* dy, const float* theta,
                             void* dw, float* partial, hipStream_t stream);

}  // namespace o1d
