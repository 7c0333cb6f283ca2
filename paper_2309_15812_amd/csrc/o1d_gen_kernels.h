// Device code of the general ("gen") kernels (included by o1d_gen_f32.hip
// and o1d_gen_bf16.hip); the host plan is in o1d_gen.h.
//
// The operation (Definition 1, Eq. 1-2): y[p,q] = sum_k w_k x(str p + rh_k,
// str q + rw_k), (rh_k, rw_k) the rotation of (0, k - pad) by theta.  The
// sample x(.) is either the pixel at the rounded-down offsets (Eq. 2) or the
// bilinear interpolation of the four pixels around the unrounded offsets
// (the alternative of the section "Discretization and Interpolation").  Both
// are a list of cells per channel, a cell being an integer offset (a, b) and
// a coefficient (1 when rounding down, the bilinear weight of a corner
// otherwise): y[p,q] = sum over cells of w_k coef x[str p + a, str q + b].
//
// Every workgroup builds the cell tables of its channels in LDS, stages the
// source plane's band with a zero margin (the paper's staging of the input
// in on-chip memory, cut into bands for large planes), and walks the cells:
// per lane RP outputs down one column, one LDS read and one FMA per output
// and cell.  The input gradient stages dy spread onto the stride lattice
// (zeros between), where it is the same gather with mirrored cells.  The
// weight gradient keeps one running sum per cell and lane (the product of dy
// with the tile under the cell) and folds the cells into taps at the end
// (coefficient times cell sum).  The fused backward walks dy with mirrored
// cells once: every value read feeds the lane's input-gradient outputs
// (times the cell's weight) and the cell's weight-gradient sum (times the
// lane's x).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_gen.h"
#include "o1d_wave.h"

namespace o1d {
namespace gen {
namespace {

using wave::static_for;

// Per-channel cell table in LDS (ncap cells per channel):
//   cw[2 j], cw[2 j + 1]: tile offset a TC + b (mirrored for the input
//   gradient) and the gather weight w_k coef (as bits);
//   tap[j], coef[j]: the cell's tap and coefficient (weight gradients);
//   cnt[ch]: number of cells.
struct Cells {
  int* cw;
  int* tap;
  float* coef;
  int* cnt;
  int ncap;
  __device__ __forceinline__ Cells(float* smem, const Params& P) {
    ncap = P.ncap;
    cw = reinterpret_cast<int*>(smem + P.cell_off);
    tap = cw + 2 * ncap * P.CB;
    coef = reinterpret_cast<float*>(tap + ncap * P.CB);
    cnt = reinterpret_cast<int*>(coef + ncap * P.CB);
  }
};

// One tap's cells: corner s at (h0 + (s >> 1), w0 + (s & 1)) with
// coefficient cf[s] (rounding down: corner 0 only, coefficient 1); n of the
// four coefficients are non-zero.  fin is false for a non-finite angle.
struct TapCells {
  double cf[4];
  int h0, w0, n;
  bool fin;
  __device__ __forceinline__ TapCells(const Params& P, float theta, int k) {
    double rh, rw;
    fin = tap_real(theta, P.K, k, &rh, &rw);
    h0 = floor_snapped(rh);
    w0 = floor_snapped(rw);
    cf[0] = cf[1] = cf[2] = cf[3] = 0.0;
    if (P.mode == 0 || !fin) {
      cf[0] = 1.0;
    } else {
      const double fh = frac_snapped(rh, h0), fw = frac_snapped(rw, w0);
#pragma unroll
      for (int s = 0; s < 4; ++s) cf[s] = ((s >> 1) ? fh : 1.0 - fh) * ((s & 1) ? fw : 1.0 - fw);
    }
    n = 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) n += cf[s] != 0.0 ? 1 : 0;
  }
};

// Builds the cell tables of channels c0 .. c0 + CB - 1: the workgroup's
// threads take the CB K (channel, tap) pairs in turn; each computes the tap's
// one (rounded down) or up to four (bilinear, corners with a zero coefficient
// dropped) cells, once to count them into `scratch` (CB K ints, for the
// prefix sum) and again to write them.  A non-finite angle gives the channel
// NaN weights and coefficients.
template <typename T>
__device__ void build_cells(const Params& P, const Cells& cl, const T* __restrict__ wgt,
                            const float* __restrict__ theta, int c0, int* scratch) {
  const int K = P.K, CB = P.CB;
  for (int t = threadIdx.x; t < CB; t += kThreads) cl.cnt[t] = 0;  // channels past C keep no cells
  // every slot starts as a dummy cell: offset 0 (the output's own centre,
  // which tap K/2 reads anyway), weight and coefficient 0, so that groups of
  // eight cells can run past the last real one
  for (int j = threadIdx.x; j < CB * cl.ncap; j += kThreads) {
    cl.cw[2 * j] = 0;
    cl.cw[2 * j + 1] = 0;
    cl.tap[j] = 0;
    cl.coef[j] = 0.f;
  }
  for (int t = threadIdx.x; t < CB * K; t += kThreads)
    if (c0 + t / K < P.C) scratch[t] = TapCells(P, theta[c0 + t / K], t % K).n;
  __syncthreads();
  for (int t = threadIdx.x; t < CB * K; t += kThreads) {
    const int ch = t / K, k = t - ch * K, c = c0 + ch;
    if (c >= P.C) continue;
    const TapCells tc(P, theta[c], k);
    int base = k;  // rounding down: one cell per tap
    if (P.mode != 0) {
      base = 0;
      for (int i = ch * K; i < t; ++i) base += scratch[i];
    }
    const float wk = wgt ? to_f32(wgt[(size_t)c * K + k]) : 0.f;
    // a non-finite angle (every tap of the channel sees it) poisons every
    // output of the channel
    int j = ch * cl.ncap + base;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (tc.cf[s] != 0.0) {
        const int off = P.sign * ((tc.h0 + (s >> 1)) * P.TC + tc.w0 + (s & 1));
        const float wc = tc.fin ? (float)((double)wk * tc.cf[s]) : __builtin_nanf("");
        cl.cw[2 * j] = off;
        cl.cw[2 * j + 1] = __float_as_int(wc);
        cl.tap[j] = k;
        cl.coef[j] = tc.fin ? (float)tc.cf[s] : __builtin_nanf("");
        ++j;
      }
    }
    if (k == K - 1) cl.cnt[ch] = base + tc.n;
  }
  __syncthreads();
}

// Geometry of one workgroup: channel block, output band, image run.  The
// blocks of one XCD (blockIdx mod 8) take consecutive logical blocks, so the
// channel blocks of one band and image run (NHWC: neighbouring channels of
// the same pixels) share that XCD's L2.
struct Work {
  int c0, p0, q0, n_begin, n_end, part;
  int r0, t0;  // tile origin in the staged plane's lattice coordinates
};

__device__ __forceinline__ Work work_of(const Params& P) {
  Work wk;
  const int b = blockIdx.x;
  const int logical = P.xcd_per ? (b % kXcds) * P.xcd_per + b / kXcds : b;
  const int cb = logical % P.ncb;
  const int rest = logical / P.ncb;
  const int band = rest % (P.nbp * P.nbq);
  const int run = rest / (P.nbp * P.nbq);
  const int bp = band / P.nbq, bq = band - bp * P.nbq;
  wk.part = rest;  // partial row of the weight gradient: (image run, band)
  wk.c0 = cb * P.CB;
  wk.p0 = bp * P.BP;
  wk.q0 = bq * P.BQ;
  wk.n_begin = run * P.npw;
  wk.n_end = min(P.N, wk.n_begin + P.npw);
  // tile row r holds lattice row r0 + r: forward and weight gradient
  // str p0 - hp (x rows); input gradient p0 - hp (dilated dy rows)
  wk.r0 = wk.p0 * P.sig - P.hp;
  wk.t0 = wk.q0 * P.sig - P.hp;
  return wk;
}

__device__ __forceinline__ int floor_div(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// q = a / b for 0 <= a < 2^24, 0 < b, from a float reciprocal of b (one
// correction step makes it exact).
__device__ __forceinline__ int fdiv(int a, int b, float rb) {
  int q = (int)((float)a * rb);
  const int r = a - q * b;
  q += r < 0 ? -1 : (r >= b ? 1 : 0);
  return q;
}

// Copies a rectangle of ni x nj elements (x 2^lcb channels for NHWC) of each
// of ng images between global memory and LDS: for every element (g, i, j,
// ch), with j (NCHW) or ch (NHWC) fastest so that neighbouring lanes touch
// neighbouring addresses, op.load(g, i, j, ch) gives the value and
// op.store(g, i, j, ch, v) puts it.  A lane keeps one position x in the
// row (rows shorter than the workgroup: rpp rows per pass; longer rows:
// chunks of kThreads) and steps through its rows with an incremental (g, i),
// so the index arithmetic is per lane, not per element.  Eight rows per lane
// are loaded before any is stored, so that their memory latencies overlap.
template <int L, class Op>
__device__ __forceinline__ void copy_rect(int ng, int ni, int nj, int lcb, Op&& op) {
  const int inner = nj << (L == kNHWC ? lcb : 0);
  const int rows = ng * ni;
  if (rows <= 0 || inner <= 0) return;
  const int t = threadIdx.x;
  const bool wide = inner >= kThreads;
  const int rpp = wide ? 1 : kThreads / inner;  // rows per pass
  const int ro = wide ? 0 : t / inner;           // the lane's first row
  if (ro >= rpp) return;                         // lanes past rpp rows of a pass
  const int rdiv = rpp / ni, rmod = rpp - rdiv * ni;
  const int g0 = ro / ni, i0 = ro - g0 * ni;
  for (int x = wide ? t : t - ro * inner; x < inner; x += kThreads) {
    const int j = L == kNHWC ? x >> lcb : x;
    const int ch = L == kNHWC ? x & ((1 << lcb) - 1) : 0;
    int g = g0, i = i0;
    for (int row = ro; row < rows;) {
      float v[8];
      int gg[8], ii[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        gg[m] = -1;
        if (row < rows) {
          gg[m] = g;
          ii[m] = i;
          v[m] = op.load(g, i, j, ch);
        }
        row += rpp;
        g += rdiv;
        i += rmod;
        if (i >= ni) {
          i -= ni;
          ++g;
        }
      }
#pragma unroll
      for (int m = 0; m < 8; ++m)
        if (gg[m] >= 0) op.store(gg[m], ii[m], j, ch, v[m]);
    }
  }
}

// Stages images n0 .. n0 + ng - 1 of the source plane (SH x SW) for the
// channel block into the tiles: element (i, j) goes to tile position
// (i dil - r0, j dil - t0).  Only in-plane lattice points are written; the
// rest of every tile stays zero from the workgroup's start.
template <typename T, int L>
struct StageOp {
  const Params& P;
  const T* __restrict__ src;
  float* tiles;
  int n0, ilo, jlo, rbase, cbase;
  __device__ __forceinline__ float load(int g, int ii, int jj, int ch) const {
    const int c = min(P.C - 1, c0 + ch);  // channels past C: a valid address, never used
    const int n = n0 + g, i = ilo + ii, j = jlo + jj;
    const size_t idx = L == kNHWC ? (((size_t)n * P.SH + i) * P.SW + j) * P.C + c
                                  : ((size_t)n * P.C + c) * ((size_t)P.SH * P.SW) + (size_t)i * P.SW + j;
    return to_f32(src[idx]);
  }
  __device__ __forceinline__ void store(int g, int ii, int jj, int ch, float v) const {
    tiles[(g * P.CB + ch) * P.TW + (rbase + ii * P.dil) * P.TC + cbase + jj * P.dil] = v;
  }
  int c0;
};

template <typename T, int L>
__device__ __forceinline__ void stage(const Params& P, const Work& wk, const T* __restrict__ src, float* tiles,
                                      int n0, int ng) {
  const int dil = P.dil;
  const int ilo = max(0, floor_div(wk.r0 + dil - 1, dil)), ihi = min(P.SH - 1, floor_div(wk.r0 + P.TR - 1, dil));
  const int jlo = max(0, floor_div(wk.t0 + dil - 1, dil)), jhi = min(P.SW - 1, floor_div(wk.t0 + P.TC - 1, dil));
  if (ihi < ilo || jhi < jlo) return;
  StageOp<T, L> op{P, src, tiles, n0, ilo, jlo, ilo * dil - wk.r0, jlo * dil - wk.t0, wk.c0};
  copy_rect<L>(ng, ihi - ilo + 1, jhi - jlo + 1, P.lcb, op);
}

// Stages the band [p0, p0 + nrow) x [q0, q0 + ncol) of an output-shaped
// tensor (dy, or x for the fused backward) into band tiles (row stride BQ);
// positions past the plane keep the zeros they were initialised with.
template <typename T, int L>
struct BandLoadOp {
  const Params& P;
  const T* __restrict__ src;
  float* band;
  int n0, p0, q0, c0;
  __device__ __forceinline__ float load(int g, int ii, int jj, int ch) const {
    const int c = min(P.C - 1, c0 + ch);
    const int n = n0 + g, p = p0 + ii, q = q0 + jj;
    const size_t idx = L == kNHWC ? (((size_t)n * P.OH + p) * P.OW + q) * P.C + c
                                  : ((size_t)n * P.C + c) * ((size_t)P.OH * P.OW) + (size_t)p * P.OW + q;
    return to_f32(src[idx]);
  }
  __device__ __forceinline__ void store(int g, int ii, int jj, int ch, float v) const {
    band[(g * P.CB + ch) * P.OS + ii * P.BQ + jj] = v;
  }
};

template <typename T, int L>
__device__ __forceinline__ void stage_band(const Params& P, const Work& wk, const T* __restrict__ src, float* band,
                                           int n0, int ng) {
  const int nrow = min(P.BP, P.OH - wk.p0), ncol = min(P.BQ, P.OW - wk.q0);
  BandLoadOp<T, L> op{P, src, band, n0, wk.p0, wk.q0, wk.c0};
  copy_rect<L>(ng, nrow, ncol, P.lcb, op);
}

// Writes a band tile (output layout) to global memory; channels past C are
// skipped.
template <typename T, int L>
struct BandStoreOp {
  const Params& P;
  T* __restrict__ dst;
  const float* band;
  int n0, p0, q0, c0;
  __device__ __forceinline__ float load(int g, int ii, int jj, int ch) const {
    return band[(g * P.CB + ch) * P.OS + ii * P.BQ + jj];
  }
  __device__ __forceinline__ void store(int g, int ii, int jj, int ch, float v) const {
    const int c = c0 + ch;
    if (c < P.C) {
      const int n = n0 + g, p = p0 + ii, q = q0 + jj;
      const size_t idx = L == kNHWC ? (((size_t)n * P.OH + p) * P.OW + q) * P.C + c
                                    : ((size_t)n * P.C + c) * ((size_t)P.OH * P.OW) + (size_t)p * P.OW + q;
      dst[idx] = from_f32<T>(v);
    }
  }
};

template <typename T, int L>
__device__ __forceinline__ void store_band(const Params& P, const Work& wk, T* __restrict__ dst, const float* band,
                                           int n0, int ng) {
  const int nrow = min(P.BP, P.OH - wk.p0), ncol = min(P.BQ, P.OW - wk.q0);
  BandStoreOp<T, L> op{P, dst, band, n0, wk.p0, wk.q0, wk.c0};
  copy_rect<L>(ng, nrow, ncol, P.lcb, op);
}

// A lane's task: channel ch of the block, image g of the pass, row group rg
// of the band, column qq of the band.
struct Task {
  int ch, g, rg, qq;
};

__device__ __forceinline__ Task task_of(const Params& P, int tau) {
  Task t;
  t.qq = tau % P.BQ;
  int r = tau / P.BQ;
  t.rg = r % P.NRG;
  r /= P.NRG;
  t.ch = r & (P.CB - 1);
  t.g = r >> P.lcb;
  return t;
}

__device__ __forceinline__ const float* tile_of(const Params& P, const float* tiles, const Task& t) {
  return tiles + (t.g * P.CB + t.ch) * P.TW + (t.rg * P.RP * P.sig + P.hp) * P.TC + t.qq * P.sig + P.hp;
}

// ---------------------------------------------------------------- gather

// out[p,q] = sum over the channel's cells of weight * tile[base(p,q) + off]:
// the forward pass (cells at +(a, b), output step str) and the input
// gradient (dy on the lattice, cells at -(a, b), output step 1).
template <typename T, int L, int RP>
__global__ __launch_bounds__(kThreads) void gen_gather(Params P, const T* __restrict__ in, const T* __restrict__ wgt,
                                                       const float* __restrict__ theta, T* __restrict__ out) {
  extern __shared__ float smem[];
  const Work wk = work_of(P);
  const Cells cl(smem, P);
  float* tiles = smem + P.tile_off;
  float* band = smem + P.band_off;  // NHWC: the output band
  build_cells<T>(P, cl, wgt, theta, wk.c0, reinterpret_cast<int*>(tiles));
  for (int i = threadIdx.x; i < P.G * P.CB * P.TW; i += kThreads) tiles[i] = 0.f;
  __syncthreads();
  const int rstep = P.sig * P.TC;
  const int per_ch = P.NRG * P.BQ;  // tasks per image and channel
  for (int n0 = wk.n_begin; n0 < wk.n_end; n0 += P.G) {
    const int ng = min(P.G, wk.n_end - n0);
    stage<T, L>(P, wk, in, tiles, n0, ng);
    __syncthreads();
    // NCHW (one channel per block): its cell count and table are uniform.
    // NHWC: the block's CB channels share one pass (a channel alone would
    // leave most lanes idle on a narrow band); every lane reads its own
    // channel's table, and the walk runs to the block's largest cell count
    // (tables are zero past their cells: offset 0, weight 0).
    const int npass = L == kNHWC ? 1 : P.CB;
    for (int ch = 0; ch < npass; ++ch) {
      int nc = 0;
      if (L == kNHWC) {
        for (int c = 0; c < P.CB; ++c) nc = max(nc, __builtin_amdgcn_readfirstlane(cl.cnt[c]));
      } else {
        nc = __builtin_amdgcn_readfirstlane(cl.cnt[ch]);
      }
      const int ntask = ng * per_ch * (L == kNHWC ? P.CB : 1);
      for (int tau = threadIdx.x; tau < ntask; tau += kThreads) {
        Task t;
        t.qq = tau % P.BQ;
        int r = tau / P.BQ;
        t.rg = r % P.NRG;
        r /= P.NRG;
        if (L == kNHWC) {
          t.ch = r & (P.CB - 1);
          t.g = r >> P.lcb;
        } else {
          t.ch = ch;
          t.g = r;
        }
        const int4* cw2 = reinterpret_cast<const int4*>(cl.cw + 2 * t.ch * cl.ncap);
        const float* tl = tile_of(P, tiles, t);
        float acc[RP];
#pragma unroll
        for (int i = 0; i < RP; ++i) acc[i] = 0.f;
        // eight cells per step (the table is padded with dummy cells to a
        // multiple of eight); the next step's table entries are read before
        // this step's tile reads, so the table read's latency is hidden
        const int n8 = (nc + 7) & ~7;
        int4 cur[4], nxt[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = cw2[u];
        for (int j = 0; j < n8; j += 8) {
          if (j + 8 < n8) {
#pragma unroll
            for (int u = 0; u < 4; ++u) nxt[u] = cw2[((j + 8) >> 1) + u];
          }
          float v[8][RP];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float* a0 = tl + cur[u].x;
            const float* a1 = tl + cur[u].z;
#pragma unroll
            for (int i = 0; i < RP; ++i) {
              v[2 * u][i] = a0[i * rstep];
              v[2 * u + 1][i] = a1[i * rstep];
            }
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int i = 0; i < RP; ++i) acc[i] = fmaf(__int_as_float(cur[u].y), v[2 * u][i], acc[i]);
#pragma unroll
            for (int i = 0; i < RP; ++i) acc[i] = fmaf(__int_as_float(cur[u].w), v[2 * u + 1][i], acc[i]);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) cur[u] = nxt[u];
        }
        if (L == kNCHW) {
          const int q = wk.q0 + t.qq;
          if (q < P.OW) {
            T* o = out + ((size_t)(n0 + t.g) * P.C + wk.c0) * P.OH * P.OW + q;
#pragma unroll
            for (int i = 0; i < RP; ++i) {
              const int p = wk.p0 + t.rg * RP + i;
              if (p < P.OH) o[(size_t)p * P.OW] = from_f32<T>(acc[i]);
            }
          }
        } else {
          float* b = band + (t.g * P.CB + t.ch) * P.OS + t.rg * RP * P.BQ + t.qq;
#pragma unroll
          for (int i = 0; i < RP; ++i) b[i * P.BQ] = acc[i];
        }
      }
    }
    __syncthreads();  // the tiles are free (NHWC: the outputs are in the band tile)
    if (L == kNHWC) {
      store_band<T, L>(P, wk, out, band, n0, ng);
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- weight gradients

// Adds the workgroup's sums of cells j0 .. j0 + KB - 1 of channel ch, times
// the cells' coefficients, to the per-tap sums dwacc[ch * K + tap] in a fixed
// order.  Every lane holds sums of channel ch (zero where it had no task).
// acc is consumed.
template <int KB>
__device__ __forceinline__ void fold_cells(const Params& P, const Cells& cl, float (&acc)[KB], int ch, int j0,
                                           float* red, float* dwacc) {
  wave::sums<KB>(acc, red);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int nc = cl.cnt[ch];
    for (int j = 0; j < KB && j0 + j < nc; ++j) {
      float v = 0.f;
      for (int w = 0; w < kThreads / 64; ++w) v += red[w * KB + j];
      const int cj = ch * cl.ncap + j0 + j;
      dwacc[ch * P.K + cl.tap[cj]] += cl.coef[cj] * v;
    }
  }
  __syncthreads();
}

// fold_cells for cpp channels c0 .. c0 + cpp - 1 at once, channel c0 + i
// held by waves i wpc .. i wpc + wpc - 1: each channel's wave sums are
// added in a fixed order by its own thread.
template <int KB>
__device__ __forceinline__ void fold_group(const Params& P, const Cells& cl, float (&acc)[KB], int c0, int cpp,
                                           int wpc, int j0, float* red, float* dwacc) {
  wave::sums<KB>(acc, red);
  __syncthreads();
  if ((int)threadIdx.x < cpp) {
    const int ch = c0 + threadIdx.x;
    const int nc = cl.cnt[ch];
    for (int j = 0; j < KB && j0 + j < nc; ++j) {
      float v = 0.f;
      for (int w = threadIdx.x * wpc; w < (int)(threadIdx.x + 1) * wpc; ++w) v += red[w * KB + j];
      const int cj = ch * cl.ncap + j0 + j;
      dwacc[ch * P.K + cl.tap[cj]] += cl.coef[cj] * v;
    }
  }
  __syncthreads();
}

// acc[j] += sum_i d[i] tile[base + off_j + i rstep] for the cells of the
// group of KB: eight cells per step (one branch per step, the 8 RP reads
// issued together), steps past nc skipped (nc uniform; cells between the
// last real one and the step's end are dummies with offset 0).
template <int RP, int KB>
__device__ __forceinline__ void cell_dots(const int2* cw, int nc, const float* tl, int rstep, const float (&d)[RP],
                                          float (&acc)[KB]) {
  static_for<KB / 8>([&](auto gc) __attribute__((always_inline)) {
    constexpr int j0 = 8 * decltype(gc)::value;
    if (j0 < nc) {
      const int4* c4 = reinterpret_cast<const int4*>(cw + j0);
      int4 c[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) c[u] = c4[u];
      float v[8][RP];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* a0 = tl + c[u].x;
        const float* a1 = tl + c[u].z;
#pragma unroll
        for (int i = 0; i < RP; ++i) {
          v[2 * u][i] = a0[i * rstep];
          v[2 * u + 1][i] = a1[i * rstep];
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < RP; ++i) sum = fmaf(d[i], v[u][i], sum);
        acc[j0 + u] += sum;
      }
    }
  });
}

// partial[(part * C + c) * K + k] = the workgroup's sum over its band and
// images of dy[p,q] * sum_cells coef x[str p + a, str q + b] for the cells of
// tap k (Eq. 1 differentiated in w_k).  NCHW: each lane's KB cell sums run
// over all its tasks and images and are folded once per group of KB cells
// (more than KB cells: bilinear with K > 31, the images staged again per
// group); NHWC (several channels per workgroup): folded per pass and channel.
template <typename T, int L, int RP, int KB>
__global__ __launch_bounds__(kThreads) void gen_wgrad(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                      const float* __restrict__ theta, float* __restrict__ partial) {
  extern __shared__ float smem[];
  const Work wk = work_of(P);
  const Cells cl(smem, P);
  float* tiles = smem + P.tile_off;
  float* band = smem + P.band_off;
  float* red = smem + P.red_off;
  float* dwacc = red + (kThreads / 64) * KB;
  build_cells<T>(P, cl, static_cast<const T*>(nullptr), theta, wk.c0, reinterpret_cast<int*>(tiles));
  for (int i = threadIdx.x; i < P.G * P.CB * P.TW; i += kThreads) tiles[i] = 0.f;
  for (int i = threadIdx.x; i < P.G * P.CB * P.OS; i += kThreads) band[i] = 0.f;
  for (int i = threadIdx.x; i < P.CB * P.K; i += kThreads) dwacc[i] = 0.f;
  __syncthreads();
  const int rstep = P.sig * P.TC;
  const int per_ch = P.NRG * P.BQ;  // tasks per image and channel
  // A lane keeps one channel: a pass covers cpp channels with wpc whole
  // waves each (NCHW: one channel, all waves), so that every wave's cell
  // count is uniform and its per-cell sums belong to one channel.
  constexpr int nw = kThreads / 64;
  const int cpp = L == kNCHW ? 1 : min(P.CB, nw), wpc = nw / cpp, npass = L == kNCHW ? 1 : P.CB / cpp;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the lane's first task in its channel and its task step
  const int lt = L == kNCHW ? (int)threadIdx.x : (wave % wpc) * 64 + (threadIdx.x & 63);
  const int lstep = L == kNCHW ? kThreads : wpc * 64;
  for (int j0 = 0; j0 < P.nck * KB; j0 += KB) {
    float acc[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) acc[j] = 0.f;
    for (int n0 = wk.n_begin; n0 < wk.n_end; n0 += P.G) {
      const int ng = min(P.G, wk.n_end - n0);
      stage<T, L>(P, wk, x, tiles, n0, ng);
      stage_band<T, L>(P, wk, dy, band, n0, ng);
      __syncthreads();
      for (int ps = 0; ps < npass; ++ps) {
        const int ch = L == kNCHW ? 0 : ps * cpp + wave / wpc;                   // uniform per wave
        const int nc = min(KB, __builtin_amdgcn_readfirstlane(cl.cnt[ch]) - j0);  // uniform per wave
        if (nc > 0) {
          const int2* cw = reinterpret_cast<const int2*>(cl.cw) + ch * cl.ncap + j0;
          for (int tau = lt; tau < ng * per_ch; tau += lstep) {
            Task t;
            t.qq = tau % P.BQ;
            const int r = tau / P.BQ;
            t.rg = r % P.NRG;
            t.g = r / P.NRG;
            t.ch = ch;
            const float* b = band + (t.g * P.CB + ch) * P.OS + t.rg * RP * P.BQ + t.qq;
            float d[RP];
#pragma unroll
            for (int i = 0; i < RP; ++i) d[i] = b[i * P.BQ];  // zero past the plane
            cell_dots<RP, KB>(cw, nc, tile_of(P, tiles, t), rstep, d, acc);
          }
        }
        if (npass > 1) {
          // the next pass takes other channels: fold these
          fold_group<KB>(P, cl, acc, ps * cpp, cpp, wpc, j0, red, dwacc);
#pragma unroll
          for (int j = 0; j < KB; ++j) acc[j] = 0.f;
        }
      }
      __syncthreads();  // the tiles are free
    }
    if (L == kNCHW) {
      if (j0 < __builtin_amdgcn_readfirstlane(cl.cnt[0])) fold_cells<KB>(P, cl, acc, 0, j0, red, dwacc);
    } else if (npass == 1) {
      fold_group<KB>(P, cl, acc, 0, cpp, wpc, j0, red, dwacc);
    }
  }
  for (int i = threadIdx.x; i < P.CB * P.K; i += kThreads) {
    const int ch = i / P.K, k = i - ch * P.K, c = wk.c0 + ch;
    if (c < P.C) partial[((size_t)wk.part * P.C + c) * P.K + k] = isfinite(theta[c]) ? dwacc[i] : __builtin_nanf("");
  }
}

// Both gradients in one pass (NCHW, stride 1, rounded-down offsets): the
// tile holds dy with its margin, a band tile x at the lane's outputs.  Per
// cell (mirrored offsets) every dy value v read for the lane's input-gradient
// outputs h adds w_c v to dx[h] and x[h] v to the cell's sum, which is the
// weight gradient of the cell's tap: dw_k = sum_h x[h] dy[h - off_k].
template <typename T, int RP, int KB>
__global__ __launch_bounds__(kThreads) void gen_bwd(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                    const T* __restrict__ wgt, const float* __restrict__ theta,
                                                    T* __restrict__ dx, float* __restrict__ partial) {
  extern __shared__ float smem[];
  const Work wk = work_of(P);
  const Cells cl(smem, P);
  float* tiles = smem + P.tile_off;
  float* xband = smem + P.band_off;
  float* oband = xband + P.G * P.OS;
  float* red = smem + P.red_off;
  float* dwacc = red + (kThreads / 64) * KB;
  build_cells<T>(P, cl, wgt, theta, wk.c0, reinterpret_cast<int*>(tiles));
  for (int i = threadIdx.x; i < P.G * P.TW; i += kThreads) tiles[i] = 0.f;
  for (int i = threadIdx.x; i < P.G * P.OS; i += kThreads) xband[i] = 0.f;
  for (int i = threadIdx.x; i < P.K; i += kThreads) dwacc[i] = 0.f;
  __syncthreads();
  const int rstep = P.TC;
  const int ntask = P.NRG * P.BQ;
  const int nc = min(KB, __builtin_amdgcn_readfirstlane(cl.cnt[0]));
  const int2* cw = reinterpret_cast<const int2*>(cl.cw);
  float acc[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) acc[j] = 0.f;
  for (int n0 = wk.n_begin; n0 < wk.n_end; n0 += P.G) {
    const int ng = min(P.G, wk.n_end - n0);
    stage<T, kNCHW>(P, wk, dy, tiles, n0, ng);
    stage_band<T, kNCHW>(P, wk, x, xband, n0, ng);
    __syncthreads();
    for (int tau = threadIdx.x; tau < ng * ntask; tau += kThreads) {
      Task t;
      t.qq = tau % P.BQ;
      const int r = tau / P.BQ;
      t.rg = r % P.NRG;
      t.g = r / P.NRG;
      t.ch = 0;
      const float* xb = xband + t.g * P.OS + t.rg * RP * P.BQ + t.qq;
      float xv[RP], o[RP];
#pragma unroll
      for (int i = 0; i < RP; ++i) {
        xv[i] = xb[i * P.BQ];
        o[i] = 0.f;
      }
      const float* tl = tile_of(P, tiles, t);
      static_for<KB / 8>([&](auto gc) __attribute__((always_inline)) {
        constexpr int j0 = 8 * decltype(gc)::value;
        if (j0 < nc) {
          const int4* c4 = reinterpret_cast<const int4*>(cw + j0);
          int4 c[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) c[u] = c4[u];
          float v[8][RP];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float* a0 = tl + c[u].x;
            const float* a1 = tl + c[u].z;
#pragma unroll
            for (int i = 0; i < RP; ++i) {
              v[2 * u][i] = a0[i * rstep];
              v[2 * u + 1][i] = a1[i * rstep];
            }
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const float wc = __int_as_float(u & 1 ? c[u >> 1].w : c[u >> 1].y);
            float sum = 0.f;
#pragma unroll
            for (int i = 0; i < RP; ++i) {
              o[i] = fmaf(wc, v[u][i], o[i]);
              sum = fmaf(xv[i], v[u][i], sum);
            }
            acc[j0 + u] += sum;
          }
        }
      });
      float* ob = oband + t.g * P.OS + t.rg * RP * P.BQ + t.qq;
#pragma unroll
      for (int i = 0; i < RP; ++i) ob[i * P.BQ] = o[i];
    }
    __syncthreads();  // the tiles are free; the input gradient is in its band tile
    store_band<T, kNCHW>(P, wk, dx, oband, n0, ng);
    __syncthreads();
  }
  if (nc > 0) fold_cells<KB>(P, cl, acc, 0, 0, red, dwacc);
  for (int k = threadIdx.x; k < P.K; k += kThreads)
    partial[((size_t)wk.part * P.C + wk.c0) * P.K + k] = isfinite(theta[wk.c0]) ? dwacc[k] : __builtin_nanf("");
}

// dw[i] = sum over the partial rows, in a fixed order.
template <typename T>
__global__ __launch_bounds__(256) void gen_wgrad_reduce(const float* __restrict__ partial, T* __restrict__ dw, int CK,
                                                        int parts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CK) return;
  float s = 0.f;
  for (int j = 0; j < parts; ++j) s += partial[(size_t)j * CK + i];
  dw[i] = from_f32<T>(s);
}

// ---------------------------------------------------------------- launch

template <const void* (*Fn)()>
hipError_t allow_lds() {
  static int done = 0;  // benign race: the attribute call is idempotent
  if (done) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(Fn(), hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLdsBytes);
  if (e == hipSuccess) done = 1;
  return e;
}
template <typename T, int L, int RP>
const void* gather_fn() { return reinterpret_cast<const void*>(gen_gather<T, L, RP>); }
template <typename T, int L, int RP, int KB>
const void* wgrad_fn() { return reinterpret_cast<const void*>(gen_wgrad<T, L, RP, KB>); }
template <typename T, int RP, int KB>
const void* bwd_fn() { return reinterpret_cast<const void*>(gen_bwd<T, RP, KB>); }

template <typename T>
hipError_t reduce_launch(const Plan& pl, const float* partial, void* dw, hipStream_t stream) {
  const int CK = pl.p.C * pl.p.K;
  hipLaunchKernelGGL(gen_wgrad_reduce<T>, dim3((unsigned)((CK + 255) / 256)), dim3(256), 0, stream, partial,
                     static_cast<T*>(dw), CK, (int)pl.parts);
  return hipGetLastError();
}

template <typename T, int L, int RP>
hipError_t gather_launch(const Plan& pl, const void* in, const void* w, const float* theta, void* out,
                         hipStream_t stream) {
  const hipError_t e = allow_lds<gather_fn<T, L, RP>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gen_gather<T, L, RP>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream,
                     pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta, static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int L, int RP, int KB>
hipError_t wgrad_launch(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                        hipStream_t stream) {
  hipError_t e = allow_lds<wgrad_fn<T, L, RP, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gen_wgrad<T, L, RP, KB>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream,
                     pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return reduce_launch<T>(pl, partial, dw, stream);
}

template <typename T, int RP, int KB>
hipError_t bwd_launch(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx,
                      void* dw, float* partial, hipStream_t stream) {
  hipError_t e = allow_lds<bwd_fn<T, RP, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gen_bwd<T, RP, KB>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream, pl.p,
                     static_cast<const T*>(x), static_cast<const T*>(dy), static_cast<const T*>(w), theta,
                     static_cast<T*>(dx), partial);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return reduce_launch<T>(pl, partial, dw, stream);
}

template <typename T>
hipError_t gather_t(const Plan& pl, int layout, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
  if (layout == kNHWC)
    return pl.p.RP == 4 ? gather_launch<T, kNHWC, 4>(pl, in, w, theta, out, stream)
                        : gather_launch<T, kNHWC, 8>(pl, in, w, theta, out, stream);
  return pl.p.RP == 4 ? gather_launch<T, kNCHW, 4>(pl, in, w, theta, out, stream)
                      : gather_launch<T, kNCHW, 8>(pl, in, w, theta, out, stream);
}

template <typename T, int L, int RP>
hipError_t wgrad_kb(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                    hipStream_t stream) {
  if (pl.p.KB == 32) return wgrad_launch<T, L, RP, 32>(pl, x, dy, theta, dw, partial, stream);
  if (pl.p.KB == 64) return wgrad_launch<T, L, RP, 64>(pl, x, dy, theta, dw, partial, stream);
  return wgrad_launch<T, L, RP, 128>(pl, x, dy, theta, dw, partial, stream);
}

// Eight outputs per lane only with 32 per-cell sums (the plan's rule).
template <typename T>
hipError_t wgrad_t(const Plan& pl, int layout, const void* x, const void* dy, const float* theta, void* dw,
                   float* partial, hipStream_t stream) {
  if (pl.p.RP == 8 && pl.p.KB != 32) return hipErrorInvalidValue;
  if (layout == kNHWC)
    return pl.p.RP == 4 ? wgrad_kb<T, kNHWC, 4>(pl, x, dy, theta, dw, partial, stream)
                        : wgrad_launch<T, kNHWC, 8, 32>(pl, x, dy, theta, dw, partial, stream);
  return pl.p.RP == 4 ? wgrad_kb<T, kNCHW, 4>(pl, x, dy, theta, dw, partial, stream)
                      : wgrad_launch<T, kNCHW, 8, 32>(pl, x, dy, theta, dw, partial, stream);
}

template <typename T, int RP>
hipError_t bwd_kb(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx, void* dw,
                  float* partial, hipStream_t stream) {
  if (pl.p.KB == 32) return bwd_launch<T, RP, 32>(pl, x, dy, w, theta, dx, dw, partial, stream);
  if (pl.p.KB == 64) return bwd_launch<T, RP, 64>(pl, x, dy, w, theta, dx, dw, partial, stream);
  return bwd_launch<T, RP, 128>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

template <typename T>
hipError_t bwd_t(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx, void* dw,
                 float* partial, hipStream_t stream) {
  if (pl.p.RP == 8 && pl.p.KB != 32) return hipErrorInvalidValue;
  return pl.p.RP == 4 ? bwd_kb<T, 4>(pl, x, dy, w, theta, dx, dw, partial, stream)
                      : bwd_launch<T, 8, 32>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace
}  // namespace gen
}  // namespace o1d
