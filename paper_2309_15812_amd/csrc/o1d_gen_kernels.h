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
// (zeros between), where it is the same gather with mirrored cells; the
// weight gradient accumulates per cell the products of dy with the tile and
// folds them into per-tap sums (coefficient times cell sum).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_gen.h"

namespace o1d {
namespace gen {
namespace {

template <typename T>
__device__ __forceinline__ void store_elem(T* p, float v) {
  *p = from_f32<T>(v);
}

// Per-channel cell table in LDS (ncap cells per channel):
//   cw[2 j], cw[2 j + 1]: tile offset a TC + b (mirrored for the input
//   gradient) and the gather weight w_k coef (as bits);
//   tap[j], coef[j]: the cell's tap and coefficient (weight gradient);
//   cnt[ch]: number of cells.
struct Cells {
  int* cw;
  int* tap;
  float* coef;
  int* cnt;
  int ncap;
  __device__ __forceinline__ Cells(float* smem, const Params& P) {
    ncap = P.K * (P.mode == 1 ? 4 : 1);
    cw = reinterpret_cast<int*>(smem);
    tap = cw + 2 * ncap * P.CB;
    coef = reinterpret_cast<float*>(tap + ncap * P.CB);
    cnt = reinterpret_cast<int*>(coef + ncap * P.CB);
  }
};

// Builds the cell tables of channels c0 .. c0 + CB - 1: one thread per (channel,
// tap) computes the tap's one (rounded down) or up to four (bilinear, corners
// with a zero coefficient dropped) cells; `scratch` (CB K ints) holds the
// per-tap cell counts for the prefix sum.  A non-finite angle gives the
// channel NaN weights and coefficients.
template <typename T>
__device__ void build_cells(const Params& P, const Cells& cl, const T* __restrict__ wgt,
                            const float* __restrict__ theta, int c0, int* scratch) {
  const int K = P.K, CB = P.CB;
  const int t = threadIdx.x;
  // corner s of the tap: (h0 + (s >> 1), w0 + (s & 1)) with coefficient cf[s]
  // (rounding down: corner 0 only, coefficient 1)
  double cf[4] = {0.0, 0.0, 0.0, 0.0};
  int h0 = 0, w0 = 0, n = 0;
  bool fin = true;
  const bool act = t < CB * K && c0 + t / K < P.C;
  if (t < CB) cl.cnt[t] = 0;  // channels past C keep no cells
  if (act) {
    const int ch = t / K, k = t - ch * K, c = c0 + ch;
    double rh, rw;
    fin = tap_real(theta[c], K, k, &rh, &rw);
    h0 = floor_snapped(rh);
    w0 = floor_snapped(rw);
    if (P.mode == 0 || !fin) {
      cf[0] = 1.0;
    } else {
      const double fh = frac_snapped(rh, h0), fw = frac_snapped(rw, w0);
#pragma unroll
      for (int s = 0; s < 4; ++s) cf[s] = ((s >> 1) ? fh : 1.0 - fh) * ((s & 1) ? fw : 1.0 - fw);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) n += cf[s] != 0.0 ? 1 : 0;
    scratch[t] = n;
  }
  __syncthreads();
  if (act) {
    const int ch = t / K, k = t - ch * K, c = c0 + ch;
    int base = 0;
    for (int i = ch * K; i < t; ++i) base += scratch[i];
    const float wk = wgt ? to_f32(wgt[(size_t)c * K + k]) : 0.f;
    // a non-finite angle (every tap of the channel sees it) poisons every
    // output of the channel
    int j = ch * cl.ncap + base;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (cf[s] != 0.0) {
        const int off = P.sign * ((h0 + (s >> 1)) * P.TC + w0 + (s & 1));
        const float wc = fin ? (float)((double)wk * cf[s]) : __builtin_nanf("");
        cl.cw[2 * j] = off;
        cl.cw[2 * j + 1] = __float_as_int(wc);
        cl.tap[j] = k;
        cl.coef[j] = fin ? (float)cf[s] : __builtin_nanf("");
        ++j;
      }
    }
    if (k == K - 1) cl.cnt[ch] = base + n;
  }
  __syncthreads();
}

// Geometry of one workgroup: channel block, output band, image run.
struct Work {
  int c0, p0, q0, n_begin, n_end, blk;
  int r0, t0;  // tile origin in the staged plane's lattice coordinates
};

__device__ __forceinline__ Work work_of(const Params& P) {
  Work wk;
  wk.blk = blockIdx.x;
  const int band = blockIdx.x % (P.nbp * P.nbq);
  const int run = blockIdx.x / (P.nbp * P.nbq);
  const int bp = band / P.nbq, bq = band - bp * P.nbq;
  wk.c0 = blockIdx.y * P.CB;
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

// Stages images n0 .. n0 + ng - 1 of the source plane (SH x SW, NCHW or
// NHWC) for the channel block into the tiles: the element (i, j) goes to
// tile position (i dil - r0, j dil - t0).  Only the in-plane lattice points
// are written; the rest of every tile stays zero from the workgroup's start.
template <typename T, int L>
__device__ void stage(const Params& P, const Work& wk, const T* __restrict__ src, float* tiles, int n0, int ng) {
  const int dil = P.dil;
  const int ilo = max(0, floor_div(wk.r0 + dil - 1, dil)), ihi = min(P.SH - 1, floor_div(wk.r0 + P.TR - 1, dil));
  const int jlo = max(0, floor_div(wk.t0 + dil - 1, dil)), jhi = min(P.SW - 1, floor_div(wk.t0 + P.TC - 1, dil));
  if (ihi < ilo || jhi < jlo) return;
  const int ni = ihi - ilo + 1, nj = jhi - jlo + 1;
  const int CB = P.CB;
  const int inner = L == kNHWC ? nj * CB : nj;  // NHWC: channel fastest
  const int total = ng * ni * inner;
  const size_t plane = (size_t)P.SH * P.SW;
  for (int e = threadIdx.x; e < total; e += kThreads) {
    const int row = e / inner, x = e - row * inner;
    const int g = row / ni, ii = row - g * ni;
    int jj, ch;
    if (L == kNHWC) {
      jj = x / CB;
      ch = x - jj * CB;
    } else {
      jj = x;
      ch = 0;
    }
    const int i = ilo + ii, j = jlo + jj, c = wk.c0 + ch;
    if (c >= P.C) continue;
    const int n = n0 + g;
    size_t idx;
    if (L == kNHWC)
      idx = (((size_t)n * P.SH + i) * P.SW + j) * P.C + c;
    else
      idx = ((size_t)n * P.C + c) * plane + (size_t)i * P.SW + j;
    tiles[(g * CB + ch) * P.TW + (i * dil - wk.r0) * P.TC + (j * dil - wk.t0)] = to_f32(src[idx]);
  }
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
  t.ch = r % P.CB;
  t.g = r / P.CB;
  return t;
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
  build_cells<T>(P, cl, wgt, theta, wk.c0, reinterpret_cast<int*>(tiles));
  for (int i = threadIdx.x; i < P.G * P.CB * P.TW; i += kThreads) tiles[i] = 0.f;
  __syncthreads();
  const int rstep = P.sig * P.TC;
  const int ntask = P.CB * P.NRG * P.BQ;  // per image
  float* otile = smem + P.out_off;         // NHWC output tile
  const int ostride = P.BP * P.BQ | 1;
  for (int n0 = wk.n_begin; n0 < wk.n_end; n0 += P.G) {
    const int ng = min(P.G, wk.n_end - n0);
    stage<T, L>(P, wk, in, tiles, n0, ng);
    __syncthreads();
    for (int tau = threadIdx.x; tau < ng * ntask; tau += kThreads) {
      const Task t = task_of(P, tau);
      const int* cw = cl.cw + 2 * t.ch * cl.ncap;
      const int nc = cl.cnt[t.ch];
      const float* tl = tiles + (t.g * P.CB + t.ch) * P.TW + (t.rg * P.RP * P.sig + P.hp) * P.TC + t.qq * P.sig + P.hp;
      float acc[RP];
#pragma unroll
      for (int i = 0; i < RP; ++i) acc[i] = 0.f;
      for (int j = 0; j < nc; ++j) {
        const int off = cw[2 * j];
        const float wc = __int_as_float(cw[2 * j + 1]);
        const float* a = tl + off;
#pragma unroll
        for (int i = 0; i < RP; ++i) acc[i] = fmaf(wc, a[i * rstep], acc[i]);
      }
      const int q = wk.q0 + t.qq;
      const int c = wk.c0 + t.ch;
      if (L == kNCHW) {
        if (q < P.OW && c < P.C) {
          T* o = out + ((size_t)(n0 + t.g) * P.C + c) * P.OH * P.OW + q;
#pragma unroll
          for (int i = 0; i < RP; ++i) {
            const int p = wk.p0 + t.rg * P.RP + i;
            if (t.rg * P.RP + i < P.BP && p < P.OH) store_elem(o + (size_t)p * P.OW, acc[i]);
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < RP; ++i) {
          const int pp = t.rg * P.RP + i;
          if (pp < P.BP) otile[(t.g * P.CB + t.ch) * ostride + pp * P.BQ + t.qq] = acc[i];
        }
      }
    }
    __syncthreads();  // the tiles are free (NHWC: the outputs are in the output tile)
    if (L == kNHWC) {
      // coalesced store, channel fastest
      const int nrow = min(P.BP, P.OH - wk.p0), ncol = min(P.BQ, P.OW - wk.q0);
      const int total = ng * nrow * ncol * P.CB;
      for (int e = threadIdx.x; e < total; e += kThreads) {
        const int ch = e % P.CB;
        int r = e / P.CB;
        const int qq = r % ncol;
        r /= ncol;
        const int pp = r % nrow, g = r / nrow;
        const int c = wk.c0 + ch;
        if (c >= P.C) continue;
        const size_t o = (((size_t)(n0 + g) * P.OH + wk.p0 + pp) * P.OW + wk.q0 + qq) * P.C + c;
        store_elem(out + o, otile[(g * P.CB + ch) * ostride + pp * P.BQ + qq]);
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- weight gradient

// Sum over the 64 lanes of each of 32 values: five halving exchanges leave
// lane L with the sum over its lane pair of value (L >> 1) & 31; the last
// exchange adds the pair.  Returns the total of value (L >> 1) & 31.
__device__ __forceinline__ float wave_sum32(float (&v)[kChunk]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 32, half = 16; m >= 2; m >>= 1, half >>= 1) {
    const bool up = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < half; ++i) {
      const float give = up ? v[i] : v[i + half];
      const float keep = up ? v[i + half] : v[i];
      v[i] = keep + __shfl_xor(give, m, 64);
    }
  }
  return v[0] + __shfl_xor(v[0], 1, 64);
}

// Adds the workgroup's sums of cells j0 .. j0 + 31 of channel ch, times the
// cells' coefficients, to the per-tap sums dwacc[ch * K + tap] in a fixed
// order.  All lanes hold accumulators of channel ch.
__device__ __forceinline__ void fold_chunk(const Params& P, const Cells& cl, float (&acc)[kChunk], int ch, int j0,
                                           float* red, float* dwacc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float s = wave_sum32(acc);
  if ((lane & 1) == 0) red[wave * kChunk + ((lane >> 1) & 31)] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int nc = cl.cnt[ch];
    for (int j = 0; j < kChunk && j0 + j < nc; ++j) {
      float v = 0.f;
      for (int w = 0; w < kThreads / 64; ++w) v += red[w * kChunk + j];
      const int cj = ch * cl.ncap + j0 + j;
      dwacc[ch * P.K + cl.tap[cj]] += cl.coef[cj] * v;
    }
  }
  __syncthreads();
}

// The dy values of a lane's RP outputs (zero outside the output plane).
template <typename T, int L, int RP>
__device__ __forceinline__ void load_dy(const Params& P, const Work& wk, const Task& t, const T* __restrict__ dy,
                                        const float* dtile, int n, float (&d)[RP]) {
  const int q = wk.q0 + t.qq, c = wk.c0 + t.ch;
  const int ostride = P.BP * P.BQ | 1;
#pragma unroll
  for (int i = 0; i < RP; ++i) {
    const int pp = t.rg * P.RP + i, p = wk.p0 + pp;
    float v = 0.f;
    if (pp < P.BP && p < P.OH && q < P.OW && c < P.C) {
      if (L == kNCHW)
        v = to_f32(dy[((size_t)n * P.C + c) * P.OH * P.OW + (size_t)p * P.OW + q]);
      else
        v = dtile[(t.g * P.CB + t.ch) * ostride + pp * P.BQ + t.qq];
    }
    d[i] = v;
  }
}

// NHWC: stages dy of the band into the dy tile (channel fastest in memory).
template <typename T>
__device__ void stage_dy_nhwc(const Params& P, const Work& wk, const T* __restrict__ dy, float* dtile, int n0,
                              int ng) {
  const int nrow = min(P.BP, P.OH - wk.p0), ncol = min(P.BQ, P.OW - wk.q0);
  const int ostride = P.BP * P.BQ | 1;
  const int total = ng * nrow * ncol * P.CB;
  for (int e = threadIdx.x; e < total; e += kThreads) {
    const int ch = e % P.CB;
    int r = e / P.CB;
    const int qq = r % ncol;
    r /= ncol;
    const int pp = r % nrow, g = r / nrow;
    const int c = wk.c0 + ch;
    if (c >= P.C) continue;
    const size_t o = (((size_t)(n0 + g) * P.OH + wk.p0 + pp) * P.OW + wk.q0 + qq) * P.C + c;
    dtile[(g * P.CB + ch) * ostride + pp * P.BQ + qq] = to_f32(dy[o]);
  }
}

// partial[(blk * C + c) * K + k] = the workgroup's sum over its band and
// images of dy[p,q] * sum_cells coef x[str p + a, str q + b] for the cells of
// tap k (Eq. 1 differentiated in w_k).  Cells are taken 32 at a time (one
// accumulator register each); per group of 32 the images are staged again.
template <typename T, int L, int RP>
__global__ __launch_bounds__(kThreads) void gen_wgrad(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                      const float* __restrict__ theta, float* __restrict__ partial) {
  extern __shared__ float smem[];
  const Work wk = work_of(P);
  const Cells cl(smem, P);
  float* tiles = smem + P.tile_off;
  build_cells<T>(P, cl, static_cast<const T*>(nullptr), theta, wk.c0, reinterpret_cast<int*>(tiles));
  for (int i = threadIdx.x; i < P.G * P.CB * P.TW; i += kThreads) tiles[i] = 0.f;
  float* red = smem + P.red_off;
  float* dwacc = red + (kThreads / 64) * kChunk;
  for (int i = threadIdx.x; i < P.CB * P.K; i += kThreads) dwacc[i] = 0.f;
  float* dtile = smem + P.out_off;
  __syncthreads();
  const int rstep = P.sig * P.TC;
  const int per_ch = P.NRG * P.BQ;  // tasks per image and channel
  int maxc = 0;
  for (int ch = 0; ch < P.CB; ++ch) maxc = max(maxc, cl.cnt[ch]);
  for (int j0 = 0; j0 < maxc; j0 += kChunk) {
    for (int ch = 0; ch < P.CB; ++ch) {
      if (j0 >= cl.cnt[ch]) continue;  // uniform: every lane reads the same count
      float acc[kChunk];
#pragma unroll
      for (int j = 0; j < kChunk; ++j) acc[j] = 0.f;
      const int nc = min(kChunk, cl.cnt[ch] - j0);
      const int* cw = cl.cw + 2 * (ch * cl.ncap + j0);
      for (int n0 = wk.n_begin; n0 < wk.n_end; n0 += P.G) {
        const int ng = min(P.G, wk.n_end - n0);
        // the tiles hold x of this pass's images (staged again for every
        // channel and cell group: the accumulators of one channel's 32 cells
        // run over all the workgroup's images)
        __syncthreads();
        stage<T, L>(P, wk, x, tiles, n0, ng);
        if (L == kNHWC) stage_dy_nhwc<T>(P, wk, dy, dtile, n0, ng);
        __syncthreads();
        for (int tau = threadIdx.x; tau < ng * per_ch; tau += kThreads) {
          Task t;
          t.qq = tau % P.BQ;
          const int r = tau / P.BQ;
          t.rg = r % P.NRG;
          t.g = r / P.NRG;
          t.ch = ch;
          float d[RP];
          load_dy<T, L, RP>(P, wk, t, dy, dtile, n0 + t.g, d);
          const float* tl =
              tiles + (t.g * P.CB + ch) * P.TW + (t.rg * P.RP * P.sig + P.hp) * P.TC + t.qq * P.sig + P.hp;
#pragma unroll
          for (int j = 0; j < kChunk; ++j) {
            if (j < nc) {
              const float* a = tl + cw[2 * j];
              float s = 0.f;
#pragma unroll
              for (int i = 0; i < RP; ++i) s = fmaf(d[i], a[i * rstep], s);
              acc[j] += s;
            }
          }
        }
      }
      fold_chunk(P, cl, acc, ch, j0, red, dwacc);
    }
  }
  for (int i = threadIdx.x; i < P.CB * P.K; i += kThreads) {
    const int ch = i / P.K, k = i - ch * P.K, c = wk.c0 + ch;
    if (c < P.C) partial[((size_t)wk.blk * P.C + c) * P.K + k] = isfinite(theta[c]) ? dwacc[i] : __builtin_nanf("");
  }
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
template <typename T, int L, int RP>
const void* wgrad_fn() { return reinterpret_cast<const void*>(gen_wgrad<T, L, RP>); }

template <typename T, int L, int RP>
hipError_t gather_launch(const Plan& pl, const void* in, const void* w, const float* theta, void* out,
                         hipStream_t stream) {
  const hipError_t e = allow_lds<gather_fn<T, L, RP>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gen_gather<T, L, RP>), dim3((unsigned)pl.grid_x, (unsigned)pl.grid_y), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta,
                     static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int L, int RP>
hipError_t wgrad_launch(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                        hipStream_t stream) {
  hipError_t e = allow_lds<wgrad_fn<T, L, RP>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gen_wgrad<T, L, RP>), dim3((unsigned)pl.grid_x, (unsigned)pl.grid_y), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int CK = pl.p.C * pl.p.K;
  hipLaunchKernelGGL(gen_wgrad_reduce<T>, dim3((unsigned)((CK + 255) / 256)), dim3(256), 0, stream, partial,
                     static_cast<T*>(dw), CK, (int)pl.parts);
  return hipGetLastError();
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

template <typename T>
hipError_t wgrad_t(const Plan& pl, int layout, const void* x, const void* dy, const float* theta, void* dw,
                   float* partial, hipStream_t stream) {
  if (layout == kNHWC)
    return pl.p.RP == 4 ? wgrad_launch<T, kNHWC, 4>(pl, x, dy, theta, dw, partial, stream)
                        : wgrad_launch<T, kNHWC, 8>(pl, x, dy, theta, dw, partial, stream);
  return pl.p.RP == 4 ? wgrad_launch<T, kNCHW, 4>(pl, x, dy, theta, dw, partial, stream)
                      : wgrad_launch<T, kNCHW, 8>(pl, x, dy, theta, dw, partial, stream);
}

}  // namespace
}  // namespace gen
}  // namespace o1d
