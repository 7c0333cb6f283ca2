// Device code of the plane kernels (included by o1d_plane_f32.hip and
// o1d_plane_bf16.hip); the host plan is in o1d_plane.h.
//
// The operation (Definition 1, Eq. 1-2) is a list of cells per channel: a
// cell is an integer offset (a, b) (Eq. 2's rounded-down offsets of a tap,
// or one corner of the bilinear interpolation at its unrounded offsets, the
// alternative of the section "Discretization and Interpolation") with the
// weight w_k coef.  y[p,q] = sum over cells of weight x[sig p + a, sig q + b],
// zero outside the plane; the input gradients use the mirrored cells (-a, -b)
// on dy spread onto the stride lattice.
//
// Cells are kept in tap order.  Along a line through the origin both
// components of the rounded-down offset change monotonically with the tap,
// so the cells that reach the plane from a group of RP x R outputs are one
// contiguous run: the run of the group's rows intersected with the run of
// its columns.  Between two bilinear corners that reach the plane every cell
// lies at most one row or column further out (the corners' base offsets are
// monotone too), which the tile margin's extra row and column absorb.  A
// group's lanes read only the cells of its run, so taps that fall outside a
// small plane cost nothing.
//
// Lanes of a wave are NI images x R columns of one channel; the tile is
// [row][column][image] in 32-bit words, so one cell's read by the wave hits
// NI consecutive words (no bank conflicts).  Outputs go through an
// output-shaped tile [image][element] (an odd word stride per image), from
// which each image's plane is stored with vector writes.
#pragma once

#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_plane.h"
#include "o1d_wave.h"

namespace o1d {
namespace plane {
namespace {

using wave::static_for;

// LDS of one workgroup (byte offsets from the plan).
struct Lds {
  int2* cw;     // per cell: tile offset (a TCm + b) NI in words, weight bits
  int2* ab;     // per cell: (a, b), mirrored for the input gradients
  int* tap;     // per cell: its tap
  float* coef;  // per cell: its coefficient
  int* first;   // per tap: its first cell (first[K]: the cell count)
  int2* rr;     // per row group: cell run [lo, hi) of its rows
  int2* cc;     // per column group: cell run of its columns
  float* tile;
  unsigned char* aux;
  float* red;
  __device__ __forceinline__ Lds(unsigned char* s, const Params& P) {
    cw = reinterpret_cast<int2*>(s + P.cell_off);
    ab = cw + P.ncap;
    tap = reinterpret_cast<int*>(ab + P.ncap);
    coef = reinterpret_cast<float*>(tap + P.ncap);
    first = reinterpret_cast<int*>(coef + P.ncap);
    rr = reinterpret_cast<int2*>(s + P.ival_off);
    cc = rr + P.nrg;
    tile = reinterpret_cast<float*>(s + P.tile_off);
    aux = s + P.aux_off;
    red = reinterpret_cast<float*>(s + P.red_off);
  }
};

// Builds channel c's cells: thread k computes tap k's one (rounded down) or
// up to four (bilinear; corners with a zero coefficient dropped) cells;
// `scratch` (K ints) holds the per-tap counts for the prefix sum.  A
// non-finite angle gives every tap one cell at (0, 0) with a NaN weight and
// coefficient, which makes every output of the channel NaN.  Slots past the
// last cell hold offset 0 and weight 0.  Ends with a barrier.
template <typename T>
__device__ void build_cells(const Params& P, const Lds& L, const T* __restrict__ wgt, const float* __restrict__ theta,
                            int c, int* scratch) {
  const int t = threadIdx.x, K = P.K;
  double cf[4] = {0.0, 0.0, 0.0, 0.0};
  int h0 = 0, w0 = 0, n = 0;
  bool fin = true;
  for (int j = t; j < P.ncap; j += kThreads) {
    L.cw[j] = make_int2(0, 0);
    L.ab[j] = make_int2(0, 0);
    L.tap[j] = 0;
    L.coef[j] = 0.f;
  }
  if (t < K) {
    double rh, rw;
    fin = tap_real(theta[c], K, t, &rh, &rw);
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
  if (t < K) {
    int base = t;
    if (P.mode != 0) {
      base = 0;
      for (int i = 0; i < t; ++i) base += scratch[i];
    }
    const float wk = wgt ? to_f32(wgt[(size_t)c * K + t]) : 0.f;
    int j = base;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (cf[s] != 0.0) {
        const int a = P.sign * (h0 + (s >> 1)), b = P.sign * (w0 + (s & 1));
        const float wc = fin ? (float)((double)wk * cf[s]) : __builtin_nanf("");
        L.cw[j] = make_int2((a * P.TCm + b) * P.NI, __float_as_int(wc));
        L.ab[j] = make_int2(a, b);
        L.tap[j] = t;
        L.coef[j] = fin ? (float)cf[s] : __builtin_nanf("");
        ++j;
      }
    }
    L.first[t] = base;
    if (t == K - 1) L.first[K] = base + n;
  }
  __syncthreads();
}

// Empty cell runs and a zero tile (its margins stay zero; staging writes the
// plane).  A barrier must follow before cell_runs and staging.
__device__ __forceinline__ void prepare(const Params& P, const Lds& L) {
  for (int g = threadIdx.x; g < P.nrg + P.ncg; g += kThreads) L.rr[g] = make_int2(INT_MAX, INT_MIN);
  float4* t4 = reinterpret_cast<float4*>(L.tile);
  const int n4 = P.TRm * P.TCm * P.NI / 4;
  for (int i = threadIdx.x; i < n4; i += kThreads) t4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

// Cell runs: row group g (output rows g RP .. g RP + RP - 1) can reach the
// plane with cell j iff its frame rows sig p + a span a range that meets
// [0, H); likewise for columns.  Each run is the hull [min j, max j + 1).
__device__ __forceinline__ void cell_runs(const Params& P, const Lds& L) {
  const int n = L.first[P.K];
  const int ng = P.nrg + P.ncg;
  for (int m = threadIdx.x; m < ng * n; m += kThreads) {
    const int g = m / n, j = m - g * n;
    const int2 ab = L.ab[j];
    bool ok;
    if (g < P.nrg) {
      const int f0 = g * P.RP * P.sig + ab.x;
      ok = f0 <= P.H - 1 && f0 + (P.RP - 1) * P.sig >= 0;
    } else {
      const int f0 = (g - P.nrg) * P.R * P.sig + ab.y;
      ok = f0 <= P.W - 1 && f0 + (P.R - 1) * P.sig >= 0;
    }
    if (ok) {
      atomicMin(&L.rr[g].x, j);
      atomicMax(&L.rr[g].y, j + 1);
    }
  }
}

// q = a / b for 0 <= a < 2^24, 0 < b, from a float reciprocal of b (one
// correction step makes it exact).
__device__ __forceinline__ int fdiv(int a, int b, float rb) {
  int q = (int)((float)a * rb);
  const int r = a - q * b;
  q += r < 0 ? -1 : (r >= b ? 1 : 0);
  return q;
}

template <typename T, int V>
struct VecT;
template <> struct VecT<float, 4> { using type = float4; };
template <> struct VecT<float, 2> { using type = float2; };
template <> struct VecT<float, 1> { using type = float; };
template <> struct VecT<uint16_t, 4> { using type = uint2; };
template <> struct VecT<uint16_t, 2> { using type = uint32_t; };
template <> struct VecT<uint16_t, 1> { using type = uint16_t; };

template <typename T, int V>
__device__ __forceinline__ void load_raw(const T* p, T (&v)[V]) {
  using VT = typename VecT<T, V>::type;
  const VT x = *reinterpret_cast<const VT*>(p);
  __builtin_memcpy(v, &x, sizeof(VT));
}

template <typename T, int V>
__device__ __forceinline__ void store_raw(T* p, const T (&v)[V]) {
  using VT = typename VecT<T, V>::type;
  VT x;
  __builtin_memcpy(&x, v, sizeof(VT));
  *reinterpret_cast<VT*>(p) = x;
}

// Images n0 .. n0 + ng - 1 of channel c of the staged plane (SH x SW) into
// the tile: element (i, j) of image g goes to frame position (i dil, j dil).
// Work item m is (image m mod NI, chunk m / NI of V elements), so that the
// LDS writes of a wave go to consecutive words; four chunks per lane are
// loaded before any is written.
template <typename T, int V>
__device__ __forceinline__ void stage_tile_v(const Params& P, const T* __restrict__ src, int n0, int ng, int c,
                                             float* tile) {
  const int E = P.SH * P.SW, total = (E / V) << P.lni;
  const float rsw = 1.f / (float)P.SW;
  for (int m0 = threadIdx.x; m0 < total; m0 += 4 * kThreads) {
    T v[4][V];
    int e[4], img[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int m = m0 + u * kThreads;
      img[u] = m & (P.NI - 1);
      e[u] = -1;
      if (m < total && img[u] < ng) {
        e[u] = (m >> P.lni) * V;
        load_raw<T, V>(src + ((size_t)(n0 + img[u]) * P.C + c) * E + e[u], v[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (e[u] >= 0) {
        int row = fdiv(e[u], P.SW, rsw), col = e[u] - row * P.SW;
#pragma unroll
        for (int s = 0; s < V; ++s) {
          tile[((row * P.dil + P.mr) * P.TCm + col * P.dil + P.mc) * P.NI + img[u]] = to_f32(v[u][s]);
          if (++col == P.SW) {
            col = 0;
            ++row;
          }
        }
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ void stage_tile(const Params& P, const T* __restrict__ src, int n0, int ng, int c,
                                           float* tile) {
  if (P.vt == 4)
    stage_tile_v<T, 4>(P, src, n0, ng, c, tile);
  else if (P.vt == 2)
    stage_tile_v<T, 2>(P, src, n0, ng, c, tile);
  else
    stage_tile_v<T, 1>(P, src, n0, ng, c, tile);
}

// Images n0 .. n0 + ng - 1 of channel c of an output-shaped plane (OH x OW)
// into the output-shaped tile aux[image OSz + element], unconverted.
template <typename T, int V>
__device__ __forceinline__ void stage_aux_v(const Params& P, const T* __restrict__ src, int n0, int ng, int c,
                                            T* aux) {
  const int E = P.OH * P.OW, total = (E / V) << P.lni;
  for (int m0 = threadIdx.x; m0 < total; m0 += 4 * kThreads) {
    T v[4][V];
    int e[4], img[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int m = m0 + u * kThreads;
      img[u] = m & (P.NI - 1);
      e[u] = -1;
      if (m < total && img[u] < ng) {
        e[u] = (m >> P.lni) * V;
        load_raw<T, V>(src + ((size_t)(n0 + img[u]) * P.C + c) * E + e[u], v[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (e[u] >= 0) {
#pragma unroll
        for (int s = 0; s < V; ++s) aux[img[u] * P.OSz + e[u] + s] = v[u][s];
      }
  }
}

template <typename T>
__device__ __forceinline__ void stage_aux(const Params& P, const T* __restrict__ src, int n0, int ng, int c, T* aux) {
  if (P.va == 4)
    stage_aux_v<T, 4>(P, src, n0, ng, c, aux);
  else if (P.va == 2)
    stage_aux_v<T, 2>(P, src, n0, ng, c, aux);
  else
    stage_aux_v<T, 1>(P, src, n0, ng, c, aux);
}

// The output-shaped tile's images n0 .. n0 + ng - 1 to channel c of dst.
template <typename T, int V>
__device__ __forceinline__ void store_aux_v(const Params& P, T* __restrict__ dst, int n0, int ng, int c,
                                            const T* aux) {
  const int E = P.OH * P.OW, total = (E / V) << P.lni;
  for (int m = threadIdx.x; m < total; m += kThreads) {
    const int img = m & (P.NI - 1), e = (m >> P.lni) * V;
    if (img < ng) {
      T v[V];
#pragma unroll
      for (int s = 0; s < V; ++s) v[s] = aux[img * P.OSz + e + s];
      store_raw<T, V>(dst + ((size_t)(n0 + img) * P.C + c) * E + e, v);
    }
  }
}

template <typename T>
__device__ __forceinline__ void store_aux(const Params& P, T* __restrict__ dst, int n0, int ng, int c, const T* aux) {
  if (P.va == 4)
    store_aux_v<T, 4>(P, dst, n0, ng, c, aux);
  else if (P.va == 2)
    store_aux_v<T, 2>(P, dst, n0, ng, c, aux);
  else
    store_aux_v<T, 1>(P, dst, n0, ng, c, aux);
}

// A lane's place: image img of the workgroup, column r of its group.
struct Lane {
  int img, r;
  __device__ __forceinline__ explicit Lane(const Params& P) {
    const int l = threadIdx.x & 63;
    img = l & (P.NI - 1);
    r = l >> P.lni;
  }
};

// Group `it`: its first output row p0, the lane's output column q, the cell
// run [lo, hi) (uniform) and the lane's tile address at cell offset 0.
struct Group {
  int p0, q, lo, hi;
  const float* tb;
  __device__ __forceinline__ Group(const Params& P, const Lds& L, const Lane& ln, int it, int RP) {
    const int rg = it / P.ncg, cg = it - rg * P.ncg;
    const int2 a = L.rr[rg], b = L.cc[cg];
    lo = __builtin_amdgcn_readfirstlane(max(a.x, b.x));
    hi = __builtin_amdgcn_readfirstlane(min(a.y, b.y));
    p0 = rg * RP;
    q = cg * P.R + ln.r;
    tb = L.tile + ((p0 * P.sig + P.mr) * P.TCm + q * P.sig + P.mc) * P.NI + ln.img;
  }
};

// ---------------------------------------------------------------- gather

// out[p,q] = sum over the channel's cells of weight * frame[sig p + a, sig q + b]:
// the forward pass (x, cells at +(a, b)) and the input gradient (dy on the
// stride lattice, cells at -(a, b), sig 1).
template <typename T, int RP>
__global__ __launch_bounds__(kThreads) void plane_gather(Params P, const T* __restrict__ in,
                                                         const T* __restrict__ wgt, const float* __restrict__ theta,
                                                         T* __restrict__ out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Lds L(smem, P);
  const int c = blockIdx.x % P.C, n0 = (blockIdx.x / P.C) * P.NI, ng = min(P.NI, P.N - n0);
  build_cells<T>(P, L, wgt, theta, c, reinterpret_cast<int*>(L.tile));
  prepare(P, L);
  __syncthreads();
  cell_runs(P, L);
  stage_tile<T>(P, in, n0, ng, c, L.tile);
  __syncthreads();
  T* aux = reinterpret_cast<T*>(L.aux);
  const Lane ln(P);
  const int rs = P.sig * P.TCm * P.NI;  // words per output row
  for (int it = threadIdx.x >> 6; it < P.nitems; it += kWaves) {
    const Group gr(P, L, ln, it, RP);
    float acc[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) acc[i] = 0.f;
    int t = gr.lo;
    if (t + 4 <= gr.hi) {
      // four cells per step; the next four table entries (inside the table:
      // it has eight slots past the last cell) are read before this step's
      // tile reads
      int2 cur[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) cur[u] = L.cw[t + u];
      for (;;) {
        int2 nxt[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) nxt[u] = L.cw[t + 4 + u];
        float v[4][RP];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int i = 0; i < RP; ++i) v[u][i] = gr.tb[cur[u].x + i * rs];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int i = 0; i < RP; ++i) acc[i] = fmaf(__int_as_float(cur[u].y), v[u][i], acc[i]);
        t += 4;
        if (t + 4 > gr.hi) break;
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = nxt[u];
      }
    }
    for (; t < gr.hi; ++t) {
      const int2 cl = L.cw[t];
#pragma unroll
      for (int i = 0; i < RP; ++i) acc[i] = fmaf(__int_as_float(cl.y), gr.tb[cl.x + i * rs], acc[i]);
    }
    if (gr.q < P.OW) {
      T* ax = aux + ln.img * P.OSz + gr.q;
#pragma unroll
      for (int i = 0; i < RP; ++i)
        if (gr.p0 + i < P.OH) ax[(gr.p0 + i) * P.OW] = from_f32<T>(acc[i]);
    }
  }
  __syncthreads();
  store_aux<T>(P, out, n0, ng, c, aux);
}

// ---------------------------------------------------------------- weight gradients

// Cells J of the group of KB (table cw) taken four at a time; a cell of the
// four outside the run [lo, hi) reads the lane's own tile word (inside the
// tile) and counts for nothing.  f(J, in, weight, v[RP]) consumes a cell.
template <int RP, int KB, class F>
__device__ __forceinline__ void each_cell(const int2* cw, int lo, int hi, const float* tb, int rs, F&& f) {
  static_for<KB / 4>([&](auto g) __attribute__((always_inline)) {
    constexpr int J0 = 4 * decltype(g)::value;
    if (J0 + 4 > lo && J0 < hi) {
      const int4* c4 = reinterpret_cast<const int4*>(cw + J0);
      const int4 a = c4[0], b = c4[1];
      const int off[4] = {a.x, a.z, b.x, b.z};
      const int wb[4] = {a.y, a.w, b.y, b.w};
      float v[4][RP];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool in = J0 + u >= lo && J0 + u < hi;
        const int o = in ? off[u] : 0;
#pragma unroll
        for (int i = 0; i < RP; ++i) v[u][i] = tb[o + i * rs];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) f(J0 + u, J0 + u >= lo && J0 + u < hi, __int_as_float(wb[u]), v[u]);
    }
  });
}

// Adds the workgroup's per-cell sums (cells j0 .. j0 + KB - 1 of the
// channel, in acc of every lane) times their coefficients to the per-tap sums
// dwacc[k]: thread k folds the cells of tap k (a contiguous run) in order.
template <int KB>
__device__ __forceinline__ void fold_cells(const Params& P, const Lds& L, float (&acc)[KB], int j0, float* dwacc) {
  wave::sums<KB>(acc, L.red);
  __syncthreads();
  for (int k = threadIdx.x; k < P.K; k += kThreads) {
    const int j1 = max(L.first[k], j0), j2 = min(L.first[k + 1], j0 + KB);
    float s = dwacc[k];
    for (int j = j1; j < j2; ++j) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += L.red[w * KB + (j - j0)];
      s += L.coef[j] * v;
    }
    dwacc[k] = s;
  }
  __syncthreads();
}

// partial[(chunk C + c) K + k] = sum over the workgroup's images and outputs
// of dy[p,q] * sum over the cells of tap k of coef x[sig p + a, sig q + b]
// (Eq. 1 differentiated in w_k).
template <typename T, int RP, int KB>
__global__ __launch_bounds__(kThreads) void plane_wgrad(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                        const float* __restrict__ theta,
                                                        float* __restrict__ partial) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Lds L(smem, P);
  const int c = blockIdx.x % P.C, chunk = blockIdx.x / P.C, n0 = chunk * P.NI, ng = min(P.NI, P.N - n0);
  build_cells<T>(P, L, static_cast<const T*>(nullptr), theta, c, reinterpret_cast<int*>(L.tile));
  prepare(P, L);
  float* dwacc = L.red + kWaves * KB;
  for (int k = threadIdx.x; k < P.K; k += kThreads) dwacc[k] = 0.f;
  __syncthreads();
  cell_runs(P, L);
  stage_tile<T>(P, x, n0, ng, c, L.tile);
  T* aux = reinterpret_cast<T*>(L.aux);
  stage_aux<T>(P, dy, n0, ng, c, aux);
  __syncthreads();
  const Lane ln(P);
  const int rs = P.sig * P.TCm * P.NI;
  const int n = __builtin_amdgcn_readfirstlane(L.first[P.K]);
  for (int j0 = 0; j0 < n; j0 += KB) {
    float acc[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) acc[j] = 0.f;
    for (int it = threadIdx.x >> 6; it < P.nitems; it += kWaves) {
      const Group gr(P, L, ln, it, RP);
      const int lo = max(gr.lo, j0) - j0, hi = min(gr.hi, j0 + KB) - j0;
      if (lo >= hi) continue;
      float d[RP];
      const bool col_ok = ln.img < ng && gr.q < P.OW;
#pragma unroll
      for (int i = 0; i < RP; ++i)
        d[i] = col_ok && gr.p0 + i < P.OH ? to_f32(aux[ln.img * P.OSz + (gr.p0 + i) * P.OW + gr.q]) : 0.f;
      each_cell<RP, KB>(L.cw + j0, lo, hi, gr.tb, rs,
                        [&](int J, bool in, float, const float (&v)[RP]) __attribute__((always_inline)) {
                          float s = 0.f;
#pragma unroll
                          for (int i = 0; i < RP; ++i) s = fmaf(d[i], v[i], s);
                          acc[J] += in ? s : 0.f;
                        });
    }
    fold_cells<KB>(P, L, acc, j0, dwacc);
  }
  for (int k = threadIdx.x; k < P.K; k += kThreads)
    partial[((size_t)chunk * P.C + c) * P.K + k] = isfinite(theta[c]) ? dwacc[k] : __builtin_nanf("");
}

// Both gradients in one pass (stride 1, rounded-down offsets): the tile holds
// dy, the output-shaped tile x.  Per mirrored cell every dy value v read for
// the lane's input-gradient outputs h adds w_c v to dx[h] and x[h] v to the
// cell's sum, which is the weight gradient of the cell's tap:
// dw_k = sum_h x[h] dy[h - off_k].  dx replaces x in the output-shaped tile
// (each output is read and written by one lane only).
template <typename T, int RP, int KB>
__global__ __launch_bounds__(kThreads) void plane_bwd(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                      const T* __restrict__ wgt, const float* __restrict__ theta,
                                                      T* __restrict__ dx, float* __restrict__ partial) {
  extern __shared__ __align__(16) unsigned char smem[];
  const Lds L(smem, P);
  const int c = blockIdx.x % P.C, chunk = blockIdx.x / P.C, n0 = chunk * P.NI, ng = min(P.NI, P.N - n0);
  build_cells<T>(P, L, wgt, theta, c, reinterpret_cast<int*>(L.tile));
  prepare(P, L);
  float* dwacc = L.red + kWaves * KB;
  for (int k = threadIdx.x; k < P.K; k += kThreads) dwacc[k] = 0.f;
  __syncthreads();
  cell_runs(P, L);
  stage_tile<T>(P, dy, n0, ng, c, L.tile);
  T* aux = reinterpret_cast<T*>(L.aux);
  stage_aux<T>(P, x, n0, ng, c, aux);
  __syncthreads();
  const Lane ln(P);
  const int rs = P.TCm * P.NI;
  float acc[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) acc[j] = 0.f;
  for (int it = threadIdx.x >> 6; it < P.nitems; it += kWaves) {
    const Group gr(P, L, ln, it, RP);
    const bool col_ok = ln.img < ng && gr.q < P.OW;
    T* ax = aux + ln.img * P.OSz + gr.q;
    float xv[RP], o[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) {
      xv[i] = col_ok && gr.p0 + i < P.OH ? to_f32(ax[(gr.p0 + i) * P.OW]) : 0.f;
      o[i] = 0.f;
    }
    each_cell<RP, KB>(L.cw, gr.lo, gr.hi, gr.tb, rs,
                      [&](int J, bool in, float wc, const float (&v)[RP]) __attribute__((always_inline)) {
                        const float we = in ? wc : 0.f;
                        float s = 0.f;
#pragma unroll
                        for (int i = 0; i < RP; ++i) {
                          o[i] = fmaf(we, v[i], o[i]);
                          s = fmaf(xv[i], v[i], s);
                        }
                        acc[J] += in ? s : 0.f;
                      });
    if (col_ok) {
#pragma unroll
      for (int i = 0; i < RP; ++i)
        if (gr.p0 + i < P.OH) ax[(gr.p0 + i) * P.OW] = from_f32<T>(o[i]);
    }
  }
  __syncthreads();
  store_aux<T>(P, dx, n0, ng, c, aux);
  fold_cells<KB>(P, L, acc, 0, dwacc);
  for (int k = threadIdx.x; k < P.K; k += kThreads)
    partial[((size_t)chunk * P.C + c) * P.K + k] = isfinite(theta[c]) ? dwacc[k] : __builtin_nanf("");
}

// ---------------------------------------------------------------- launch

template <typename T>
constexpr Dtype dtype_of() {
  return sizeof(T) == 4 ? Dtype::F32 : Dtype::BF16;
}

template <const void* (*Fn)()>
hipError_t allow_lds() {
  static int done = 0;  // benign race: the attribute call is idempotent
  if (done) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(Fn(), hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLdsBytes);
  if (e == hipSuccess) done = 1;
  return e;
}
template <typename T, int RP>
const void* gather_fn() { return reinterpret_cast<const void*>(plane_gather<T, RP>); }
template <typename T, int RP, int KB>
const void* wgrad_fn() { return reinterpret_cast<const void*>(plane_wgrad<T, RP, KB>); }
template <typename T, int RP, int KB>
const void* bwd_fn() { return reinterpret_cast<const void*>(plane_bwd<T, RP, KB>); }

template <typename T, int RP>
hipError_t gather_launch(const Plan& pl, const void* in, const void* w, const float* theta, void* out,
                         hipStream_t stream) {
  const hipError_t e = allow_lds<gather_fn<T, RP>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((plane_gather<T, RP>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream,
                     pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta, static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int RP, int KB>
hipError_t wgrad_launch(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                        hipStream_t stream) {
  hipError_t e = allow_lds<wgrad_fn<T, RP, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((plane_wgrad<T, RP, KB>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream,
                     pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_partial_sum(dtype_of<T>(), partial, dw, pl.p.C * pl.p.K, (int)pl.parts, stream);
}

template <typename T, int RP, int KB>
hipError_t bwd_launch(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx,
                      void* dw, float* partial, hipStream_t stream) {
  hipError_t e = allow_lds<bwd_fn<T, RP, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((plane_bwd<T, RP, KB>), dim3((unsigned)pl.p.nblocks), dim3(kThreads), pl.lds_bytes, stream,
                     pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), static_cast<const T*>(w), theta,
                     static_cast<T*>(dx), partial);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_partial_sum(dtype_of<T>(), partial, dw, pl.p.C * pl.p.K, (int)pl.parts, stream);
}

template <typename T>
hipError_t gather_t(const Plan& pl, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
  return pl.p.RP == 4 ? gather_launch<T, 4>(pl, in, w, theta, out, stream)
                      : gather_launch<T, 2>(pl, in, w, theta, out, stream);
}

template <typename T, int RP>
hipError_t wgrad_kb(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                    hipStream_t stream) {
  if (pl.p.KB == 32) return wgrad_launch<T, RP, 32>(pl, x, dy, theta, dw, partial, stream);
  if (pl.p.KB == 64) return wgrad_launch<T, RP, 64>(pl, x, dy, theta, dw, partial, stream);
  return wgrad_launch<T, RP, 128>(pl, x, dy, theta, dw, partial, stream);
}

template <typename T>
hipError_t wgrad_t(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                   hipStream_t stream) {
  return pl.p.RP == 4 ? wgrad_kb<T, 4>(pl, x, dy, theta, dw, partial, stream)
                      : wgrad_kb<T, 2>(pl, x, dy, theta, dw, partial, stream);
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
  return pl.p.RP == 4 ? bwd_kb<T, 4>(pl, x, dy, w, theta, dx, dw, partial, stream)
                      : bwd_kb<T, 2>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace
}  // namespace plane
}  // namespace o1d
