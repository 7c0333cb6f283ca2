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
// Lanes of a wave are NI / 2 image pairs x R columns of one channel; the tile
// is [row][column][image] in 32-bit words, so a lane reads its two images of
// one cell with a 64-bit access and the wave's reads hit consecutive words
// (no bank conflicts).  Outputs go through an
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

// LDS of one workgroup (byte offsets from the plan): the cell table of slot
// `use(slot)`, the tile, the output-shaped tile and the reduction area.
struct Lds {
  int2* cw;     // per cell: tile offset (a TCm + b) NI in bytes, weight bits
  int2* ab;     // per cell: (a, b), mirrored for the input gradients
  int* tap;     // per cell: its tap
  float* coef;  // per cell: its coefficient
  int* first;   // per tap: its first cell (first[K]: the cell count)
  int* counts;  // per tap: its number of cells (scratch of the build)
  int2* rr;     // per row group: cell run [lo, hi) of its rows
  int2* cc;     // per column group: cell run of its columns
  float* tile;
  unsigned char* aux;
  float* red;
  unsigned char* base;
  __device__ __forceinline__ Lds(unsigned char* s, const Params& P) : base(s) {
    use(P, 0);
    tile = reinterpret_cast<float*>(s + P.tile_off);
    aux = s + P.aux_off;
    red = reinterpret_cast<float*>(s + P.red_off);
  }
  __device__ __forceinline__ void use(const Params& P, int slot) {
    unsigned char* t = base + slot * P.table_bytes;
    cw = reinterpret_cast<int2*>(t);
    ab = cw + P.ncap;
    tap = reinterpret_cast<int*>(ab + P.ncap);
    coef = reinterpret_cast<float*>(tap + P.ncap);
    first = reinterpret_cast<int*>(coef + P.ncap);
    counts = first + P.K + 1;
    rr = reinterpret_cast<int2*>(t + P.ival_off);
    cc = rr + P.nrg;
  }
};

// Builds the channel's cells from its angle th (every thread) and thread k's
// tap weight wk: thread k computes tap k's one (rounded down) or up to four
// (bilinear; corners with a zero coefficient dropped) cells.  A
// non-finite angle gives every tap one cell at (0, 0) with a NaN weight and
// coefficient, which makes every output of the channel NaN.  Slots past the
// last cell hold offset 0 and weight 0; the cell runs are emptied for
// cell_runs.  Ends with a barrier.
__device__ void build_cells(const Params& P, const Lds& L, float th, float wk) {
  int* scratch = L.counts;
  const int t = threadIdx.x, K = P.K;
  double cf[4] = {0.0, 0.0, 0.0, 0.0};
  int h0 = 0, w0 = 0, n = 0;
  bool fin = true;
  for (int g = t; g < P.nrg + P.ncg; g += kThreads) L.rr[g] = make_int2(INT_MAX, INT_MIN);
  for (int j = t; j < P.ncap; j += kThreads) {
    L.cw[j] = make_int2(0, 0);
    L.ab[j] = make_int2(0, 0);
    L.tap[j] = 0;
    L.coef[j] = 0.f;
  }
  if (t < K) {
    double rh, rw;
    fin = tap_real(th, K, t, &rh, &rw);
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
    int j = base;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (cf[s] != 0.0) {
        const int a = P.sign * (h0 + (s >> 1)), b = P.sign * (w0 + (s & 1));
        const float wc = fin ? (float)((double)wk * cf[s]) : __builtin_nanf("");
        L.cw[j] = make_int2((a * P.TCm + b) * P.NI * 4, __float_as_int(wc));
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

// A zero tile (its margins stay zero for every item; staging writes the
// plane).  The barriers of build_cells order it before staging.
__device__ __forceinline__ void prepare(const Params& P, const Lds& L) {
  float4* t4 = reinterpret_cast<float4*>(L.tile);
  const int n4 = (P.TRm * P.TCm + P.mc) * P.NI / 4;
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
  const int r = a - __mul24(q, b);
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

// A lane's share of copying image-major data: image img = tid mod NI (the
// work-item stride, kThreads, is a multiple of NI, so a lane keeps its image)
// and chunks tid / NI + k (kThreads / NI) of V elements of that image's plane.
struct Share {
  int img, ch0, step;
  __device__ __forceinline__ explicit Share(const Params& P) {
    img = threadIdx.x & (P.NI - 1);
    ch0 = threadIdx.x >> P.lni;
    step = kThreads >> P.lni;
  }
};

// chunks per lane loaded before any is written: 16 elements (8 single ones)
template <int V>
constexpr int batch() {
  return V == 1 ? 8 : 16 / V;
}

// Work item i: channel c, image group `chunk` (images n0 .. n0 + ng - 1).
// Items of one channel are consecutive.
struct Item {
  int c, chunk, n0, ng;
  __device__ __forceinline__ Item(const Params& P, int i) {
    c = i / P.nchunk;
    chunk = i - c * P.nchunk;
    n0 = chunk * P.NI;
    ng = min(P.NI, P.N - n0);
  }
};

// A lane's loads of one item's plane of E elements (channel c, images n0 ..
// n0 + ng - 1) in chunks of V: the first `batch` chunks are held in
// registers from `issue` to `commit` (a 32-bit offset from a wave-uniform
// base keeps one register per address).
template <typename T, int V>
struct PlaneLoad {
  static constexpr int B = batch<V>();
  using VT = typename VecT<T, V>::type;
  VT v[B];  // packed as loaded (two bfloat16 per register)
  const T* base;
  int off, nch;  // off < 0: the lane has no image
  int c0;        // the lane's first chunk

  __device__ __forceinline__ void issue(const Params& P, const Share& sh, const T* src, const Item& it, int E) {
    base = src + ((size_t)it.n0 * P.C + it.c) * E;
    off = sh.img < it.ng ? sh.img * P.C * E : -1;
    nch = E / V;
    c0 = sh.ch0;
    load(sh, 0);
  }
  __device__ __forceinline__ void load(const Share& sh, int k0) {
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int ch = c0 + (k0 + u) * sh.step;
      if (off >= 0 && ch < nch)
        v[u] = *reinterpret_cast<const VT*>(reinterpret_cast<const char*>(base) +
                                            (unsigned)((off + ch * V) * (int)sizeof(T)));
    }
  }
  __device__ __forceinline__ T elem(int u, int e) const {
    T t[V];
    __builtin_memcpy(t, &v[u], sizeof(VT));
    return t[e];
  }
  __device__ __forceinline__ int batches(const Share& sh) const { return ((nch + sh.step - 1) / sh.step + B - 1) / B; }

  // The staged plane (SH x SW, V dividing SW) into the tile: element (i, j)
  // at frame position (i dil, j dil); a lane without an image writes zeros
  // (its slots may hold an earlier item's values).  The LDS writes of a wave
  // go to consecutive words (consecutive images).
  __device__ __forceinline__ void commit_tile_batch(const Params& P, const Share& sh, int k0, float* tile) const {
    const int cpr = P.SW / V;  // chunks per row
    const float rcpr = 1.f / (float)cpr;
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int ch = c0 + (k0 + u) * sh.step;
      if (ch < nch) {
        const int row = fdiv(ch, cpr, rcpr), col = (ch - __mul24(row, cpr)) * V;
        float* t = tile + ((__mul24(__mul24(row, P.dil) + P.mr, P.TCm) + __mul24(col, P.dil) + P.mc) << P.lni) + sh.img;
#pragma unroll
        for (int e = 0; e < V; ++e) t[__mul24(e, P.dil) << P.lni] = off >= 0 ? to_f32(elem(u, e)) : 0.f;
      }
    }
  }
  __device__ __forceinline__ void commit_tile(const Params& P, const Share& sh, float* tile) {
    commit_tile_batch(P, sh, 0, tile);
    for (int k0 = B; k0 < batches(sh) * B; k0 += B) {
      load(sh, k0);
      commit_tile_batch(P, sh, k0, tile);
    }
  }

  // An output-shaped plane into aux[image OSz + element], unconverted.
  __device__ __forceinline__ void commit_aux_batch(const Params& P, const Share& sh, int k0, T* aux) const {
    if (off < 0) return;
    T* a = aux + sh.img * P.OSz;
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int ch = c0 + (k0 + u) * sh.step;
      if (ch < nch) {
#pragma unroll
        for (int e = 0; e < V; ++e) a[ch * V + e] = elem(u, e);
      }
    }
  }
  __device__ __forceinline__ void commit_aux(const Params& P, const Share& sh, T* aux) {
    commit_aux_batch(P, sh, 0, aux);
    for (int k0 = B; k0 < batches(sh) * B; k0 += B) {
      load(sh, k0);
      commit_aux_batch(P, sh, k0, aux);
    }
  }
};

// Thread k's tap weight of channel c (0 past the taps, or without weights).
// Loaded before the plane's loads, so that the cell tables wait for this
// load only: vector loads complete in order.
template <typename T>
__device__ __forceinline__ float tap_weight(const Params& P, const T* __restrict__ wgt, int c) {
  return wgt && (int)threadIdx.x < P.K ? to_f32(wgt[(size_t)c * P.K + threadIdx.x]) : 0.f;
}

// The cell tables (and their runs) of one channel from its angle th and
// thread k's tap weight wk, into slot 0.  Barriers inside; the caller orders
// the runs before their use.
__device__ __forceinline__ void tables(const Params& P, Lds& L, float th, float wk) {
  L.use(P, 0);
  build_cells(P, L, th, wk);
  cell_runs(P, L);
}

// The output-shaped tile's images of item `it` to channel c of dst.
template <typename T, int V>
__device__ __forceinline__ void store_aux_v(const Params& P, T* __restrict__ dst, const Item& it, const T* aux) {
  const Share sh(P);
  if (sh.img >= it.ng) return;
  const int E = P.OH * P.OW, nch = E / V;
  T* base = dst + ((size_t)it.n0 * P.C + it.c) * E;
  const int off = sh.img * P.C * E;
  const T* a = aux + sh.img * P.OSz;
  for (int ch = sh.ch0; ch < nch; ch += sh.step) {
    T v[V];
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = a[ch * V + e];
    store_raw<T, V>(reinterpret_cast<T*>(reinterpret_cast<char*>(base) + (unsigned)((off + ch * V) * (int)sizeof(T))), v);
  }
}

template <typename T>
__device__ __forceinline__ void store_aux(const Params& P, T* __restrict__ dst, const Item& it, const T* aux) {
  if (P.va == 4)
    store_aux_v<T, 4>(P, dst, it, aux);
  else if (P.va == 2)
    store_aux_v<T, 2>(P, dst, it, aux);
  else
    store_aux_v<T, 1>(P, dst, it, aux);
}

// A lane's place: images img, img + 1 of the workgroup, column r of its group.
struct Lane {
  int img, r;
  __device__ __forceinline__ explicit Lane(const Params& P) {
    const int l = threadIdx.x & 63;
    img = 2 * (l & (P.NI / 2 - 1));
    r = l >> (P.lni - 1);
  }
};

// Group `g`: its first output row p0, the lane's output column q, the cell
// run [lo, hi) (uniform) and the lane's tile byte address at cell offset 0.
struct Group {
  int p0, q, lo, hi;
  const unsigned char* tb;
  __device__ __forceinline__ Group(const Params& P, const Lds& L, const Lane& ln, int g, int RP) {
    const int rg = g / P.ncg, cg = g - rg * P.ncg;
    const int2 a = L.rr[rg], b = L.cc[cg];
    lo = __builtin_amdgcn_readfirstlane(max(a.x, b.x));
    hi = __builtin_amdgcn_readfirstlane(min(a.y, b.y));
    p0 = rg * RP;
    q = cg * P.R + ln.r;
    tb = reinterpret_cast<const unsigned char*>(
        L.tile + ((__mul24(__mul24(p0, P.sig) + P.mr, P.TCm) + __mul24(q, P.sig) + P.mc) << P.lni) + ln.img);
  }
};

// ---------------------------------------------------------------- gather

// The gather of one item from the staged tile into the output-shaped tile:
// out[p,q] = sum over the channel's cells of weight * frame[sig p + a, sig q + b].
template <typename T, int RP>
__device__ __forceinline__ void gather_item(const Params& P, const Lds& L, T* aux) {
  const Lane ln(P);
  const int rsb = P.sig * P.TCm * P.NI * 4;  // bytes per output row
  for (int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); g < P.nitems; g += kWaves) {
    const Group gr(P, L, ln, g, RP);
    const unsigned char* tr[RP];  // the lane's row addresses at cell offset 0
#pragma unroll
    for (int i = 0; i < RP; ++i) tr[i] = gr.tb + i * rsb;
    float2 acc[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) acc[i] = make_float2(0.f, 0.f);
    // four cells per step (their table entries read together, then their
    // tile reads together)
    int t = gr.lo;
    for (; t + 4 <= gr.hi; t += 4) {
      int2 cl[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) cl[u] = L.cw[t + u];
      float2 v[4][RP];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int i = 0; i < RP; ++i) v[u][i] = *reinterpret_cast<const float2*>(tr[i] + cl[u].x);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float wc = __int_as_float(cl[u].y);
#pragma unroll
        for (int i = 0; i < RP; ++i) {
          acc[i].x = fmaf(wc, v[u][i].x, acc[i].x);
          acc[i].y = fmaf(wc, v[u][i].y, acc[i].y);
        }
      }
    }
    for (; t < gr.hi; ++t) {
      const int2 cl = L.cw[t];
      const float wc = __int_as_float(cl.y);
#pragma unroll
      for (int i = 0; i < RP; ++i) {
        const float2 v = *reinterpret_cast<const float2*>(tr[i] + cl.x);
        acc[i].x = fmaf(wc, v.x, acc[i].x);
        acc[i].y = fmaf(wc, v.y, acc[i].y);
      }
    }
    if (gr.q < P.OW) {
      T* ax = aux + ln.img * P.OSz + gr.q;
#pragma unroll
      for (int i = 0; i < RP; ++i)
        if (gr.p0 + i < P.OH) {
          ax[(gr.p0 + i) * P.OW] = from_f32<T>(acc[i].x);
          ax[P.OSz + (gr.p0 + i) * P.OW] = from_f32<T>(acc[i].y);
        }
    }
  }
}

// The forward pass (x, cells at +(a, b)) and the input gradient (dy on the
// stride lattice, cells at -(a, b), sig 1) of work item blockIdx.x.  The
// plane's loads are issued first; the tile is cleared and the cells are
// built while they are in flight.
template <typename T, int RP, int V>
__device__ __forceinline__ void gather_one(const Params& P, Lds& L, const T* __restrict__ in,
                                           const T* __restrict__ wgt, const float* __restrict__ theta,
                                           T* __restrict__ out) {
  const Share sh(P);
  const Item it(P, blockIdx.x);
  T* aux = reinterpret_cast<T*>(L.aux);
  const float th = theta[it.c];
  const float wk = tap_weight<T>(P, wgt, it.c);
  PlaneLoad<T, V> pl;
  pl.issue(P, sh, in, it, P.SH * P.SW);
  prepare(P, L);
  tables(P, L, th, wk);
  pl.commit_tile(P, sh, L.tile);
  __syncthreads();
  gather_item<T, RP>(P, L, aux);
  __syncthreads();
  store_aux<T>(P, out, it, aux);
}

template <typename T, int RP>
__global__ __launch_bounds__(kThreads) void plane_gather(Params P, const T* __restrict__ in,
                                                         const T* __restrict__ wgt, const float* __restrict__ theta,
                                                         T* __restrict__ out) {
  extern __shared__ __align__(16) unsigned char smem[];
  Lds L(smem, P);
  if (P.vt == 4)
    gather_one<T, RP, 4>(P, L, in, wgt, theta, out);
  else if (P.vt == 2)
    gather_one<T, RP, 2>(P, L, in, wgt, theta, out);
  else
    gather_one<T, RP, 1>(P, L, in, wgt, theta, out);
}

// ---------------------------------------------------------------- weight gradients

// Cells J of the group of KB (table cw) taken four at a time; a cell of the
// four outside the run [lo, hi) reads the lane's own tile words (inside the
// tile) and counts for nothing.  f(J, in, weight, v[RP]) consumes a cell (v:
// the lane's two images at its RP rows).
template <int RP, int KB, class F>
__device__ __forceinline__ void each_cell(const int2* cw, int lo, int hi, const unsigned char* tb, int rsb, F&& f) {
  static_for<KB / 4>([&](auto g) __attribute__((always_inline)) {
    constexpr int J0 = 4 * decltype(g)::value;
    if (J0 + 4 > lo && J0 < hi) {
      const int4* c4 = reinterpret_cast<const int4*>(cw + J0);
      const int4 a = c4[0], b = c4[1];
      const int off[4] = {a.x, a.z, b.x, b.z};
      const int wb[4] = {a.y, a.w, b.y, b.w};
      float2 v[4][RP];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool in = J0 + u >= lo && J0 + u < hi;
        const int o = in ? off[u] : 0;
#pragma unroll
        for (int i = 0; i < RP; ++i) v[u][i] = *reinterpret_cast<const float2*>(tb + o + i * rsb);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) f(J0 + u, J0 + u >= lo && J0 + u < hi, __int_as_float(wb[u]), v[u]);
    }
  });
}

// Adds the workgroup's per-cell sums (cells j0 .. j0 + KB - 1 of the
// channel, in acc of every lane) times their coefficients to the per-tap sums
// dwacc[k]: thread k folds the cells of tap k (a contiguous run) in order.
// acc is consumed.
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

// The item's partial row of the weight gradient, then dwacc cleared.
__device__ __forceinline__ void write_partial(const Params& P, const Item& it, const float* __restrict__ theta,
                                              float* dwacc, float* __restrict__ partial) {
  const bool fin = isfinite(theta[it.c]);
  for (int k = threadIdx.x; k < P.K; k += kThreads) {
    partial[((size_t)it.chunk * P.C + it.c) * P.K + k] = fin ? dwacc[k] : __builtin_nanf("");
    dwacc[k] = 0.f;
  }
}

// The lane's two images' values of an output-shaped tile at its outputs
// (zero past the plane and for images past N).
template <typename T, int RP>
__device__ __forceinline__ void lane_values(const Params& P, const Lane& ln, const Group& gr, const T* ax, int ng,
                                            float2 (&d)[RP]) {
#pragma unroll
  for (int i = 0; i < RP; ++i) {
    const bool ok = gr.q < P.OW && gr.p0 + i < P.OH;
    d[i].x = ok && ln.img < ng ? to_f32(ax[(gr.p0 + i) * P.OW]) : 0.f;
    d[i].y = ok && ln.img + 1 < ng ? to_f32(ax[P.OSz + (gr.p0 + i) * P.OW]) : 0.f;
  }
}

// The weight-gradient sums of one item into dwacc.
template <typename T, int RP, int KB>
__device__ __forceinline__ void wgrad_item(const Params& P, const Lds& L, const T* aux, int ng, float* dwacc) {
  const Lane ln(P);
  const int rsb = P.sig * P.TCm * P.NI * 4;
  const int n = __builtin_amdgcn_readfirstlane(L.first[P.K]);
  for (int j0 = 0; j0 < n; j0 += KB) {
    float acc[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) acc[j] = 0.f;
    for (int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); g < P.nitems; g += kWaves) {
      const Group gr(P, L, ln, g, RP);
      const int lo = max(gr.lo, j0) - j0, hi = min(gr.hi, j0 + KB) - j0;
      if (lo >= hi) continue;
      float2 d[RP];
      lane_values<T, RP>(P, ln, gr, aux + ln.img * P.OSz + gr.q, ng, d);
      each_cell<RP, KB>(L.cw + j0, lo, hi, gr.tb, rsb,
                        [&](int J, bool in, float, const float2 (&v)[RP]) __attribute__((always_inline)) {
                          float s = 0.f;
#pragma unroll
                          for (int i = 0; i < RP; ++i) s = fmaf(d[i].y, v[i].y, fmaf(d[i].x, v[i].x, s));
                          acc[J] += in ? s : 0.f;
                        });
    }
    fold_cells<KB>(P, L, acc, j0, dwacc);
  }
}

// partial[(chunk C + c) K + k] = sum over the item's images and outputs of
// dy[p,q] * sum over the cells of tap k of coef x[sig p + a, sig q + b]
// (Eq. 1 differentiated in w_k).  One item per workgroup; the tile holds x,
// the output-shaped tile dy.
template <typename T, int RP, int KB>
__global__ __launch_bounds__(kThreads) void plane_wgrad(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                        const float* __restrict__ theta,
                                                        float* __restrict__ partial) {
  extern __shared__ __align__(16) unsigned char smem[];
  Lds L(smem, P);
  const Share sh(P);
  float* dwacc = L.red + kWaves * KB;
  T* aux = reinterpret_cast<T*>(L.aux);
  for (int k = threadIdx.x; k < P.K; k += kThreads) dwacc[k] = 0.f;
  prepare(P, L);
  {
    const Item it(P, blockIdx.x);
    tables(P, L, theta[it.c], 0.f);
    if (P.vt == 4) {
      PlaneLoad<T, 4> pl;
      pl.issue(P, sh, x, it, P.SH * P.SW);
      pl.commit_tile(P, sh, L.tile);
    } else if (P.vt == 2) {
      PlaneLoad<T, 2> pl;
      pl.issue(P, sh, x, it, P.SH * P.SW);
      pl.commit_tile(P, sh, L.tile);
    } else {
      PlaneLoad<T, 1> pl;
      pl.issue(P, sh, x, it, P.SH * P.SW);
      pl.commit_tile(P, sh, L.tile);
    }
    if (P.va == 4) {
      PlaneLoad<T, 4> pa;
      pa.issue(P, sh, dy, it, P.OH * P.OW);
      pa.commit_aux(P, sh, aux);
    } else if (P.va == 2) {
      PlaneLoad<T, 2> pa;
      pa.issue(P, sh, dy, it, P.OH * P.OW);
      pa.commit_aux(P, sh, aux);
    } else {
      PlaneLoad<T, 1> pa;
      pa.issue(P, sh, dy, it, P.OH * P.OW);
      pa.commit_aux(P, sh, aux);
    }
    __syncthreads();
    wgrad_item<T, RP, KB>(P, L, aux, it.ng, dwacc);
    write_partial(P, it, theta, dwacc, partial);
  }
}

// Both gradients of one item in one pass (stride 1, rounded-down offsets):
// the tile holds dy, the output-shaped tile x.  Per mirrored cell every dy
// value v read for the lane's input-gradient outputs h adds w_c v to dx[h]
// and x[h] v to the cell's sum, which is the weight gradient of the cell's
// tap: dw_k = sum_h x[h] dy[h - off_k].  dx replaces x in the output-shaped
// tile (each output is read and written by one lane only).
template <typename T, int RP, int KB>
__device__ __forceinline__ void bwd_item(const Params& P, const Lds& L, T* aux, int ng, float* dwacc) {
  const Lane ln(P);
  const int rsb = P.TCm * P.NI * 4;
  float acc[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) acc[j] = 0.f;
  for (int g = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); g < P.nitems; g += kWaves) {
    const Group gr(P, L, ln, g, RP);
    T* ax = aux + ln.img * P.OSz + gr.q;
    float2 xv[RP], o[RP];
    lane_values<T, RP>(P, ln, gr, ax, ng, xv);
#pragma unroll
    for (int i = 0; i < RP; ++i) o[i] = make_float2(0.f, 0.f);
    each_cell<RP, KB>(L.cw, gr.lo, gr.hi, gr.tb, rsb,
                      [&](int J, bool in, float wc, const float2 (&v)[RP]) __attribute__((always_inline)) {
                        const float we = in ? wc : 0.f;
                        float s = 0.f;
#pragma unroll
                        for (int i = 0; i < RP; ++i) {
                          o[i].x = fmaf(we, v[i].x, o[i].x);
                          o[i].y = fmaf(we, v[i].y, o[i].y);
                          s = fmaf(xv[i].y, v[i].y, fmaf(xv[i].x, v[i].x, s));
                        }
                        acc[J] += in ? s : 0.f;
                      });
    if (gr.q < P.OW) {
#pragma unroll
      for (int i = 0; i < RP; ++i)
        if (gr.p0 + i < P.OH) {
          ax[(gr.p0 + i) * P.OW] = from_f32<T>(o[i].x);
          ax[P.OSz + (gr.p0 + i) * P.OW] = from_f32<T>(o[i].y);
        }
    }
  }
  fold_cells<KB>(P, L, acc, 0, dwacc);  // its barriers also end the item's reads of both tiles
}

template <typename T, int RP, int KB, int V>
__device__ __forceinline__ void bwd_one(const Params& P, Lds& L, const T* __restrict__ x, const T* __restrict__ dy,
                                        const T* __restrict__ wgt, const float* __restrict__ theta,
                                        T* __restrict__ dx, float* __restrict__ partial) {
  const Share sh(P);
  const Item it(P, blockIdx.x);
  const int E = P.H * P.W;  // dy, x and dx share the plane (stride 1)
  T* aux = reinterpret_cast<T*>(L.aux);
  float* dwacc = L.red + kWaves * KB;
  for (int k = threadIdx.x; k < P.K; k += kThreads) dwacc[k] = 0.f;
  const float th = theta[it.c];
  const float wk = tap_weight<T>(P, wgt, it.c);
  PlaneLoad<T, V> pd, px;
  pd.issue(P, sh, dy, it, E);
  px.issue(P, sh, x, it, E);
  prepare(P, L);
  tables(P, L, th, wk);
  pd.commit_tile(P, sh, L.tile);
  px.commit_aux(P, sh, aux);
  __syncthreads();
  bwd_item<T, RP, KB>(P, L, aux, it.ng, dwacc);
  store_aux<T>(P, dx, it, aux);
  write_partial(P, it, theta, dwacc, partial);
}

template <typename T, int RP, int KB>
__global__ __launch_bounds__(kThreads) void plane_bwd(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                      const T* __restrict__ wgt, const float* __restrict__ theta,
                                                      T* __restrict__ dx, float* __restrict__ partial) {
  extern __shared__ __align__(16) unsigned char smem[];
  Lds L(smem, P);
  if (P.vt == 4)
    bwd_one<T, RP, KB, 4>(P, L, x, dy, wgt, theta, dx, partial);
  else if (P.vt == 2)
    bwd_one<T, RP, KB, 2>(P, L, x, dy, wgt, theta, dx, partial);
  else
    bwd_one<T, RP, KB, 1>(P, L, x, dy, wgt, theta, dx, partial);
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

// Four rows per lane only with up to 64 per-cell sums (the plan's rule).
template <typename T>
hipError_t bwd_t(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx, void* dw,
                 float* partial, hipStream_t stream) {
  if (pl.p.RP == 4) {
    if (pl.p.KB == 32) return bwd_launch<T, 4, 32>(pl, x, dy, w, theta, dx, dw, partial, stream);
    if (pl.p.KB == 64) return bwd_launch<T, 4, 64>(pl, x, dy, w, theta, dx, dw, partial, stream);
    return hipErrorInvalidValue;
  }
  if (pl.p.KB == 32) return bwd_launch<T, 2, 32>(pl, x, dy, w, theta, dx, dw, partial, stream);
  if (pl.p.KB == 64) return bwd_launch<T, 2, 64>(pl, x, dy, w, theta, dx, dw, partial, stream);
  return bwd_launch<T, 2, 128>(pl, x, dy, w, theta, dx, dw, partial, stream);
}

}  // namespace
}  // namespace plane
}  // namespace o1d
