// Run-decomposed kernels for depthwise convolution with oriented 1D kernels.
//
// For one channel every output reads the same K cells of a digital line
// (Eq. 2).  Consecutive cells of that line step by one pixel vertically,
// horizontally or diagonally, and stretches of the line repeat the same step
// ("runs").  If a lane computes R = 7 outputs that are themselves spaced by
// the run's step u, the R x L products of a run of length L need only
// R + L - 1 distinct LDS values instead of R * L.  This register reuse is
// what lets the oriented gather run at the cost of a horizontal one: LDS
// reads, not multiply-adds, are the scarce resource on gfx950 (a wave-wide
// 32-bit LDS read costs about 2.5 clocks per CU against 1 clock for a
// wave-wide FMA spread over the four SIMDs).
//
// Per channel, wave 0 of the workgroup builds a small program in LDS (one
// tap per lane, ballots and shuffles): the cells (duplicate taps merged,
// weights summed), the staging frame (the plane is staged transposed when
// the line is closer to horizontal, so every line becomes closer to
// vertical), the strip direction u = (1, s) with s in {-1, 0, +1} (the most
// frequent cell-to-cell step), and the runs along u (at most kLmax cells per
// piece) with their LDS offsets and weights.  The plane is staged in LDS
// with a zero halo, so the tap loop has no bounds checks.  The tile row
// stride S is a compile-time constant, so each load of a run uses an
// immediate offset m * (S + s); the host picks S so that the 64 lanes of a
// wave-tile hit 64 distinct LDS banks.
//
// The forward pass and the input gradient share the gather kernel (the
// gradient gathers dy through the negated cells).  The weight gradient walks
// the plane's own strips, keeps one register partial sum per distinct cell
// and reduces them in a fixed order (no atomics).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_launch.h"
#include "o1d_runs.h"

namespace o1d {
namespace runs {
namespace {

// ---------------------------------------------------------------- program

struct Prog {
  int nruns;
  int ncells;
  int s;           // strip direction u = (1, s) in the staging frame
  int transposed;  // staging frame = transposed plane
  int finite;      // the channel's angle is finite
  int pad_[3];
  int group[8];            // runs of length L occupy [group[L-1], group[L]) (group[0] = 0)
  int run_off[kMaxRuns];   // LDS offset of the run's first cell (along +u) from the output pixel
  int cell_off[kMaxTaps];  // LDS offset of every distinct cell (cell order)
  int tap_cell[kMaxTaps];  // cell of every tap (duplicate taps share one)
  int pad2_[64];
  float run_w[kMaxRuns * 8];
};
static_assert(sizeof(Prog) == kProgBytes, "kProgBytes must match the program layout");
static_assert(sizeof(Prog) % 16 == 0, "the program must keep the tile 16-byte aligned");
constexpr int kProgDwords = (int)(sizeof(Prog) / 4);

__device__ __forceinline__ int wave_min_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = min(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = max(v, __shfl_xor(v, m, 64));
  return v;
}
// lanes strictly below lane n (n in [0, 64])
__device__ __forceinline__ uint64_t below_mask(int n) { return n <= 0 ? 0ull : (n >= 64 ? ~0ull : (~0ull >> (64 - n))); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int hibit(uint64_t m) { return 63 - __clzll(m); }
__device__ __forceinline__ int lobit(uint64_t m) { return __ffsll((long long)m) - 1; }

// Builds the channel's program; called by all 64 lanes of wave 0 (K <= 63).
// `sign` = -1 negates the cells (input gradient); `allow_transpose` = false
// keeps the plane's own frame (the weight gradient does not use runs).
template <typename T, int S>
__device__ void build_program(Prog* pg, const T* __restrict__ wgt, float theta, int c, int K, int sign,
                              bool allow_transpose) {
  const int k = threadIdx.x;
  const bool act = k < K;
  int dh = 0, dw = 0;
  bool fin = true;
  float wk = 0.f;
  if (act) {
    fin = tap_offset(theta, K, k, &dh, &dw);
    dh *= sign;
    dw *= sign;
    if (wgt) wk = to_f32(wgt[(size_t)c * K + k]);
  }
  const int hmin = wave_min_i(act ? dh : 1 << 20), hmax = wave_max_i(act ? dh : -(1 << 20));
  const int wmin = wave_min_i(act ? dw : 1 << 20), wmax = wave_max_i(act ? dw : -(1 << 20));
  const bool tr = allow_transpose && (wmax - wmin) > (hmax - hmin);
  const int a = tr ? dw : dh;  // staging-frame row offset of the tap
  const int b = tr ? dh : dw;  // staging-frame column offset

  // Consecutive taps on the same pixel are merged (they come at most in pairs
  // because max(|sin|, |cos|) >= 1/sqrt(2)); the first of a pair carries the sum.
  const int pa = __shfl_up(a, 1, 64), pb = __shfl_up(b, 1, 64);
  const bool dup = act && k > 0 && pa == a && pb == b;
  const uint64_t dupm = __ballot(dup);
  const float nw = __shfl_down(wk, 1, 64);
  const bool next_dup = k < 63 && ((dupm >> (k + 1)) & 1ull);
  const float cw = wk + (next_dup ? nw : 0.f);
  const bool cell = act && !dup;
  const uint64_t cellm = __ballot(cell);
  const uint64_t below = below_mask(k), upto = below | (1ull << k);
  const int ci = popc(cellm & below);
  const int ncells = popc(cellm);

  // Step from the previous cell, normalised so that rows increase.
  const int prev = (k >= 1 && ((dupm >> (k - 1)) & 1ull)) ? k - 2 : k - 1;
  const int ppa = __shfl(a, prev < 0 ? 0 : prev, 64), ppb = __shfl(b, prev < 0 ? 0 : prev, 64);
  const int a_first = __shfl(a, 0, 64), a_last = __shfl(a, K - 1, 64);
  const int sg = (a_last >= a_first) ? 1 : -1;  // rows move monotonically with k
  const int da = (a - ppa) * sg, db = (b - ppb) * sg;
  const bool has_step = cell && ci > 0;
  const int n0 = popc(__ballot(has_step && da == 1 && db == 0));
  const int np = popc(__ballot(has_step && da == 1 && db == 1));
  const int nm = popc(__ballot(has_step && da == 1 && db == -1));
  int s = 0;
  if (np > n0 && np >= nm) s = 1;
  else if (nm > n0 && nm > np) s = -1;

  // Runs: a cell starts a run unless it steps by exactly +u from the previous
  // cell; runs are then cut into pieces of at most kLmax cells.
  const bool cont = has_step && da == 1 && db == s;
  const uint64_t startm = __ballot(cell && !cont);
  const int st = hibit((startm & upto) | 1ull);
  const int pos = ci - popc(cellm & below_mask(st));
  const uint64_t start2 = __ballot(cell && (pos % kLmax) == 0);
  const int st2 = hibit((start2 & upto) | 1ull);
  const int ci_st2 = popc(cellm & below_mask(st2));
  const int pos2 = ci - ci_st2;
  const int run = popc(start2 & upto) - 1;
  const uint64_t later = start2 & ~upto;
  const int nxt = later ? lobit(later) : 64;
  const int L = popc(cellm & below_mask(nxt)) - ci_st2;
  const int t = (sg > 0) ? pos2 : (L - 1 - pos2);  // position along +u
  const bool allfin = popc(__ballot(act && !fin)) == 0;

  // Runs are stored grouped by length so the kernels can run one tight loop
  // per length: run `run` goes to slot group_start(L) + rank among runs of length L.
  const bool is_start = cell && ((start2 >> k) & 1ull);
  int rstart = 0, rslot = 0;
  for (int l = 1; l <= kLmax; ++l) {
    const uint64_t m = __ballot(is_start && L == l);
    if (is_start && L == l) rslot = rstart + popc(m & below);
    if (k == 0) pg->group[l - 1] = rstart;
    rstart += popc(m);
  }
  if (k == 0) pg->group[kLmax] = rstart;
  // the slot of a cell's run, read from the run's start lane
  const int my_slot = __shfl(rslot, st2, 64);

  // (the index checks below never fail for a well-formed program; they keep
  // every LDS write inside its array whatever the inputs)
  if (cell && my_slot >= 0 && my_slot < kMaxRuns && t >= 0 && t < 8 && L >= 1 && L <= kLmax) {
    pg->run_w[my_slot * 8 + t] = allfin ? cw : __builtin_nanf("");  // a non-finite angle poisons the channel
    if (t == 0) pg->run_off[my_slot] = a * S + b;
  }
  if (cell && ci >= 0 && ci < kMaxTaps) pg->cell_off[ci] = a * S + b;
  const int tcell = __shfl(ci, dup ? k - 1 : k, 64);
  if (act) pg->tap_cell[k] = (tcell >= 0 && tcell < K) ? tcell : 0;
  if (k == 0) {
    pg->nruns = popc(start2);
    pg->ncells = ncells;
    pg->s = s;
    pg->transposed = tr ? 1 : 0;
    pg->finite = allfin ? 1 : 0;
  }
  (void)run;
}

// ---------------------------------------------------------------- strips

// Lane geometry of one wave-tile: RB bands x CB columns of strips.
struct Strip {
  int g;     // plane slot within the group
  int band;  // strip rows band*R .. band*R + R - 1
  int j;     // column of the strip's first output (staging frame)
};

__device__ __forceinline__ Strip strip_of(int wt, int lane, int RB, int CB, int nb_tiles, int nc_tiles, int jlo) {
  Strip sp;
  const int per_plane = nb_tiles * nc_tiles;
  sp.g = wt / per_plane;
  const int rem = wt - sp.g * per_plane;
  const int tb = rem / nc_tiles;
  const int tc = rem - tb * nc_tiles;
  const int rb = lane / CB;
  const int cb = lane - rb * CB;
  sp.band = tb * RB + rb;
  sp.j = jlo + tc * CB + cb;
  return sp;
}

// All runs of length L along u = (1, SD): acc[i] += w[t] * V[i + t], V[m] = p[m * (S + SD)].
template <int S, int SD, int L>
__device__ __forceinline__ void run_group(const Prog* __restrict__ pg, const float* __restrict__ base, int r0, int r1,
                                          float (&acc)[kR]) {
  for (int r = r0; r < r1; ++r) {
    const float* p = base + pg->run_off[r];
    const float4 wa = *reinterpret_cast<const float4*>(&pg->run_w[r * 8]);
    float4 wb = wa;
    if (L > 4) wb = *reinterpret_cast<const float4*>(&pg->run_w[r * 8 + 4]);
    const float w[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
    constexpr int M = kR + L - 1;
    float v[M];
#pragma unroll
    for (int m = 0; m < M; ++m) v[m] = p[m * (S + SD)];
#pragma unroll
    for (int t = 0; t < L; ++t)
#pragma unroll
      for (int i = 0; i < kR; ++i) acc[i] = fmaf(w[t], v[i + t], acc[i]);
  }
}

template <int S, int SD>
__device__ __forceinline__ void strip_gather(const Prog* __restrict__ pg, const int (&grp)[kLmax + 1],
                                             const float* __restrict__ base, float (&acc)[kR]) {
  run_group<S, SD, 1>(pg, base, grp[0], grp[1], acc);
  run_group<S, SD, 2>(pg, base, grp[1], grp[2], acc);
  run_group<S, SD, 3>(pg, base, grp[2], grp[3], acc);
  run_group<S, SD, 4>(pg, base, grp[3], grp[4], acc);
  run_group<S, SD, 5>(pg, base, grp[4], grp[5], acc);
  run_group<S, SD, 6>(pg, base, grp[5], grp[6], acc);
  run_group<S, SD, 7>(pg, base, grp[6], grp[7], acc);
}

// Channel-level geometry shared by both kernels.
struct Frame {
  int tr, s, Hs, Ws, nb, nj, jlo, nb_tiles, nc_tiles, tiles;
};

__device__ __forceinline__ Frame frame_of(const Prog* pg, const RunsParams& P) {
  Frame f;
  f.tr = pg->transposed;
  f.s = pg->s;
  f.Hs = f.tr ? P.W : P.H;
  f.Ws = f.tr ? P.H : P.W;
  f.nb = (f.Hs + kR - 1) / kR;
  f.nj = f.Ws + (f.s != 0 ? kR - 1 : 0);
  f.jlo = (f.s > 0) ? -(kR - 1) : 0;
  f.nb_tiles = (f.nb + P.RB - 1) / P.RB;
  f.nc_tiles = (f.nj + P.CB - 1) / P.CB;
  f.tiles = P.G * f.nb_tiles * f.nc_tiles;
  return f;
}

// Per-thread staging slots of one group of G planes: source offset (from the
// group's first plane of this channel) and LDS destination in the staging frame.
template <int S>
__device__ __forceinline__ void staging_slots(const RunsParams& P, const Frame& f, int (&src)[kMaxStage],
                                              int (&dst)[kMaxStage], int (&cmp)[kMaxStage], int (&gq)[kMaxStage]) {
  const int HW = P.H * P.W;
  const int gel = P.G * HW;
#pragma unroll
  for (int q = 0; q < kMaxStage; ++q) {
    const int e = threadIdx.x + q * (int)blockDim.x;
    src[q] = -1;
    dst[q] = 0;
    cmp[q] = 0;
    gq[q] = 0;
    if (e < gel) {
      const int g = e / HW;
      const int rem = e - g * HW;
      const int h = rem / P.W;
      const int w = rem - h * P.W;
      const int rs = f.tr ? w : h, cs = f.tr ? h : w;
      src[q] = g * P.C * HW + rem;
      dst[q] = g * P.PS + (rs + P.RT) * S + cs;
      cmp[q] = g * HW + rs * f.Ws + cs;
      gq[q] = g;
    }
  }
}

// ---------------------------------------------------------------- forward / input gradient

template <typename T, int S>
__global__ __launch_bounds__(kThreads2) void gather_runs(RunsParams P, const T* __restrict__ in,
                                                         const T* __restrict__ wgt, const float* __restrict__ theta,
                                                         T* __restrict__ out) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tile = smem + kProgDwords;
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nwaves = blockDim.x >> 6;
  const int HW = P.H * P.W;

  for (int i = tid; i < P.G * P.PS; i += blockDim.x) tile[i] = 0.f;  // halos and margins stay zero
  if (wave == 0) build_program<T, S>(pg, wgt, theta[c], c, P.K, P.sign, true);
  __syncthreads();
  const Frame f = frame_of(pg, P);
  int grp[kLmax + 1];
#pragma unroll
  for (int l = 0; l <= kLmax; ++l) grp[l] = min(__builtin_amdgcn_readfirstlane(pg->group[l]), kMaxRuns);
  int src[kMaxStage], dst[kMaxStage], cmp[kMaxStage], gq[kMaxStage];
  staging_slots<S>(P, f, src, dst, cmp, gq);

  const int n_begin = blockIdx.x * P.NPW;
  const int n_end = min(P.N, n_begin + P.NPW);
  const size_t cHW = (size_t)c * HW;
  float pre[kMaxStage];
  auto load_group = [&](int n0) {
    const T* sp = in + (size_t)n0 * P.C * HW + cHW;
#pragma unroll
    for (int q = 0; q < kMaxStage; ++q) {
      pre[q] = 0.f;
      if (src[q] >= 0 && n0 + gq[q] < n_end) pre[q] = to_f32(sp[src[q]]);
    }
  };
  load_group(n_begin);

  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    __syncthreads();  // the previous group is no longer read
#pragma unroll
    for (int q = 0; q < kMaxStage; ++q)
      if (src[q] >= 0) tile[dst[q]] = pre[q];
    __syncthreads();
    if (n0 + P.G < n_end) load_group(n0 + P.G);  // next group's loads fly behind this group's math

    for (int wt = wave; wt < f.tiles; wt += nwaves) {
      const Strip sp = strip_of(wt, lane, P.RB, P.CB, f.nb_tiles, f.nc_tiles, f.jlo);
      const int n = n0 + sp.g;
      const bool ok = sp.band < f.nb && sp.j - f.jlo < f.nj && n < n_end;
      const int b0 = sp.band * kR;
      // lanes outside the plane read a harmless in-tile address and store nothing
      const float* base = tile + (ok ? sp.g * P.PS + (b0 + P.RT) * S + sp.j : P.RT * S);
      float acc[kR];
#pragma unroll
      for (int i = 0; i < kR; ++i) acc[i] = 0.f;
      if (f.s == 0)
        strip_gather<S, 0>(pg, grp, base, acc);
      else if (f.s > 0)
        strip_gather<S, 1>(pg, grp, base, acc);
      else
        strip_gather<S, -1>(pg, grp, base, acc);
      if (ok) {
        T* o = out + ((size_t)n * P.C + c) * HW;
#pragma unroll
        for (int i = 0; i < kR; ++i) {
          const int rs = b0 + i, cs = sp.j + f.s * i;
          if (rs < f.Hs && cs >= 0 && cs < f.Ws) o[f.tr ? cs * P.W + rs : rs * P.W + cs] = from_f32<T>(acc[i]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- weight gradient

// The weight gradient keeps one register accumulator per distinct cell and
// lane (a static loop over the cells, so every accumulator index is a
// compile-time constant), reads the staged x through each cell's offset for
// the 7 outputs of the lane's strip and multiplies by the strip's dy.  No
// atomics: the lanes' sums are reduced once per workgroup at the end, in a
// fixed order, so the result is bitwise reproducible.
template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads2) void wgrad_runs(RunsParams P, const T* __restrict__ x, const T* __restrict__ dy,
                                                        const float* __restrict__ theta, float* __restrict__ partial) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  const int HW = P.H * P.W;
  float* red = smem + kProgDwords;  // [8 waves][64] per-wave cell sums
  float* gt = red + 8 * 64;         // dy, compact: [G][H][W]
  float* tile = gt + ((P.G * HW + 3) & ~3);
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nwaves = blockDim.x >> 6;

  for (int i = tid; i < P.G * P.PS; i += blockDim.x) tile[i] = 0.f;
  if (wave == 0) build_program<T, S>(pg, static_cast<const T*>(nullptr), theta[c], c, P.K, 1, false);
  __syncthreads();
  Frame f = frame_of(pg, P);  // plane frame (no transpose); vertical strips
  f.s = 0;
  f.nj = f.Ws;
  f.jlo = 0;
  f.nc_tiles = (f.nj + P.CB - 1) / P.CB;
  f.tiles = P.G * f.nb_tiles * f.nc_tiles;
  const int ncells = min(__builtin_amdgcn_readfirstlane(pg->ncells), KB);
  int src[kMaxStage], dst[kMaxStage], cmp[kMaxStage], gq[kMaxStage];
  staging_slots<S>(P, f, src, dst, cmp, gq);

  float acc[KB];
#pragma unroll
  for (int ci = 0; ci < KB; ++ci) acc[ci] = 0.f;

  const int n_begin = blockIdx.z * P.NPW;
  const int n_end = min(P.N, n_begin + P.NPW);
  const size_t cHW = (size_t)c * HW;
  float px[kMaxStage], pd[kMaxStage];
  auto load_group = [&](int n0) {
    const T* sx = x + (size_t)n0 * P.C * HW + cHW;
    const T* sd = dy + (size_t)n0 * P.C * HW + cHW;
#pragma unroll
    for (int q = 0; q < kMaxStage; ++q) {
      px[q] = 0.f;
      pd[q] = 0.f;
      if (src[q] >= 0 && n0 + gq[q] < n_end) {
        px[q] = to_f32(sx[src[q]]);
        pd[q] = to_f32(sd[src[q]]);
      }
    }
  };
  load_group(n_begin);

  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kMaxStage; ++q)
      if (src[q] >= 0) {
        tile[dst[q]] = px[q];
        gt[cmp[q]] = pd[q];
      }
    __syncthreads();
    if (n0 + P.G < n_end) load_group(n0 + P.G);

    for (int wt = wave; wt < f.tiles; wt += nwaves) {
      const Strip sp = strip_of(wt, lane, P.RB, P.CB, f.nb_tiles, f.nc_tiles, 0);
      const int n = n0 + sp.g;
      const bool ok = sp.band < f.nb && sp.j < f.Ws && n < n_end;
      const int b0 = sp.band * kR;
      const float* base = tile + (ok ? sp.g * P.PS + (b0 + P.RT) * S + sp.j : P.RT * S);
      float g[kR];
#pragma unroll
      for (int i = 0; i < kR; ++i) {
        const int rs = b0 + i;
        g[i] = (ok && rs < f.Hs) ? gt[sp.g * HW + rs * f.Ws + sp.j] : 0.f;
      }
#pragma unroll
      for (int ci = 0; ci < KB; ++ci) {
        if (ci >= ncells) break;
        const float* p = base + pg->cell_off[ci];
#pragma unroll
        for (int i = 0; i < kR; ++i) acc[ci] = fmaf(g[i], p[i * S], acc[ci]);
      }
    }
  }
  // lane sums -> per-wave sums -> per-tap partial of this workgroup, fixed order
#pragma unroll
  for (int ci = 0; ci < KB; ++ci) {
    if (ci >= ncells) break;
    float v = acc[ci];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    if (lane == 0) red[wave * 64 + ci] = v;
  }
  __syncthreads();
  const size_t part = blockIdx.z;
  for (int k = tid; k < P.K; k += blockDim.x) {
    const int ci = min(pg->tap_cell[k], KB - 1);
    float v = 0.f;
    for (int w = 0; w < nwaves; ++w) v += red[w * 64 + ci];
    partial[(part * P.C + c) * (size_t)P.K + k] = pg->finite ? v : __builtin_nanf("");
  }
}

template <typename T>
__global__ __launch_bounds__(256) void wgrad_reduce(const float* __restrict__ partial, T* __restrict__ dw, int CK,
                                                    int parts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CK) return;
  float s = 0.f;
  for (int j = 0; j < parts; ++j) s += partial[(size_t)j * CK + i];
  dw[i] = from_f32<T>(s);
}

// ---------------------------------------------------------------- launch

template <typename K_>
hipError_t lds_attr(K_ kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)kMaxLdsBytes);
}

template <typename T, int S>
hipError_t gather_s(const RunsPlan& pl, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
  hipError_t e = lds_attr(gather_runs<T, S>);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gather_runs<T, S>), dim3((unsigned)pl.blocks_n, (unsigned)pl.p.C, 1), dim3(pl.threads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta,
                     static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int S, int KB>
hipError_t wgrad_launch(const RunsPlan& pl, const void* x, const void* dy, const float* theta, float* partial,
                        hipStream_t stream) {
  hipError_t e = lds_attr(wgrad_runs<T, S, KB>);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((wgrad_runs<T, S, KB>), dim3(1, (unsigned)pl.p.C, (unsigned)pl.blocks_n), dim3(pl.threads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  return hipGetLastError();
}

template <typename T, int S>
hipError_t wgrad_s(const RunsPlan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                   hipStream_t stream) {
  hipError_t e = pl.p.K <= 32 ? wgrad_launch<T, S, 32>(pl, x, dy, theta, partial, stream)
                              : wgrad_launch<T, S, 64>(pl, x, dy, theta, partial, stream);
  if (e != hipSuccess) return e;
  const int CK = pl.p.C * pl.p.K;
  hipLaunchKernelGGL(wgrad_reduce<T>, dim3((unsigned)((CK + 255) / 256)), dim3(256), 0, stream, partial,
                     static_cast<T*>(dw), CK, pl.blocks_n);
  return hipGetLastError();
}

#define O1D_FOR_EACH_S(X) X(32) X(48) X(72) X(80) X(88) X(104) X(112) X(120) X(136)

template <typename T>
hipError_t gather_t(const RunsPlan& pl, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
  switch (pl.S) {
#define O1D_CASE(SV) \
  case SV: return gather_s<T, SV>(pl, in, w, theta, out, stream);
    O1D_FOR_EACH_S(O1D_CASE)
#undef O1D_CASE
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t wgrad_t(const RunsPlan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                   hipStream_t stream) {
  switch (pl.S) {
#define O1D_CASE(SV) \
  case SV: return wgrad_s<T, SV>(pl, x, dy, theta, dw, partial, stream);
    O1D_FOR_EACH_S(O1D_CASE)
#undef O1D_CASE
  }
  return hipErrorInvalidValue;
}

}  // namespace
}  // namespace runs

hipError_t launch_gather_runs(Dtype dt, const runs::RunsPlan& pl, const void* in, const void* w, const float* theta,
                              void* out, hipStream_t stream) {
  if (dt == Dtype::F32) return runs::gather_t<float>(pl, in, w, theta, out, stream);
  return runs::gather_t<uint16_t>(pl, in, w, theta, out, stream);
}

hipError_t launch_wgrad_runs(Dtype dt, const runs::RunsPlan& pl, const void* x, const void* dy, const float* theta,
                             void* dw, float* partial, hipStream_t stream) {
  if (dt == Dtype::F32) return runs::wgrad_t<float>(pl, x, dy, theta, dw, partial, stream);
  return runs::wgrad_t<uint16_t>(pl, x, dy, theta, dw, partial, stream);
}

}  // namespace o1d
