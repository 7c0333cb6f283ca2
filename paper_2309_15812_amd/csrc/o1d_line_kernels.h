// Device code of the line kernels (included by the per-dtype, per-kind
// translation units o1d_line_{gather,wgrad}_{f32,bf16}.hip, which compile in
// parallel).
// Line kernels: depthwise convolution with oriented 1D kernels on gfx950.
//
// For one channel every output pixel reads the same set of cells, the digital
// line of Eq. (2) shifted to the pixel.  The kernels stage whole planes in LDS
// with a zero halo (the paper's one-read staging of the input in on-chip
// memory), then let every lane compute R outputs that are themselves spaced by
// a fixed step u = (1, s), s in {-1, 0, +1}, in the staging frame.  Walking the
// line's cells in order, two consecutive cells usually differ by exactly u;
// for such a cell the R values a lane needs are its previous R values shifted
// by one, so a sliding window of R registers is refilled with ONE LDS read.
// Only at a break of the line (a step other than u) are R values reloaded.
// The FMAs, not the LDS reads, are then the dominant cost at every angle.
//
// Geometry per channel (built once per workgroup by wave 0, one tap per lane):
//  * the staging frame: the plane, or its transpose when the line spans more
//    columns than rows, so that the line always advances at least one row
//    per cell;
//  * cells: the taps' offsets with duplicate taps merged (weights added) and
//    taps that can never land inside the plane dropped;
//  * the strip step s (the most frequent row-advancing step between cells);
//    vertical strips (s = 0) hold kRv outputs, diagonal strips kRd;
//  * per cell: its LDS offset, its weight and whether it continues the
//    previous cell by u.
//
// The cell loop is unrolled over a compile-time bound with the window index
// (c + i) mod R known at compile time; the cell data live in registers.
// Lanes of a task cover consecutive strip columns, so their LDS addresses are
// consecutive.  The tile row stride S is odd and compile-time: the window
// reads use immediate offsets m * (S + s) and the transposed staging writes
// of a half-wave hit 32 distinct banks.
//
// The weight gradient runs the same cell walk with data and weights
// exchanged: a lane multiplies its R dy values by the window and keeps one
// register accumulator per cell; lanes and waves are reduced in a fixed order
// at the end (no atomics, bitwise reproducible).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "o1d_device.h"
#include "o1d_launch.h"
#include "o1d_line.h"

#include <utility>

namespace o1d {
namespace line {
namespace {

// Calls f(std::integral_constant<int, i>) for i = 0 .. N-1, so that indices
// into register arrays are compile-time constants whatever the loop body.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Wave-uniform value read from LDS.  Geometry that is the same for every
// plane group is fetched this way inside the group loop (whose LDS stores
// and barriers keep the read there), so that the compiler recomputes the few
// values derived from it per group with scalar instructions instead of
// hoisting dozens of them out of the loop and spilling them.
__device__ __forceinline__ int opaque(const int* p) { return __builtin_amdgcn_readfirstlane(*p); }

// ---------------------------------------------------------------- program

struct Prog {
  int ncells;
  int tr;      // staging frame = transposed plane
  int s;       // strip step u = (1, s) in the staging frame
  int finite;  // the channel's angle is finite
  int pad_[12];
  uint32_t contm[2];  // bit c: cell c is cell c - 1 moved by u
  int pad2_[30];
  int16_t off[64];    // LDS offset of every cell from the output pixel, cell order (rows increasing)
  float w[64];        // weight of every cell (duplicate taps summed)
  int tap_cell[64];   // cell of every tap, -1 if the tap never lands in the plane
};
static_assert(sizeof(Prog) == kProgFloats * 4, "kProgFloats must match the program layout");

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
__device__ __forceinline__ uint64_t below_mask(int n) { return n <= 0 ? 0ull : (n >= 64 ? ~0ull : (~0ull >> (64 - n))); }
__device__ __forceinline__ uint64_t above_mask(int n) { return n >= 63 ? 0ull : (~0ull << (n + 1)); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int hibit(uint64_t m) { return m ? 63 - __clzll(m) : -1; }
__device__ __forceinline__ int lobit(uint64_t m) { return m ? __ffsll((long long)m) - 1 : 64; }

// Builds the channel's program.  Called by the 64 lanes of wave 0, lane k =
// tap k (K <= 63).  sign = -1 negates the offsets (input gradient).  Taps
// move monotonically along the line, so taps on one pixel are consecutive
// (and at most two: max(|sin|, |cos|) >= 1/sqrt(2)), and the taps that can
// land in the plane form one contiguous range.
template <typename T>
__device__ void build_program(Prog* pg, const T* __restrict__ wgt, float theta, int c, int K, int sign, int H,
                              int W, int S) {
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
  const bool tr = (wmax - wmin) > (hmax - hmin);
  const int a = tr ? dw : dh;  // row offset in the staging frame
  const int b = tr ? dh : dw;  // column offset in the staging frame
  const int Hs = tr ? W : H, Ws = tr ? H : W;
  const bool keep = act && a > -Hs && a < Hs && b > -Ws && b < Ws;
  const uint64_t keptm = __ballot(keep);

  // duplicates: the previous kept tap on the same pixel; the first tap of a
  // pair carries the summed weight
  const int pk = hibit(keptm & below_mask(k));
  const int pa = __shfl(a, pk < 0 ? 0 : pk, 64), pb = __shfl(b, pk < 0 ? 0 : pk, 64);
  const bool dup = keep && pk >= 0 && pa == a && pb == b;
  const uint64_t dupm = __ballot(dup);
  const int nk = lobit(keptm & above_mask(k));
  const float nw = __shfl(wk, nk > 63 ? 63 : nk, 64);
  const bool next_dup = nk < 64 && ((dupm >> nk) & 1ull);
  const float cw = wk + (next_dup ? nw : 0.f);
  const bool cell = keep && !dup;
  const uint64_t cellm = __ballot(cell);
  const int ncells = popc(cellm);
  const int ci = popc(cellm & below_mask(k));

  // cell order: rows increasing
  const int lfirst = lobit(cellm), llast = hibit(cellm);
  const int a_first = __shfl(a, lfirst > 63 ? 0 : lfirst, 64), a_last = __shfl(a, llast < 0 ? 0 : llast, 64);
  const bool rev = a_last < a_first;
  const int co = rev ? ncells - 1 - ci : ci;
  const int pc = rev ? lobit(cellm & above_mask(k)) : hibit(cellm & below_mask(k));  // predecessor cell lane
  const bool hp = cell && pc >= 0 && pc < 64;
  const int qa = __shfl(a, hp ? pc : 0, 64), qb = __shfl(b, hp ? pc : 0, 64);
  const int da = a - qa, db = b - qb;
  const int n0 = popc(__ballot(hp && da == 1 && db == 0));
  const int np = popc(__ballot(hp && da == 1 && db == 1));
  const int nm = popc(__ballot(hp && da == 1 && db == -1));
  int s = 0;
  if (np > n0 && np >= nm)
    s = 1;
  else if (nm > n0 && nm > np)
    s = -1;
  const bool cont = hp && da == 1 && db == s;
  const bool allfin = __ballot(act && !fin) == 0ull;

  // unused entries stay 0 / inside the tile (the walks prefetch one cell ahead)
  pg->off[k] = 0;
  pg->w[k] = 0.f;
  if (cell && co >= 0 && co < 64) {
    pg->off[co] = (int16_t)(a * S + b);
    pg->w[co] = allfin ? cw : __builtin_nanf("");  // a non-finite angle poisons the channel
  }
  // continuation bits in cell order
  uint64_t cm = (cell && cont && co >= 0 && co < 64) ? (1ull << co) : 0ull;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)cm, m, 64), hi = __shfl_xor((uint32_t)(cm >> 32), m, 64);
    cm |= ((uint64_t)hi << 32) | lo;
  }
  const int own = dup ? pk : k;  // the lane of the cell that owns this tap
  const int oco = __shfl(co, own < 0 ? 0 : own, 64);
  if (act) pg->tap_cell[k] = keep ? oco : -1;
  if (k == 0) {
    pg->contm[0] = (uint32_t)cm;
    pg->contm[1] = (uint32_t)(cm >> 32);
    pg->ncells = ncells;
    pg->tr = tr ? 1 : 0;
    pg->s = s;
    pg->finite = allfin ? 1 : 0;
  }
}

// ---------------------------------------------------------------- cell walks

// Cell data of the channel: offsets packed two per 32-bit word and the
// continuation bits, all wave-uniform (SGPRs).  They are re-read from LDS at
// the start of every strip walk: the plane loop's barriers keep the compiler
// from hoisting the reads, so it decodes each cell with a few scalar
// instructions inside the walk instead of keeping every decoded value alive
// (and spilled) across the loop.
template <int KB>
struct Cells {
  int offp[KB / 2];
  uint32_t cont_lo, cont_hi;
  int ncells;
  __device__ __forceinline__ int off(int c) const {
    const int v = offp[c >> 1];
    return (c & 1) ? (v >> 16) : ((v << 16) >> 16);
  }
  __device__ __forceinline__ bool cont(int c) const { return ((c < 32 ? cont_lo >> c : cont_hi >> (c - 32)) & 1u) != 0; }
};

template <int KB>
__device__ __forceinline__ Cells<KB> fetch_cells(const Prog* pg) {
  Cells<KB> cl;
  const int* op = reinterpret_cast<const int*>(pg->off);
#pragma unroll
  for (int i = 0; i < KB / 2; ++i) cl.offp[i] = __builtin_amdgcn_readfirstlane(op[i]);
  const int n = __builtin_amdgcn_readfirstlane(pg->ncells);
  cl.ncells = n < KB ? n : KB;
  cl.cont_lo = __builtin_amdgcn_readfirstlane(pg->contm[0]);
  cl.cont_hi = __builtin_amdgcn_readfirstlane(pg->contm[1]);
  return cl;
}

// The 32-bit LDS address of a pointer into dynamic shared memory.
__device__ __forceinline__ uint32_t lds_addr(const float* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)p;
}

// One cell step of the sliding window, in inline assembly so that the
// register slots are updated in place and every LDS wait is exact.  The
// window of a strip is R values x[p + i * ST], i < R, at the cell's LDS
// address p; R + 1 registers rotate through it.
//  * The first cell of a walk (FIRST) loads all R values and waits.
//  * Every later cell first waits for the read its predecessor left in
//    flight (the window's last value, tied in as `wl`), then, if its
//    continuation bit is clear (a line break), reloads the R - 1 leading
//    values (immediate offsets along u) and waits again.
//  * With PF, and if the walk has a next cell (c1 < n), the step then reads
//    that cell's last value into the spare register `wn` and leaves the
//    read in flight, so that it overlaps this cell's multiplies.  The next
//    step takes the same register as its `wl`, so that no instruction of
//    the compiler touches it before the wait; no read is in flight when a
//    walk ends.
// Neither a reload nor a prefetch creates values that need copying, so the
// rotating window costs no register moves.
template <int R, int ST, bool FIRST, bool PF>
struct Refill;

template <int ST>
struct Refill<14, ST, true, true> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6, float& w7, float& w8, float& w9, float& w10, float& w11, float& w12, float& w13, float& wn) {
    asm volatile(
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "ds_read_b32 %[w7], %[a] offset:%[o7]\n"
        "ds_read_b32 %[w8], %[a] offset:%[o8]\n"
        "ds_read_b32 %[w9], %[a] offset:%[o9]\n"
        "ds_read_b32 %[w10], %[a] offset:%[o10]\n"
        "ds_read_b32 %[w11], %[a] offset:%[o11]\n"
        "ds_read_b32 %[w12], %[a] offset:%[o12]\n"
        "ds_read_b32 %[w13], %[a] offset:%[o13]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "s_cmp_le_u32 %[n], %[c1]\n"
        "s_cbranch_scc1 2f\n"
        "ds_read_b32 %[wn], %[an] offset:%[opf]\n"
        "2:\n"
        : [w0] "=&v"(w0), [w1] "=&v"(w1), [w2] "=&v"(w2), [w3] "=&v"(w3), [w4] "=&v"(w4), [w5] "=&v"(w5), [w6] "=&v"(w6), [w7] "=&v"(w7), [w8] "=&v"(w8), [w9] "=&v"(w9), [w10] "=&v"(w10), [w11] "=&v"(w11), [w12] "=&v"(w12), [w13] "=&v"(w13), [wn] "=&v"(wn)
        : [a] "v"(a), [an] "v"(an), [n] "s"(n), [c1] "i"(c1), [opf] "i"(13 * ST * 4), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4), [o7] "i"(7 * ST * 4), [o8] "i"(8 * ST * 4), [o9] "i"(9 * ST * 4), [o10] "i"(10 * ST * 4), [o11] "i"(11 * ST * 4), [o12] "i"(12 * ST * 4), [o13] "i"(13 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<14, ST, true, false> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6, float& w7, float& w8, float& w9, float& w10, float& w11, float& w12, float& w13) {
    asm volatile(
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "ds_read_b32 %[w7], %[a] offset:%[o7]\n"
        "ds_read_b32 %[w8], %[a] offset:%[o8]\n"
        "ds_read_b32 %[w9], %[a] offset:%[o9]\n"
        "ds_read_b32 %[w10], %[a] offset:%[o10]\n"
        "ds_read_b32 %[w11], %[a] offset:%[o11]\n"
        "ds_read_b32 %[w12], %[a] offset:%[o12]\n"
        "ds_read_b32 %[w13], %[a] offset:%[o13]\n"
        "s_waitcnt lgkmcnt(0)\n"
        : [w0] "=&v"(w0), [w1] "=&v"(w1), [w2] "=&v"(w2), [w3] "=&v"(w3), [w4] "=&v"(w4), [w5] "=&v"(w5), [w6] "=&v"(w6), [w7] "=&v"(w7), [w8] "=&v"(w8), [w9] "=&v"(w9), [w10] "=&v"(w10), [w11] "=&v"(w11), [w12] "=&v"(w12), [w13] "=&v"(w13)
        : [a] "v"(a), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4), [o7] "i"(7 * ST * 4), [o8] "i"(8 * ST * 4), [o9] "i"(9 * ST * 4), [o10] "i"(10 * ST * 4), [o11] "i"(11 * ST * 4), [o12] "i"(12 * ST * 4), [o13] "i"(13 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<14, ST, false, true> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6, float& w7, float& w8, float& w9, float& w10, float& w11, float& w12, float& wl, float& wn) {
    asm volatile(
        "s_waitcnt lgkmcnt(0)\n"
        "s_bitcmp1_b32 %[bits], %[bit]\n"
        "s_cbranch_scc1 1f\n"
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "ds_read_b32 %[w7], %[a] offset:%[o7]\n"
        "ds_read_b32 %[w8], %[a] offset:%[o8]\n"
        "ds_read_b32 %[w9], %[a] offset:%[o9]\n"
        "ds_read_b32 %[w10], %[a] offset:%[o10]\n"
        "ds_read_b32 %[w11], %[a] offset:%[o11]\n"
        "ds_read_b32 %[w12], %[a] offset:%[o12]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "1:\n"
        "s_cmp_le_u32 %[n], %[c1]\n"
        "s_cbranch_scc1 2f\n"
        "ds_read_b32 %[wn], %[an] offset:%[opf]\n"
        "2:\n"
        : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3), [w4] "+v"(w4), [w5] "+v"(w5), [w6] "+v"(w6), [w7] "+v"(w7), [w8] "+v"(w8), [w9] "+v"(w9), [w10] "+v"(w10), [w11] "+v"(w11), [w12] "+v"(w12), [wl] "+v"(wl), [wn] "=&v"(wn)
        : [a] "v"(a), [bits] "s"(bits), [bit] "i"(bit), [an] "v"(an), [n] "s"(n), [c1] "i"(c1), [opf] "i"(13 * ST * 4), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4), [o7] "i"(7 * ST * 4), [o8] "i"(8 * ST * 4), [o9] "i"(9 * ST * 4), [o10] "i"(10 * ST * 4), [o11] "i"(11 * ST * 4), [o12] "i"(12 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<14, ST, false, false> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6, float& w7, float& w8, float& w9, float& w10, float& w11, float& w12, float& wl) {
    asm volatile(
        "s_waitcnt lgkmcnt(0)\n"
        "s_bitcmp1_b32 %[bits], %[bit]\n"
        "s_cbranch_scc1 1f\n"
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "ds_read_b32 %[w7], %[a] offset:%[o7]\n"
        "ds_read_b32 %[w8], %[a] offset:%[o8]\n"
        "ds_read_b32 %[w9], %[a] offset:%[o9]\n"
        "ds_read_b32 %[w10], %[a] offset:%[o10]\n"
        "ds_read_b32 %[w11], %[a] offset:%[o11]\n"
        "ds_read_b32 %[w12], %[a] offset:%[o12]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "1:\n"
        : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3), [w4] "+v"(w4), [w5] "+v"(w5), [w6] "+v"(w6), [w7] "+v"(w7), [w8] "+v"(w8), [w9] "+v"(w9), [w10] "+v"(w10), [w11] "+v"(w11), [w12] "+v"(w12), [wl] "+v"(wl)
        : [a] "v"(a), [bits] "s"(bits), [bit] "i"(bit), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4), [o7] "i"(7 * ST * 4), [o8] "i"(8 * ST * 4), [o9] "i"(9 * ST * 4), [o10] "i"(10 * ST * 4), [o11] "i"(11 * ST * 4), [o12] "i"(12 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<7, ST, true, true> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6, float& wn) {
    asm volatile(
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "s_cmp_le_u32 %[n], %[c1]\n"
        "s_cbranch_scc1 2f\n"
        "ds_read_b32 %[wn], %[an] offset:%[opf]\n"
        "2:\n"
        : [w0] "=&v"(w0), [w1] "=&v"(w1), [w2] "=&v"(w2), [w3] "=&v"(w3), [w4] "=&v"(w4), [w5] "=&v"(w5), [w6] "=&v"(w6), [wn] "=&v"(wn)
        : [a] "v"(a), [an] "v"(an), [n] "s"(n), [c1] "i"(c1), [opf] "i"(6 * ST * 4), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<7, ST, true, false> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& w6) {
    asm volatile(
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "ds_read_b32 %[w6], %[a] offset:%[o6]\n"
        "s_waitcnt lgkmcnt(0)\n"
        : [w0] "=&v"(w0), [w1] "=&v"(w1), [w2] "=&v"(w2), [w3] "=&v"(w3), [w4] "=&v"(w4), [w5] "=&v"(w5), [w6] "=&v"(w6)
        : [a] "v"(a), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4), [o6] "i"(6 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<7, ST, false, true> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& wl, float& wn) {
    asm volatile(
        "s_waitcnt lgkmcnt(0)\n"
        "s_bitcmp1_b32 %[bits], %[bit]\n"
        "s_cbranch_scc1 1f\n"
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "1:\n"
        "s_cmp_le_u32 %[n], %[c1]\n"
        "s_cbranch_scc1 2f\n"
        "ds_read_b32 %[wn], %[an] offset:%[opf]\n"
        "2:\n"
        : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3), [w4] "+v"(w4), [w5] "+v"(w5), [wl] "+v"(wl), [wn] "=&v"(wn)
        : [a] "v"(a), [bits] "s"(bits), [bit] "i"(bit), [an] "v"(an), [n] "s"(n), [c1] "i"(c1), [opf] "i"(6 * ST * 4), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4)
        : "scc");
  }
};

template <int ST>
struct Refill<7, ST, false, false> {
  static __device__ __forceinline__ void run(uint32_t a, uint32_t an, uint32_t bits, int bit, uint32_t n, int c1, float& w0, float& w1, float& w2, float& w3, float& w4, float& w5, float& wl) {
    asm volatile(
        "s_waitcnt lgkmcnt(0)\n"
        "s_bitcmp1_b32 %[bits], %[bit]\n"
        "s_cbranch_scc1 1f\n"
        "ds_read_b32 %[w0], %[a] offset:%[o0]\n"
        "ds_read_b32 %[w1], %[a] offset:%[o1]\n"
        "ds_read_b32 %[w2], %[a] offset:%[o2]\n"
        "ds_read_b32 %[w3], %[a] offset:%[o3]\n"
        "ds_read_b32 %[w4], %[a] offset:%[o4]\n"
        "ds_read_b32 %[w5], %[a] offset:%[o5]\n"
        "s_waitcnt lgkmcnt(0)\n"
        "1:\n"
        : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3), [w4] "+v"(w4), [w5] "+v"(w5), [wl] "+v"(wl)
        : [a] "v"(a), [bits] "s"(bits), [bit] "i"(bit), [o0] "i"(0 * ST * 4), [o1] "i"(1 * ST * 4), [o2] "i"(2 * ST * 4), [o3] "i"(3 * ST * 4), [o4] "i"(4 * ST * 4), [o5] "i"(5 * ST * 4)
        : "scc");
  }
};

template <int C, int R, int ST, bool FIRST, bool PF, int... I>
__device__ __forceinline__ void refill_slots(uint32_t a, uint32_t an, uint32_t bits, uint32_t n, float (&win)[R + 1],
                                             std::integer_sequence<int, I...>) {
  constexpr int NS = R + 1;
  if constexpr (FIRST && PF)
    Refill<R, ST, true, true>::run(a, an, bits, C & 31, n, C + 1, win[(C + I) % NS]..., win[(C + R - 1) % NS],
                                   win[(C + R) % NS]);
  else if constexpr (FIRST)
    Refill<R, ST, true, false>::run(a, an, bits, C & 31, n, C + 1, win[(C + I) % NS]..., win[(C + R - 1) % NS]);
  else if constexpr (PF)
    Refill<R, ST, false, true>::run(a, an, bits, C & 31, n, C + 1, win[(C + I) % NS]..., win[(C + R - 1) % NS],
                                    win[(C + R) % NS]);
  else
    Refill<R, ST, false, false>::run(a, an, bits, C & 31, n, C + 1, win[(C + I) % NS]..., win[(C + R - 1) % NS]);
}

// The sliding window of one strip: R + 1 register slots.  At cell C the
// window is slots (C + i) % (R + 1), i < R, holding x[p_C + i * (S + SD)]
// (p_C = the strip's base moved by the cell's offset); slot (C + R) % (R + 1)
// receives the last value of cell C + 1, read while cell C is multiplied.
// A continuing cell therefore costs one LDS read, a line break R - 1.
// Cells [C0, CE) form one walk: C0 loads the whole window, CE - 1 reads
// nothing ahead.
template <int C, int C0, int CE, int R, int ST, int KB>
__device__ __forceinline__ void window_step(const Cells<KB>& cl, uint32_t lbase, uint32_t a, float (&win)[R + 1],
                                            uint32_t& a_next) {
  constexpr bool PF = C + 1 < CE;
  a_next = lbase + (uint32_t)(cl.off(C + 1 < KB ? C + 1 : C) * 4);  // the next walk may start at C + 1
  refill_slots<C, R, ST, C == C0, PF>(a, a_next, C < 32 ? cl.cont_lo : cl.cont_hi, (uint32_t)cl.ncells, win,
                                      std::make_integer_sequence<int, R - 1>{});
}

// acc[i] += sum_c w[c] * x[p_c + i * (S + SD)]: the gather of one strip.
template <int C, int KB, int S, int R, int SD>
struct GatherWalk {
  static __device__ __forceinline__ void run(const Cells<KB>& cl, uint32_t lbase, uint32_t a, const float (&wt)[KB],
                                             float (&win)[R + 1], float (&acc)[R]) {
    if (C >= cl.ncells) return;
    constexpr int NS = R + 1;
    uint32_t a_next;
    window_step<C, 0, KB, R, S + SD, KB>(cl, lbase, a, win, a_next);
#pragma unroll
    for (int i = 0; i < R; ++i) acc[i] = fmaf(wt[C], win[(C + i) % NS], acc[i]);
    GatherWalk<C + 1, KB, S, R, SD>::run(cl, lbase, a_next, wt, win, acc);
  }
};
template <int KB, int S, int R, int SD>
struct GatherWalk<KB, KB, S, R, SD> {
  static __device__ __forceinline__ void run(const Cells<KB>&, uint32_t, uint32_t, const float (&)[KB],
                                             float (&)[R + 1], float (&)[R]) {}
};

// acc[c] += sum_i g[i] * x[p_c + i * (S + SD)]: the same walk with data and
// weights exchanged (the weight gradient of one strip), over cells [C, CE).
// `a` enters as the LDS address of cell C and leaves as that of cell CE, so
// a 64-cell walk runs as two halves (each half's early exits then only merge
// its own 32 accumulators).
template <int C, int C0, int CE, int KB, int S, int R, int SD>
struct WgradWalk {
  static __device__ __forceinline__ void run(const Cells<KB>& cl, uint32_t lbase, uint32_t& a, const float (&g)[R],
                                             float (&win)[R + 1], float (&acc)[32]) {
    if (C >= cl.ncells) return;
    constexpr int NS = R + 1;
    uint32_t a_next;
    window_step<C, C0, CE, R, S + SD, KB>(cl, lbase, a, win, a_next);
    float t0 = 0.f, t1 = 0.f;
#pragma unroll
    for (int i = 0; i < R; i += 2) {
      t0 = fmaf(g[i], win[(C + i) % NS], t0);
      if (i + 1 < R) t1 = fmaf(g[i + 1], win[(C + i + 1) % NS], t1);
    }
    acc[C - C0] += t0 + t1;
    // keep the cell's sum ahead of the next cell's exit test: otherwise the
    // compiler sinks it past the test and keeps the window alive there
    asm volatile("" : "+v"(acc[C - C0]));
    a = a_next;
    WgradWalk<C + 1, C0, CE, KB, S, R, SD>::run(cl, lbase, a, g, win, acc);
  }
};
template <int C0, int CE, int KB, int S, int R, int SD>
struct WgradWalk<CE, C0, CE, KB, S, R, SD> {
  static __device__ __forceinline__ void run(const Cells<KB>&, uint32_t, uint32_t&, const float (&)[R],
                                             float (&)[R + 1], float (&)[32]) {}
};

// ---------------------------------------------------------------- geometry

// Frame of one channel and the strip tiling for its strip shape.
struct Frame {
  int tr, s, R, Hs, Ws;
  Tiling t;
};

__device__ __forceinline__ Frame frame_of(const Prog* pg, const LineParams& P) {
  Frame f;
  f.tr = opaque(&pg->tr);
  f.s = opaque(&pg->s);
  f.R = f.s == 0 ? kRv : kRd;
  f.Hs = f.tr ? P.W : P.H;
  f.Ws = f.tr ? P.H : P.W;
  f.t = tiling(f.Hs, f.Ws, f.R, f.s);
  return f;
}

// A lane's strip task for lane iteration `it`: the strip of plane slot g
// starting at row b0 and column j of the staging frame.  Lanes without a
// strip of their own (padding lanes of a segment, tasks past the end) get
// g = kNoPlane and point at a real strip, so that their reads stay inside
// the tile.  Divisions by the (small) tiling counts are multiplications by
// 2^20 reciprocals: exact for quotients of numbers below 1024.
constexpr int kNoPlane = 255;

struct TaskMap {
  int lg, li;           // the lane's task within the wave, strip within the task
  int per_plane, T, nit;
  uint32_t rpp, rns;    // ceil(2^20 / per_plane), ceil(2^20 / nseg)
};

__device__ __forceinline__ TaskMap task_map(const LineParams& P, const Frame& f, int lane) {
  const Tiling& t = f.t;
  TaskMap m;
  m.lg = lane / t.segw;
  m.li = lane - m.lg * t.segw;
  m.per_plane = t.nb * t.nseg;
  m.T = P.G * m.per_plane;
  m.nit = cdiv(m.T, kWaves * t.tpw);
  m.rpp = ((1u << 20) + (uint32_t)m.per_plane - 1) / (uint32_t)m.per_plane;
  m.rns = ((1u << 20) + (uint32_t)t.nseg - 1) / (uint32_t)t.nseg;
  return m;
}

struct Task {
  int g, b0, j;
};

template <int S>
__device__ __forceinline__ Task task_at(const LineParams& P, const Frame& f, const TaskMap& m, int it, int wave) {
  const Tiling& t = f.t;
  int ti = (it * kWaves + wave) * t.tpw + m.lg;
  bool valid = ti < m.T;
  if (!valid) ti = 0;
  const int g = (int)(((uint32_t)ti * m.rpp) >> 20);
  const int rem = ti - g * m.per_plane;
  const int band = (int)(((uint32_t)rem * m.rns) >> 20);
  const int seg = rem - band * t.nseg;
  int jj = seg * t.segw + m.li;
  if (jj >= t.nj) {
    jj = t.nj - 1;
    valid = false;
  }
  Task k;
  k.g = valid ? g : kNoPlane;
  k.b0 = band * f.R;
  k.j = t.jlo + jj;
  return k;
}

// Staging of one plane group through registers.  Every lane moves 4
// consecutive elements of a plane row per slot with one 16-byte (bf16:
// 8-byte) buffer access.  A half-wave covers 4 rows x 8 quads: lane -> row
// (lane >> 3) & 3 (+4 in the second half-wave, +8 per wave), quad lane & 7.
// For an odd LDS row stride the 32 component writes of a half-wave then hit
// 32 distinct banks in either frame.  Slot q = (g, k, m): plane g of the
// group, row step k (32 rows), column segment m (32 columns), m fastest.
//
// A lane's slot addresses are computed once per workgroup:
//  * goff[q]: byte offset of its 4 elements from the group's first element,
//    or kOob for a slot outside the plane.  Buffer accesses beyond the
//    resource's size read zeros and drop stores, and a group's resource
//    covers only its ng planes, so absent slots and planes need no branch.
//  * LDS addresses of the first element in a tile, or of the lane's word
//    in the trash area (written, never read) for a slot outside the plane.
constexpr uint32_t kOob = 0x80000000u;
constexpr int kQ = kMaxSlots / 4;  // vector slots per lane

// Calls f(q, ok, g, h, w) for every slot: plane g of the group, plane row h
// and first column w of the lane's 4 elements, ok = they lie in the plane.
template <class F>
__device__ __forceinline__ void for_each_slot(const LineParams& P, F&& f) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hr = wave * 8 + (lane >> 5) * 4 + ((lane >> 3) & 3);
  const int w0 = 4 * (lane & 7);
  const int per = P.ks * P.ms;
  static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    const int g = q / per, r = q - g * per, k = r / P.ms, m = r - k * P.ms;
    const int h = hr + 32 * k, w = w0 + 32 * m;
    f(q, g < P.G && h < P.H && w < P.W, g, h, w);
  });
}

template <typename T>
__device__ __forceinline__ void slot_offsets(const LineParams& P, uint32_t (&goff)[kQ]) {
  const int img = P.C * P.H * P.W;
  for_each_slot(P, [&](int q, bool ok, int g, int h, int w) __attribute__((always_inline)) {
    goff[q] = ok ? (uint32_t)((g * img + h * P.W + w) * (int)sizeof(T)) : kOob;
  });
}

// Element (r, c) of tile slot g (frame coordinates: (h, w), or (w, h) when
// transposed) is the float at byte address base + 4 * (g * pitch + r * S + c).
template <int S>
__device__ __forceinline__ void slot_lds(const LineParams& P, uint32_t base, int pitch, bool tr, uint32_t trash,
                                         uint32_t (&a)[kQ]) {
  const uint32_t tl = trash + 4 * (threadIdx.x & 63);
  for_each_slot(P, [&](int q, bool ok, int g, int h, int w) __attribute__((always_inline)) {
    a[q] = ok ? base + 4 * (uint32_t)(g * pitch + (tr ? w * S + h : h * S + w)) : tl;
  });
}

// A buffer resource over `bytes` bytes from p (raw, no swizzle).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ float lds_load(uint32_t a) {
  return *(const __attribute__((address_space(3))) float*)(uintptr_t)a;
}
__device__ __forceinline__ void lds_store(uint32_t a, float v) {
  *(__attribute__((address_space(3))) float*)(uintptr_t)a = v;
}

// Raw staging registers: the loaded words are not touched until they are
// written to LDS (converting them at load time would make the compiler wait
// for every load right after issuing it).  float32: one word per element;
// bfloat16: 4 elements in 2 words.
template <typename T>
struct Raw;
template <>
struct Raw<float> {
  static constexpr int kWords = 4;
  static __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint32_t* r) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    r[0] = v[0]; r[1] = v[1]; r[2] = v[2]; r[3] = v[3];
  }
  static __device__ __forceinline__ float elem(const uint32_t* r, int j) { return __uint_as_float(r[j]); }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float (&e)[4]) {
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    u4 v;
    v[0] = __float_as_uint(e[0]); v[1] = __float_as_uint(e[1]); v[2] = __float_as_uint(e[2]); v[3] = __float_as_uint(e[3]);
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, off, 0, 0);
  }
};
template <>
struct Raw<uint16_t> {
  static constexpr int kWords = 2;
  static __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint32_t* r) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0);
    r[0] = v[0]; r[1] = v[1];
  }
  static __device__ __forceinline__ float elem(const uint32_t* r, int j) {
    const uint32_t w = r[j >> 1];
    return __uint_as_float((j & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float (&e)[4]) {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    u2 v;
    v[0] = (uint32_t)from_f32<uint16_t>(e[0]) | ((uint32_t)from_f32<uint16_t>(e[1]) << 16);
    v[1] = (uint32_t)from_f32<uint16_t>(e[2]) | ((uint32_t)from_f32<uint16_t>(e[3]) << 16);
    __builtin_amdgcn_raw_buffer_store_b64(v, rs, off, 0, 0);
  }
};

// Loads the slots of a group (ng >= 1 planes from `src`) into raw registers.
template <typename T>
__device__ __forceinline__ void stage_load(const LineParams& P, const T* src, int ng, const uint32_t (&goff)[kQ],
                                           uint32_t (&v)[kMaxSlots]) {
  const __amdgpu_buffer_rsrc_t rs = buffer_of(src, ng * P.C * P.H * P.W * (int)sizeof(T));
  static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    Raw<T>::load(rs, goff[q], &v[Raw<T>::kWords * q]);
  });
}

// Writes the slots into a tile: the 4 elements of a slot are consecutive
// along the frame's rows, or along its columns (stride S) when transposed.
template <typename T, int S>
__device__ __forceinline__ void stage_store(const uint32_t (&a)[kQ], bool tr, const uint32_t (&v)[kMaxSlots]) {
  if (tr) {
    static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      static_for<4>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        lds_store(a[q] + j * S * 4, Raw<T>::elem(&v[Raw<T>::kWords * q], j));
      });
    });
  } else {
    static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      static_for<4>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        lds_store(a[q] + j * 4, Raw<T>::elem(&v[Raw<T>::kWords * q], j));
      });
    });
  }
}

// ---------------------------------------------------------------- forward / input gradient

template <typename T, int S, int R, int SD, int KB>
__device__ __forceinline__ void gather_group(const LineParams& P, const Frame& f, const TaskMap& tm, int wave,
                                             const float* tiles, float* otiles, T* __restrict__ outn, int ng,
                                             const Prog* pg, const float (&wt)[KB]) {
  const int CHW = P.C * P.H * P.W;
  for (int it = 0; it < tm.nit; ++it) {
    const Task k = task_at<S>(P, f, tm, it, wave);
    const int g = k.g, b0 = k.b0, j = k.j;
    const uint32_t lbase = lds_addr(tiles + (g < kNoPlane ? g : 0) * P.PS + kGuard + (b0 + P.halo) * S + j + P.halo);
    const Cells<KB> cl = fetch_cells<KB>(pg);
    float acc[R], win[R + 1];
#pragma unroll
    for (int i = 0; i < R; ++i) acc[i] = 0.f;
    const uint32_t a0 = lbase + (uint32_t)(cl.off(0) * 4);
    GatherWalk<0, KB, S, R, SD>::run(cl, lbase, a0, wt, win, acc);
    if (g >= ng) continue;
    if (f.tr) {
      // frame (row, col) = plane (w, h): bounce through LDS (row stride S)
      // for coalesced stores; for vertical strips a ragged band only writes
      // past column W of the bounce row, which is never read
      float* o = otiles + (g * P.OPS + j * S + b0);
#pragma unroll
      for (int i = 0; i < R; ++i) {
        if (SD == 0) {
          o[i] = acc[i];
        } else {
          const int cc = j + SD * i;
          if (b0 + i < f.Hs && cc >= 0 && cc < f.Ws) o[i * (SD * S + 1)] = acc[i];
        }
      }
    } else {
      const int off = g * CHW + b0 * P.W + j;
      if (SD == 0 && b0 + R <= f.Hs) {
#pragma unroll
        for (int i = 0; i < R; ++i) {
          T* rowp = outn + i * P.W;  // wave-uniform row, per-lane column
          rowp[off] = from_f32<T>(acc[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < R; ++i) {
          const int cc = j + SD * i;
          if (b0 + i < f.Hs && cc >= 0 && cc < f.Ws) outn[off + i * (P.W + SD)] = from_f32<T>(acc[i]);
        }
      }
    }
  }
}

// Output bounce tile (plane orientation, row stride OS) -> global, planes
// [0, ng) of the group at `dst`, with the staging lane layout.
// Stores a group's outputs from the bounce tile (plane orientation, row
// stride S) as coalesced rows.
template <typename T>
__device__ __forceinline__ void flush_bounce(const LineParams& P, T* dst, int ng, const uint32_t (&lb)[kQ],
                                             const uint32_t (&goff)[kQ]) {
  const __amdgpu_buffer_rsrc_t rs = buffer_of(dst, ng * P.C * P.H * P.W * (int)sizeof(T));
  float e[kQ][4];  // all reads first, so that their latencies overlap
  static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    static_for<4>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      e[q][j] = lds_load(lb[q] + 4 * j);
    });
  });
  static_for<kQ>([&](auto qc) __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    Raw<T>::store(rs, goff[q], e[q]);
  });
}

template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads) void line_gather(LineParams P, const T* __restrict__ in,
                                                        const T* __restrict__ wgt, const float* __restrict__ theta,
                                                        T* __restrict__ out) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tiles = smem + kProgFloats;
  float* otiles = smem + P.aux;
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int HW = P.H * P.W;
  const size_t img = (size_t)P.C * HW;
  const int n_begin = blockIdx.x * P.npw;
  const int n_end = min(P.N, n_begin + P.npw);
  const T* inc = in + (size_t)c * HW;
  T* outc = out + (size_t)c * HW;

  // The first two groups' loads do not depend on the frame: issue them before
  // the program is built.  Two register buffers alternate, so every group's
  // loads are in flight for two groups' worth of compute.
  uint32_t goff[kQ];
  slot_offsets<T>(P, goff);
  uint32_t pa[kMaxSlots], pb[kMaxSlots];
  stage_load(P, inc + (size_t)n_begin * img, min(P.G, n_end - n_begin), goff, pa);
  if (n_begin + P.G < n_end)  // a second group exists (its first image is in the tensor)
    stage_load(P, inc + (size_t)(n_begin + P.G) * img, min(P.G, n_end - n_begin - P.G), goff, pb);
  for (int i = tid; i < P.G * P.PS; i += kThreads) tiles[i] = 0.f;  // halos and guards stay zero
  if (wave == 0) build_program<T>(pg, wgt, theta[c], c, P.K, P.sign, P.H, P.W, S);
  __syncthreads();
  const bool tr = opaque(&pg->tr) != 0;
  uint32_t lt[kQ], lb[kQ];  // the slots in the tile (staging frame) and in the bounce tile (plane)
  slot_lds<S>(P, lds_addr(tiles + kGuard + P.halo * S + P.halo), P.PS, tr, lds_addr(smem + P.trash), lt);
  slot_lds<S>(P, lds_addr(otiles), P.OPS, false, lds_addr(smem + P.trash), lb);
  float wt[KB];  // the cells' weights, wave-uniform, for the whole workgroup
#pragma unroll
  for (int i = 0; i < KB; ++i) wt[i] = pg->w[i];

  int prev = -1;  // first image of the group whose outputs wait in the bounce tile
  auto step = [&](uint32_t (&pre)[kMaxSlots], int n0) __attribute__((always_inline)) {
    const int ng = min(P.G, n_end - n0);
    const Frame f = frame_of(pg, P);
    __syncthreads();  // the tile and the bounce tile are free
    stage_store<T, S>(lt, tr, pre);
    if (prev >= 0) flush_bounce<T>(P, outc + (size_t)prev * img, min(P.G, n_end - prev), lb, goff);
    __syncthreads();  // the group is staged
    if (n0 + 2 * P.G < n_end)
      stage_load(P, inc + (size_t)(n0 + 2 * P.G) * img, min(P.G, n_end - n0 - 2 * P.G), goff, pre);
    T* outn = outc + (size_t)n0 * img;
    if (f.s == 0)
      gather_group<T, S, kRv, 0, KB>(P, f, task_map(P, f, lane), wave, tiles, otiles, outn, ng, pg, wt);
    else if (f.s > 0)
      gather_group<T, S, kRd, 1, KB>(P, f, task_map(P, f, lane), wave, tiles, otiles, outn, ng, pg, wt);
    else
      gather_group<T, S, kRd, -1, KB>(P, f, task_map(P, f, lane), wave, tiles, otiles, outn, ng, pg, wt);
    if (f.tr) prev = n0;
  };
  for (int n0 = n_begin; n0 < n_end; n0 += 2 * P.G) {
    step(pa, n0);
    if (n0 + P.G < n_end) step(pb, n0 + P.G);
  }
  if (prev >= 0) {
    __syncthreads();
    flush_bounce<T>(P, outc + (size_t)prev * img, min(P.G, n_end - prev), lb, goff);
  }
}

// ---------------------------------------------------------------- weight gradient

template <int S, int R, int SD, int KB>
__device__ __forceinline__ void wgrad_group(const LineParams& P, const Frame& f, const TaskMap& tm, int wave,
                                            const float* tiles, const float* gtiles, int ng, const Prog* pg,
                                            float (&acc0)[32], float (&acc1)[32]) {
  for (int it = 0; it < tm.nit; ++it) {
    const Task k = task_at<S>(P, f, tm, it, wave);
    const int g = k.g, b0 = k.b0, j = k.j;
    const uint32_t lbase = lds_addr(tiles + (g < kNoPlane ? g : 0) * P.PS + kGuard + (b0 + P.halo) * S + j + P.halo);
    // dy of the strip (dy tile: frame orientation, row stride S, zero margins
    // cover strip positions outside the plane); lanes without a strip of
    // their own multiply by 0
    const float* gp = gtiles + ((g < ng ? g : 0) * P.GPS + b0 * S + j + 6);
    const float m = g < ng ? 1.f : 0.f;
    float gv[R], win[R + 1];
#pragma unroll
    for (int i = 0; i < R; ++i) gv[i] = m * gp[i * (S + SD)];
    const Cells<KB> cl = fetch_cells<KB>(pg);
    const uint32_t a0 = lbase + (uint32_t)(cl.off(0) * 4);
    uint32_t a = a0;
    WgradWalk<0, 0, 32, KB, S, R, SD>::run(cl, lbase, a, gv, win, acc0);
    if (KB > 32 && cl.ncells > 32) WgradWalk<32, 32, KB, KB, S, R, SD>::run(cl, lbase, a, gv, win, acc1);
  }
}

template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads) void line_wgrad(LineParams P, const T* __restrict__ x, const T* __restrict__ dy,
                                                       const float* __restrict__ theta, float* __restrict__ partial) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tiles = smem + kProgFloats;
  float* gtiles = smem + P.aux;
  float* red = smem + P.red;  // [kWaves][64] per-wave cell sums
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int HW = P.H * P.W;
  const size_t img = (size_t)P.C * HW;
  const int n_begin = blockIdx.z * P.npw;
  const int n_end = min(P.N, n_begin + P.npw);
  const T* xc = x + (size_t)c * HW;
  const T* dc = dy + (size_t)c * HW;

  uint32_t goff[kQ];
  slot_offsets<T>(P, goff);
  uint32_t px[kMaxSlots], pd[kMaxSlots];
  stage_load(P, xc + (size_t)n_begin * img, min(P.G, n_end - n_begin), goff, px);
  stage_load(P, dc + (size_t)n_begin * img, min(P.G, n_end - n_begin), goff, pd);
  for (int i = tid; i < P.G * P.PS; i += kThreads) tiles[i] = 0.f;
  for (int i = tid; i < P.G * P.GPS; i += kThreads) gtiles[i] = 0.f;
  if (wave == 0) build_program<T>(pg, static_cast<const T*>(nullptr), theta[c], c, P.K, 1, P.H, P.W, S);
  __syncthreads();
  const bool tr = opaque(&pg->tr) != 0;
  uint32_t lx[kQ], ld[kQ];  // the slots in the x tile and in the dy tile (both in the staging frame)
  slot_lds<S>(P, lds_addr(tiles + kGuard + P.halo * S + P.halo), P.PS, tr, lds_addr(smem + P.trash), lx);
  slot_lds<S>(P, lds_addr(gtiles + 6), P.GPS, tr, lds_addr(smem + P.trash), ld);

  // per-lane cell sums: cells 0..31 and 32..63 (two arrays, so that each is
  // split into scalar registers)
  float acc0[32], acc1[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    acc0[i] = 0.f;
    acc1[i] = 0.f;
  }
  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    const int ng = min(P.G, n_end - n0);
    const Frame f = frame_of(pg, P);
    __syncthreads();
    stage_store<T, S>(lx, tr, px);
    stage_store<T, S>(ld, tr, pd);
    __syncthreads();
    if (n0 + P.G < n_end) {
      stage_load(P, xc + (size_t)(n0 + P.G) * img, min(P.G, n_end - n0 - P.G), goff, px);
      stage_load(P, dc + (size_t)(n0 + P.G) * img, min(P.G, n_end - n0 - P.G), goff, pd);
    }
    if (f.s == 0)
      wgrad_group<S, kRv, 0, KB>(P, f, task_map(P, f, lane), wave, tiles, gtiles, ng, pg, acc0, acc1);
    else if (f.s > 0)
      wgrad_group<S, kRd, 1, KB>(P, f, task_map(P, f, lane), wave, tiles, gtiles, ng, pg, acc0, acc1);
    else
      wgrad_group<S, kRd, -1, KB>(P, f, task_map(P, f, lane), wave, tiles, gtiles, ng, pg, acc0, acc1);
  }
  // lanes -> per-wave sums -> per-tap partial of this workgroup, fixed order
  const int ncells = min(__builtin_amdgcn_readfirstlane(pg->ncells), KB);
#pragma unroll
  for (int ci = 0; ci < KB; ++ci) {
    if (ci < ncells) {
      float v = ci < 32 ? acc0[ci & 31] : acc1[ci & 31];
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
      if (lane == 0) red[wave * 64 + ci] = v;
    }
  }
  __syncthreads();
  const size_t part = blockIdx.z;
  for (int k = tid; k < P.K; k += kThreads) {
    const int ci = pg->tap_cell[k];
    float v = 0.f;
    if (ci >= 0 && ci < KB)
      for (int w = 0; w < kWaves; ++w) v += red[w * 64 + ci];
    partial[(part * P.C + c) * (size_t)P.K + k] = pg->finite ? v : __builtin_nanf("");
  }
}

template <typename T>
__global__ __launch_bounds__(256) void line_wgrad_reduce(const float* __restrict__ partial, T* __restrict__ dw,
                                                         int CK, int parts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= CK) return;
  float s = 0.f;
  for (int j = 0; j < parts; ++j) s += partial[(size_t)j * CK + i];
  dw[i] = from_f32<T>(s);
}

// ---------------------------------------------------------------- launch helpers

template <typename K_>
hipError_t lds_attr(K_ kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)kMaxLdsBytes);
}

template <typename T, int S, int KB>
hipError_t gather_launch(const LinePlan& pl, const void* in, const void* w, const float* theta, void* out,
                         hipStream_t stream) {
  hipError_t e = lds_attr(line_gather<T, S, KB>);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((line_gather<T, S, KB>), dim3((unsigned)pl.blocks_n, (unsigned)pl.p.C, 1), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta,
                     static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T>
hipError_t gather_t(const LinePlan& pl, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
#define O1D_CASE(SV)                                                                               \
  if (pl.S == SV) {                                                                                \
    if (pl.KB == 32) return gather_launch<T, SV, 32>(pl, in, w, theta, out, stream);               \
    if (pl.KB == 64) return gather_launch<T, SV, 64>(pl, in, w, theta, out, stream);               \
  }
  O1D_LINE_STRIDES(O1D_CASE)
#undef O1D_CASE
  return hipErrorInvalidValue;
}

template <typename T, int S, int KB>
hipError_t wgrad_launch(const LinePlan& pl, const void* x, const void* dy, const float* theta, float* partial,
                        hipStream_t stream) {
  hipError_t e = lds_attr(line_wgrad<T, S, KB>);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((line_wgrad<T, S, KB>), dim3(1, (unsigned)pl.p.C, (unsigned)pl.blocks_n), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  return hipGetLastError();
}

template <typename T>
hipError_t wgrad_t(const LinePlan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                   hipStream_t stream) {
  hipError_t e = hipErrorInvalidValue;
#define O1D_CASE(SV)                                                                               \
  if (pl.S == SV) {                                                                                \
    if (pl.KB == 32) e = wgrad_launch<T, SV, 32>(pl, x, dy, theta, partial, stream);               \
    if (pl.KB == 64) e = wgrad_launch<T, SV, 64>(pl, x, dy, theta, partial, stream);               \
  }
  O1D_LINE_STRIDES(O1D_CASE)
#undef O1D_CASE
  if (e != hipSuccess) return e;
  const int CK = pl.p.C * pl.p.K;
  hipLaunchKernelGGL(line_wgrad_reduce<T>, dim3((unsigned)((CK + 255) / 256)), dim3(256), 0, stream, partial,
                     static_cast<T*>(dw), CK, pl.blocks_n);
  return hipGetLastError();
}

}  // namespace
}  // namespace line
}  // namespace o1d
