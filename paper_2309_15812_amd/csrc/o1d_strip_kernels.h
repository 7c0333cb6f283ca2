// Device code of the strip kernels (included by the translation units
// o1d_strip_{gather,wgrad,bwd}_{f32,bf16}_k{32,64}.hip).
//
// Strip kernels: forward pass and input gradient of the oriented 1D
// depthwise convolution (Eq. 1: y[p,q] = sum_k w_k x[p + dh_k, q + dw_k],
// offsets from Eq. 2) on gfx950.
//
// For one channel every output reads the same cells, the digital line of
// Eq. (2) shifted to the output.  A workgroup stages planes of its channel
// in LDS with a zero margin (the paper's one-read staging of the input in
// on-chip memory), then every lane computes a block of outputs: NC adjacent
// strips of R outputs each, the strips stepping u = (1, s), s in {-1, 0, 1},
// in the staging frame.  Walking the line's cells in order, a cell that is
// its predecessor moved by u (a continuing cell) needs the lane's previous
// window moved by one row: R + 1 register rows rotate, and only the new
// row (NC values) is read.  A cell that starts a run reloads all R rows.
// Each cell then costs NC LDS reads and R * NC FMAs, and its bookkeeping is
// a handful of instructions:
//  * run base addresses: the LDS address of row i, column k of cell c is
//    base_run + 4 ((c + i) st + k), st = the strip step in floats, so the
//    offsets are immediates and only a run's first cell computes a base;
//  * the next cell's new row is read before the cell's multiplies.
// The issue rate of a SIMD (about one instruction per four cycles) bounds
// these kernels, so the multiplies' share of the instruction stream is
// what the design maximises.
//
// Geometry per channel, built once per workgroup by wave 0 (one tap per
// lane): the staging frame (the plane, or its transpose when the line spans
// more columns than rows, so that the line advances by at least one row per
// cell), the cells (duplicate taps merged with their weights added, taps
// that never land in the plane dropped), the strip step s (the most frequent
// row-advancing step between cells), per cell its run offset and weight,
// and the run starts.
//
// Outputs leave through LDS: after the walk the lanes write their blocks
// into the tile (frame orientation, zero outside the plane so that the
// margins stay zero), and the staging lane layout stores them as coalesced
// rows of the plane.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>
#include <utility>

#include "o1d_device.h"
#include "o1d_launch.h"
#include "o1d_strip.h"

namespace o1d {
namespace strip {
namespace {

template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------- program

struct Prog {
  int tr;      // staging frame = transposed plane
  int s;       // strip step u = (1, s) in the staging frame
  int ncells;
  int finite;  // the channel's angle is finite
  int pad0_[4];
  uint32_t brk[2];  // bit c: cell c starts a run
  int pad1_[6];
  int rbase[64];     // run offset of cell c in bytes: 4 (off_c - c st), off_c = a S + b in the frame
  float w[64];       // weight of cell c (duplicate taps summed)
  int tap_cell[64];  // walk cell of every tap, -1 if the tap never lands in the plane
};
static_assert(sizeof(Prog) == kProgWords * 4, "kProgWords must match the program layout");

// OR over the 64 lanes of a wave, returned uniform: an inclusive scan with
// DPP row shifts (1, 2, 4, 8 within rows of 16 lanes), then row broadcasts
// of lanes 15 and 31 into the rows above; lane 63 holds the total.  Lanes
// whose DPP source is outside the row or row mask contribute 0.  All 64
// lanes must be active.
template <class F>
__device__ __forceinline__ uint32_t wave_reduce_dpp(uint32_t v, F op) {
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false));  // row_shr:1
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false));  // row_shr:2
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false));  // row_shr:4
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false));  // row_shr:8
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast:15
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ uint32_t wave_or32(uint32_t v) {
  return wave_reduce_dpp(v, [](uint32_t x, uint32_t y) { return x | y; });
}
// Sum over the 64 lanes (0 is the bit pattern of +0.0f), in a fixed order.
__device__ __forceinline__ float wave_sum(float v) {
  return __uint_as_float(wave_reduce_dpp(__float_as_uint(v), [](uint32_t x, uint32_t y) {
    return __float_as_uint(__uint_as_float(x) + __uint_as_float(y));
  }));
}
__device__ __forceinline__ uint64_t wave_or(uint64_t m) {
  return ((uint64_t)wave_or32((uint32_t)(m >> 32)) << 32) | wave_or32((uint32_t)m);
}
__device__ __forceinline__ uint64_t below_mask(int n) { return n <= 0 ? 0ull : (n >= 64 ? ~0ull : (~0ull >> (64 - n))); }
__device__ __forceinline__ uint64_t above_mask(int n) { return n >= 63 ? 0ull : (~0ull << (n + 1)); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
__device__ __forceinline__ int hibit(uint64_t m) { return m ? 63 - __clzll(m) : -1; }
__device__ __forceinline__ int lobit(uint64_t m) { return m ? __ffsll((long long)m) - 1 : 64; }

// Builds the channel's program.  Called by the 64 lanes of wave 0, lane k =
// tap k (K <= 63).  sign = -1 negates the offsets (input gradient: the
// adjoint of Eq. 1 in x is the same gather with mirrored taps).  Taps move
// monotonically along the line, so taps on one pixel are consecutive (and
// at most two, max(|sin|, |cos|) >= 1/sqrt(2)) and the taps that can land
// in the plane form one contiguous range.
template <typename T>
__device__ void build_prog(Prog* pg, const T* __restrict__ wgt, float theta, int c, int K, int sign, int H, int W,
                           int S) {
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
  // The offsets of Eq. (2) are monotone in k (a floor of a linear function
  // of k, clamped), so their extremes are those of the first and last taps.
  const int h0 = __builtin_amdgcn_readlane(dh, 0), h1 = __builtin_amdgcn_readlane(dh, K - 1);
  const int w0 = __builtin_amdgcn_readlane(dw, 0), w1 = __builtin_amdgcn_readlane(dw, K - 1);
  const int hmin = min(h0, h1), hmax = max(h0, h1), wmin = min(w0, w1), wmax = max(w0, w1);
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

  // cell order: frame rows increasing
  const int lfirst = lobit(cellm), llast = hibit(cellm);
  const int a_first = __builtin_amdgcn_readlane(a, lfirst > 63 ? 0 : lfirst),
            a_last = __builtin_amdgcn_readlane(a, llast < 0 ? 0 : llast);
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

  // walk cell of this lane's cell
  const int cw_idx = co;
  const int st = S + s;
  pg->rbase[k] = 0;
  pg->w[k] = 0.f;
  if (cell && cw_idx >= 0 && cw_idx < 64) {
    pg->rbase[cw_idx] = 4 * ((a * S + b) - cw_idx * st);
    pg->w[cw_idx] = allfin ? cw : __builtin_nanf("");  // a non-finite angle poisons the channel
  }
  const uint64_t brk = wave_or((cell && !cont && cw_idx >= 0 && cw_idx < 64) ? (1ull << cw_idx) : 0ull);
  const int own = dup ? pk : k;  // the lane of the cell that owns this tap
  const int ocw = __shfl(cw_idx, own < 0 ? 0 : own, 64);
  if (act) pg->tap_cell[k] = keep ? ocw : -1;
  if (k == 0) {
    pg->brk[0] = (uint32_t)brk;
    pg->brk[1] = (uint32_t)(brk >> 32);
    pg->ncells = ncells;
    pg->tr = tr ? 1 : 0;
    pg->s = s;
    pg->finite = allfin ? 1 : 0;
  }
}

// Zeroes the group's tile slots with 16-byte stores (slots are a multiple
// of 4 words and start 16-byte aligned).
__device__ __forceinline__ void zero_tiles(const Params& P, float* tiles) {
  float4* t4 = reinterpret_cast<float4*>(tiles);
  const int n4 = (P.G * P.PS) >> 2;
  for (int i = threadIdx.x; i < n4; i += kThreads) t4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

// ---------------------------------------------------------------- walk

__device__ __forceinline__ uint32_t lds_addr(const float* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float*)p;
}
__device__ __forceinline__ float lds_load(uint32_t a) {
  return *(const __attribute__((address_space(3))) float*)(uintptr_t)a;
}
__device__ __forceinline__ void lds_store(uint32_t a, float v) {
  *(__attribute__((address_space(3))) float*)(uintptr_t)a = v;
}
// The value of v, opaque to the optimiser.  A loop-invariant LDS base used
// with constant offsets inside a loop would otherwise be hoisted as one
// precomputed address per offset (a register each); through this the
// offsets stay immediates of the accesses.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// The window step of cell C: a run's first cell reloads all R rows, every
// cell but the walk's last reads the next cell's new row (assuming that cell
// continues the run; a next cell that starts a run reloads every row).  Row
// i, column k of cell C sits at base + 4 ((C + i) ST + k), so the offsets are
// immediates; register row (C + i) mod (R + 1) holds row i.  The run bits
// pass through an empty asm statement so that the test stays a scalar bit
// test inside the walk instead of being hoisted out of the group loop.
template <int R, int NC, int ST, int C, int KB>
__device__ __forceinline__ void window_step(float (&sl)[R + 1][NC], uint32_t& base, uint32_t lb, uint32_t vrb,
                                            uint32_t bits) {
  uint32_t b = bits;
  asm volatile("" : "+s"(b));
  if (b & (1u << (C & 31))) {
    base = lb + (uint32_t)__builtin_amdgcn_readlane((int)vrb, C);
    if constexpr (NC == 1) {
      // One value per row.  Rows i and i + 1 share no base register: loads
      // from one base within 256 words of each other would be paired into
      // 64-bit reads, whose destinations must be an even-aligned register
      // pair, which the rotating rows are not (the pair would land in
      // temporaries and be copied row by row).  Row i reads through base
      // i mod kBases; rows on one base are at least 256 words apart.
      constexpr int kBases = (256 + ST - 1) / ST;
      uint32_t bb[kBases];
#pragma unroll
      for (int m = 0; m < kBases; ++m) bb[m] = opaque(base);
#pragma unroll
      for (int i = 0; i < R; ++i) sl[(C + i) % (R + 1)][0] = lds_load(bb[i % kBases] + 4u * (uint32_t)((C + i) * ST));
    } else {
#pragma unroll
      for (int i = 0; i < R; ++i)
#pragma unroll
        for (int k = 0; k < NC; ++k) sl[(C + i) % (R + 1)][k] = lds_load(base + 4u * (uint32_t)((C + i) * ST + k));
    }
  }
  if constexpr (C + 1 < KB) {
#pragma unroll
    for (int k = 0; k < NC; ++k) sl[(C + R) % (R + 1)][k] = lds_load(base + 4u * (uint32_t)((C + R) * ST + k));
  }
}

// One cell of the gather walk: the window step and the cell's R * NC
// multiplies.
template <int R, int NC, int ST, int C, int KB>
__device__ __forceinline__ void gather_cell(float (&sl)[R + 1][NC], uint32_t& base, uint32_t lb, uint32_t vrb,
                                            uint32_t bits, uint32_t vw, float (&acc)[R][NC]) {
  window_step<R, NC, ST, C, KB>(sl, base, lb, vrb, bits);
  const float wc = __int_as_float(__builtin_amdgcn_readlane((int)vw, C));
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int k = 0; k < NC; ++k) acc[i][k] = fmaf(wc, sl[(C + i) % (R + 1)][k], acc[i][k]);
}

// acc[i][k] += sum over the cells c of w_c * x[cell c + i u + (0, k)]: the
// walk of one block over cells C .. ncells - 1.
template <int R, int NC, int ST, int C, int KB>
struct GatherWalk {
  static __device__ __forceinline__ void run(int n, uint32_t& base, uint32_t lb, uint32_t vrb, uint32_t bits_lo,
                                             uint32_t bits_hi, uint32_t vw, float (&sl)[R + 1][NC],
                                             float (&acc)[R][NC]) {
    // the cell count passes through an empty asm statement, so that the
    // test stays one scalar compare here (instead of a precomputed mask per
    // cell, which costs scalar registers and reads)
    int nn = n;
    asm volatile("" : "+s"(nn));
    if (C >= nn) return;
    gather_cell<R, NC, ST, C, KB>(sl, base, lb, vrb, C < 32 ? bits_lo : bits_hi, vw, acc);
    GatherWalk<R, NC, ST, C + 1, KB>::run(n, base, lb, vrb, bits_lo, bits_hi, vw, sl, acc);
  }
};
template <int R, int NC, int ST, int KB>
struct GatherWalk<R, NC, ST, KB, KB> {
  static __device__ __forceinline__ void run(int, uint32_t&, uint32_t, uint32_t, uint32_t, uint32_t, uint32_t,
                                             float (&)[R + 1][NC], float (&)[R][NC]) {}
};

// One cell of the weight-gradient walk: the same window step, then the
// cell's dot product of the lane's dy block with the window, accumulated
// straight into the cell's sum.
template <int R, int NC, int ST, int C, int KB>
__device__ __forceinline__ void wgrad_cell(float (&sl)[R + 1][NC], uint32_t& base, uint32_t lb, uint32_t vrb,
                                           uint32_t bits, const float (&dv)[R][NC], float (&acc)[KB]) {
  window_step<R, NC, ST, C, KB>(sl, base, lb, vrb, bits);
  float t = acc[C];
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int k = 0; k < NC; ++k) t = fmaf(dv[i][k], sl[(C + i) % (R + 1)][k], t);
  acc[C] = t;
}

// acc[c] += sum over the block of dy * x[cell c + output]: the walk of one
// block over cells C .. ncells - 1 (the weight gradient of Eq. 1).
template <int R, int NC, int ST, int C, int KB>
struct WgradWalk {
  static __device__ __forceinline__ void run(int n, uint32_t& base, uint32_t lb, uint32_t vrb, uint32_t bits_lo,
                                             uint32_t bits_hi, float (&sl)[R + 1][NC], const float (&dv)[R][NC],
                                             float (&acc)[KB]) {
    int nn = n;
    asm volatile("" : "+s"(nn));
    if (C >= nn) return;
    wgrad_cell<R, NC, ST, C, KB>(sl, base, lb, vrb, C < 32 ? bits_lo : bits_hi, dv, acc);
    WgradWalk<R, NC, ST, C + 1, KB>::run(n, base, lb, vrb, bits_lo, bits_hi, sl, dv, acc);
  }
};
template <int R, int NC, int ST, int KB>
struct WgradWalk<R, NC, ST, KB, KB> {
  static __device__ __forceinline__ void run(int, uint32_t&, uint32_t, uint32_t, uint32_t, uint32_t,
                                             float (&)[R + 1][NC], const float (&)[R][NC], float (&)[KB]) {}
};

// One cell of the fused backward walk over dy with the mirrored program:
// the window step, then every window value feeds the lane's input-gradient
// block (times the cell's weight) and the cell's weight-gradient dot
// product (times the lane's x), which accumulates straight into the cell's
// sum: its chain of dependent multiply-adds interleaves with the
// independent input-gradient ones.  KW bounds the walk (its last cell reads
// no next row); acc holds KB >= KW cells.
template <int R, int NC, int ST, int C, int KW, int KB>
__device__ __forceinline__ void bwd_cell(float (&sl)[R + 1][NC], uint32_t& base, uint32_t lb, uint32_t vrb,
                                         uint32_t bits, uint32_t vw, const float (&xv)[R][NC], float (&out)[R][NC],
                                         float (&acc)[KB]) {
  window_step<R, NC, ST, C, KW>(sl, base, lb, vrb, bits);
  const float wc = __int_as_float(__builtin_amdgcn_readlane((int)vw, C));
  float t = acc[C];
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const float v = sl[(C + i) % (R + 1)][k];
      out[i][k] = fmaf(wc, v, out[i][k]);
      t = fmaf(xv[i][k], v, t);
    }
  acc[C] = t;
}

template <int R, int NC, int ST, int C, int KW, int KB>
struct BwdWalk {
  static __device__ __forceinline__ void run(int n, uint32_t& base, uint32_t lb, uint32_t vrb, uint32_t bits_lo,
                                             uint32_t bits_hi, uint32_t vw, float (&sl)[R + 1][NC],
                                             const float (&xv)[R][NC], float (&out)[R][NC], float (&acc)[KB]) {
    int nn = n;
    asm volatile("" : "+s"(nn));
    if (C >= nn) return;
    bwd_cell<R, NC, ST, C, KW, KB>(sl, base, lb, vrb, C < 32 ? bits_lo : bits_hi, vw, xv, out, acc);
    BwdWalk<R, NC, ST, C + 1, KW, KB>::run(n, base, lb, vrb, bits_lo, bits_hi, vw, sl, xv, out, acc);
  }
};
template <int R, int NC, int ST, int KW, int KB>
struct BwdWalk<R, NC, ST, KW, KW, KB> {
  static __device__ __forceinline__ void run(int, uint32_t&, uint32_t, uint32_t, uint32_t, uint32_t, uint32_t,
                                             float (&)[R + 1][NC], const float (&)[R][NC], float (&)[R][NC],
                                             float (&)[KB]) {}
};

// ---------------------------------------------------------------- staging

// Staging of a plane group through registers.  Every lane moves 4
// consecutive elements of a plane row per slot with one 16-byte (bfloat16:
// 8-byte) buffer access.  A half-wave covers 4 rows x 8 quads: lane -> row
// (lane >> 3) & 3 (+4 in the second half-wave, +8 per wave), quad lane & 7.
// For an odd tile row stride the 32 component writes of a half-wave then hit
// 32 distinct banks in either frame.  Slot q = (g, k, m): plane g of the
// group, row step k (8 kWaves rows), column segment m (32 columns).
//
// Every lane runs all kMaxSlots slots (slots past the group read zeros,
// store nothing and write the trash area), so that no register is written
// conditionally.  A lane's slot addresses are computed once per workgroup:
//  * goff[q]: byte offset of its 4 elements from the group's first element,
//    or kOob for a slot outside the plane; buffer accesses beyond the
//    resource's size read zeros and drop stores;
//  * lt(q): LDS address of the first element in the tile (frame orientation),
//    or of the lane's word in the trash area for a slot outside the plane;
//    kept as 16-bit word indices, two slots per register (LDS holds fewer
//    than 2^16 words), which saves kQ / 2 registers through the walk.
constexpr uint32_t kOob = 0x80000000u;

template <int NQ, class F>
__device__ __forceinline__ void for_each_slot(const Params& P, F&& f) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hr = wave * 8 + (lane >> 5) * 4 + ((lane >> 3) & 3);
  const int w0 = 4 * (lane & 7);
  const int per = P.ks * P.ms;
  static_for<NQ>([&](auto qc) __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    const int g = q / per, r = q - g * per, kk = r / P.ms, m = r - kk * P.ms;
    const int h = hr + 8 * kWaves * kk, w = w0 + 32 * m;
    f(q, q < P.nq && g < P.G && h < P.H && w < P.W, g, h, w);
  });
}

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
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float* e) {
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
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float* e) {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    u2 v;
    v[0] = (uint32_t)from_f32<uint16_t>(e[0]) | ((uint32_t)from_f32<uint16_t>(e[1]) << 16);
    v[1] = (uint32_t)from_f32<uint16_t>(e[2]) | ((uint32_t)from_f32<uint16_t>(e[3]) << 16);
    __builtin_amdgcn_raw_buffer_store_b64(v, rs, off, 0, 0);
  }
};

// A buffer resource over `bytes` bytes from p (raw, no swizzle).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

template <typename T>
struct Stage {
  static constexpr int kQ = kMaxSlots;
  static constexpr int kWords = kMaxSlots * Raw<T>::kWords;  // staging registers per group
  static_assert(kQ % 2 == 0, "slots are packed in pairs");
  uint32_t goff[kQ];
  uint32_t ltp[kQ / 2];  // word indices: slot 2 i in the low half, slot 2 i + 1 in the high half

  // LDS byte address of slot q's first element.  The packed pair passes
  // through opaque() so that the unpacking stays next to its use instead
  // of being hoisted out of the group loop into kQ registers.
  __device__ __forceinline__ uint32_t lt(int q) const {
    const uint32_t w = opaque(ltp[q >> 1]);
    return (q & 1) ? (w >> 16) << 2 : (w & 0xffffu) << 2;
  }

  __device__ __forceinline__ void init_global(const Params& P) {
    const int img = P.C * P.H * P.W;
    for_each_slot<kQ>(P, [&](int q, bool ok, int g, int h, int w) __attribute__((always_inline)) {
      goff[q] = ok ? (uint32_t)((g * img + h * P.W + w) * (int)sizeof(T)) : kOob;
    });
  }
  __device__ __forceinline__ void init_lds(const Params& P, int S, bool tr, uint32_t tiles, uint32_t trash) {
    const uint32_t tl = (trash >> 2) + (threadIdx.x & 63);
    for_each_slot<kQ>(P, [&](int q, bool ok, int g, int h, int w) __attribute__((always_inline)) {
      const int r = tr ? w : h, c = tr ? h : w;
      const uint32_t word = ok ? (tiles >> 2) + (uint32_t)(g * P.PS + kGuard + (P.halo + r) * S + P.mc + c) : tl;
      if (q & 1)
        ltp[q >> 1] |= word << 16;
      else
        ltp[q >> 1] = word;
    });
  }
  // Loads the group's slots (ng >= 1 planes from src) into raw registers.
  // ng = 0 reads zeros without touching memory (an empty buffer range).
  __device__ __forceinline__ void load(const Params& P, const T* src, int ng, uint32_t (&v)[kWords]) const {
    const __amdgpu_buffer_rsrc_t rs = buffer_of(src, ng * P.C * P.H * P.W * (int)sizeof(T));
    // every slot, so that each register is written unconditionally (slots
    // past the group read zeros at offset kOob)
#pragma unroll
    for (int q = 0; q < kQ; ++q) Raw<T>::load(rs, goff[q], &v[Raw<T>::kWords * q]);
  }
  // Writes the slots into the tile: the 4 elements of a slot are consecutive
  // along the frame's rows, or along its columns (stride S) when transposed.
  // The frame is uniform, so each branch has a constant step, which the LDS
  // accesses take as immediate offsets (a runtime step would hold 4 kQ
  // precomputed addresses in registers).
  template <int S>
  __device__ __forceinline__ void store_lds(bool tr, const uint32_t (&v)[kWords]) const {
    if (tr)
      store_lds_step<4 * S>(v);
    else
      store_lds_step<4>(v);
  }
  template <int STEP>
  __device__ __forceinline__ void store_lds_step(const uint32_t (&v)[kWords]) const {
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const uint32_t a = lt(q);
#pragma unroll
      for (int j = 0; j < 4; ++j) lds_store(a + j * STEP, Raw<T>::elem(&v[Raw<T>::kWords * q], j));
    }
  }
  // Reads the tile's outputs (frame orientation) in the slot layout.
  template <int S>
  __device__ __forceinline__ void read_lds(bool tr, float (&e)[kQ][4]) const {
    if (tr)
      read_lds_step<4 * S>(e);
    else
      read_lds_step<4>(e);
  }
  template <int STEP>
  __device__ __forceinline__ void read_lds_step(float (&e)[kQ][4]) const {
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const uint32_t a = lt(q);
#pragma unroll
      for (int j = 0; j < 4; ++j) e[q][j] = lds_load(a + j * STEP);
    }
  }
  __device__ __forceinline__ void store(const Params& P, T* dst, int ng, const float (&e)[kQ][4]) const {
    const __amdgpu_buffer_rsrc_t rs = buffer_of(dst, ng * P.C * P.H * P.W * (int)sizeof(T));
#pragma unroll
    for (int q = 0; q < kQ; ++q) Raw<T>::store(rs, goff[q], e[q]);
  }
};

// ---------------------------------------------------------------- forward / input gradient

struct Chan {
  int tr, s, ncells, Hs, Ws;
  uint32_t bits_lo, bits_hi, vrb, vw;
};

// A lane's block of the group: plane g, frame rows b0 .. b0 + R - 1, strip
// columns j0 .. j0 + NC - 1 (strip column j holds the outputs (b0 + i,
// j + SD i)), and the LDS address of its first output in the tile.  Lanes
// without a task point at a real block (their reads stay in the tile).
struct Block {
  int g, b0, j0;
  bool task;  // the lane has a block
  bool full;  // the block lies inside the plane
  uint32_t lb;
};

template <int S, int R, int NC, int SD>
__device__ __forceinline__ Block block_of(const Params& P, const Chan& ch, const float* tiles) {
  const Shape sh = shape_of(ch.Hs, ch.Ws, SD);
  const int t = threadIdx.x;
  int g = t / sh.ppt;
  const int r = t - g * sh.ppt;
  int band, cg;
  if (SD != 0 && sh.split) {
    // blocks: 32 q (nb / 4) lanes per plane; remainder: nb rem lanes per plane
    const int q = sh.ncg >> 3, rem = sh.ncg - 8 * q, nbk = 32 * q * (sh.nb >> 2);
    if (t < nbk * P.G) {
      g = t / nbk;
      const int u = t - g * nbk, blk = u >> 5;
      cg = 8 * (blk % q) + (u & 7);
      band = 4 * (blk / q) + ((u >> 3) & 3);
    } else {
      const int v = t - nbk * P.G, rl = sh.nb * rem;
      g = v / rl;
      const int u = v - g * rl;
      band = u / rem;
      cg = 8 * q + (u - band * rem);
    }
  } else if (SD == 0 || sh.dense) {
    band = r / sh.lpb;
    cg = r - band * sh.lpb;
  } else {
    const int blk = r >> 5, bqi = blk % sh.bq, bbi = blk / sh.bq;
    cg = 8 * bqi + (r & 7);
    band = 4 * bbi + ((r >> 3) & 3);
  }
  Block bk;
  // a lane past its band's last column group reads that group's addresses
  // (a broadcast, no extra bank traffic); lanes past the bands or planes
  // take the first block
  const bool in_band = g < P.G && band < sh.nb;
  bk.task = in_band && cg < sh.ncg;
  bk.g = in_band ? g : 0;
  bk.b0 = in_band ? band * R : 0;
  bk.j0 = in_band ? sh.jlo + min(cg, sh.ncg - 1) * NC : sh.jlo;
  bk.lb = lds_addr(tiles + bk.g * P.PS + kGuard + (P.halo + bk.b0) * S + P.mc + bk.j0);
  const int cmin = bk.j0 + (SD < 0 ? -(R - 1) : 0), cmax = bk.j0 + NC - 1 + (SD > 0 ? R - 1 : 0);
  bk.full = bk.b0 + R <= ch.Hs && cmin >= 0 && cmax < ch.Ws;
  return bk;
}

// Writes a lane's block of outputs into the tile at its own positions,
// zeros for positions outside the plane (the margins stay zero).
template <int R, int NC, int ST, int SD>
__device__ __forceinline__ void put_block(const Block& bk, const Chan& ch, const float (&v)[R][NC]) {
  if (bk.full) {
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) lds_store(bk.lb + 4 * (i * ST + k), v[i][k]);
  } else {
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) {
        const int col = bk.j0 + SD * i + k;
        const bool in = bk.b0 + i < ch.Hs && col >= 0 && col < ch.Ws;
        lds_store(bk.lb + 4 * (i * ST + k), in ? v[i][k] : 0.f);
      }
  }
}

// The group loop of one workgroup for the channel's strip shape (R, NC, SD).
template <typename T, int S, int KB, int R, int NC, int SD>
__device__ __forceinline__ void gather_groups(const Params& P, const Chan& ch, float* smem, const T* inc, T* outc,
                                              int n_begin, int n_end, Stage<T>& stg, uint32_t (&pre)[Stage<T>::kWords]) {
  constexpr int ST = S + SD;
  const size_t img = (size_t)P.C * P.H * P.W;
  float* tiles = smem + kProgWords;
  const Block bk = block_of<S, R, NC, SD>(P, ch, tiles);
  const int g = bk.g;
  const bool task = bk.task;
  const uint32_t lb = bk.lb;

  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    const int ng = min(P.G, n_end - n0);
    // the next group's loads (none past the end: an empty range, so that the
    // prefetch registers are written unconditionally and never copied)
    const int nn = max(0, min(P.G, n_end - n0 - P.G));
    stg.load(P, inc + (size_t)(nn > 0 ? n0 + P.G : n_begin) * img, nn, pre);
    float acc[R][NC];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) acc[i][k] = 0.f;
    // the window's register rows: the walk's first cell loads all of them
    float sl[R + 1][NC];
    uint32_t base = lb;
    GatherWalk<R, NC, ST, 0, KB>::run(ch.ncells, base, lb, ch.vrb, ch.bits_lo, ch.bits_hi, ch.vw, sl, acc);
    __syncthreads();  // every lane has finished reading the tile
    if (task && g < ng) put_block<R, NC, ST, SD>(bk, ch, acc);
    __syncthreads();  // the group's outputs are in the tile
    float e[Stage<T>::kQ][4];
    stg.template read_lds<S>(ch.tr != 0, e);
    __syncthreads();  // the tile is free
    stg.template store_lds<S>(ch.tr != 0, pre);  // past the end: zeros into a tile nobody reads
    stg.store(P, outc + (size_t)n0 * img, ng, e);
    __syncthreads();  // the next group is staged
  }
}

template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads) void strip_gather(Params P, const T* __restrict__ in, const T* __restrict__ wgt,
                                                         const float* __restrict__ theta, T* __restrict__ out) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tiles = smem + kProgWords;
  const int c = blockIdx.y;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t HW = (size_t)P.H * P.W;
  const size_t img = (size_t)P.C * HW;
  const int n_begin = blockIdx.x * P.npw;
  const int n_end = min(P.N, n_begin + P.npw);
  const T* inc = in + (size_t)c * HW;
  T* outc = out + (size_t)c * HW;

  // The first group's loads do not depend on the frame: issue them first.
  Stage<T> stg;
  stg.init_global(P);
  uint32_t pre[Stage<T>::kWords];
  stg.load(P, inc + (size_t)n_begin * img, min(P.G, n_end - n_begin), pre);
  zero_tiles(P, tiles);  // margins and guards stay zero
  if (wave == 0) build_prog<T>(pg, wgt, theta[c], c, P.K, P.sign, P.H, P.W, S);
  __syncthreads();
  Chan ch;
  ch.tr = __builtin_amdgcn_readfirstlane(pg->tr);
  ch.s = __builtin_amdgcn_readfirstlane(pg->s);
  ch.ncells = min(__builtin_amdgcn_readfirstlane(pg->ncells), KB);
  ch.bits_lo = __builtin_amdgcn_readfirstlane(pg->brk[0]);
  ch.bits_hi = __builtin_amdgcn_readfirstlane(pg->brk[1]);
  ch.vrb = (uint32_t)pg->rbase[tid & 63];
  ch.vw = __float_as_uint(pg->w[tid & 63]);
  ch.Hs = ch.tr ? P.W : P.H;
  ch.Ws = ch.tr ? P.H : P.W;
  stg.init_lds(P, S, ch.tr != 0, lds_addr(tiles), lds_addr(smem + P.trash));
  stg.template store_lds<S>(ch.tr != 0, pre);
  __syncthreads();
  if (ch.s == 0)
    gather_groups<T, S, KB, kRv, kNv, 0>(P, ch, smem, inc, outc, n_begin, n_end, stg, pre);
  else if (ch.s > 0)
    gather_groups<T, S, KB, kRd, kNd, 1>(P, ch, smem, inc, outc, n_begin, n_end, stg, pre);
  else
    gather_groups<T, S, KB, kRd, kNd, -1>(P, ch, smem, inc, outc, n_begin, n_end, stg, pre);
}

// ---------------------------------------------------------------- weight gradient

// The group loop of the weight gradient.  Per group the tile first holds dy
// (every lane copies the dy of its block into registers; the tile's zero
// margins give zeros outside the plane), then x, which the lanes walk.  The
// next group's x is prefetched during the walk; dy is loaded at the start
// of its group (one prefetch buffer keeps the registers for the walk).
template <typename T, int S, int KB, int R, int NC, int SD>
__device__ __forceinline__ void wgrad_groups(const Params& P, const Chan& ch, float* smem, const T* xc, const T* dc,
                                             int n_begin, int n_end, Stage<T>& stg,
                                             uint32_t (&xpre)[Stage<T>::kWords], float (&acc)[KB]) {
  constexpr int ST = S + SD;
  const size_t img = (size_t)P.C * P.H * P.W;
  float* tiles = smem + kProgWords;
  const Block bk = block_of<S, R, NC, SD>(P, ch, tiles);
  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    {
      uint32_t dpre[Stage<T>::kWords];
      stg.load(P, dc + (size_t)n0 * img, min(P.G, n_end - n0), dpre);
      stg.template store_lds<S>(ch.tr != 0, dpre);
    }
    __syncthreads();  // dy of the group is in the tile
    float dv[R][NC];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) dv[i][k] = bk.task ? lds_load(bk.lb + 4 * (i * ST + k)) : 0.f;
    __syncthreads();  // every lane has its dy
    stg.template store_lds<S>(ch.tr != 0, xpre);
    __syncthreads();  // x of the group is in the tile
    // the next group's x (past the end: an empty range, see gather_groups)
    const int nn = max(0, min(P.G, n_end - n0 - P.G));
    stg.load(P, xc + (size_t)(nn > 0 ? n0 + P.G : n_begin) * img, nn, xpre);
    float sl[R + 1][NC];
    uint32_t base = bk.lb;
    WgradWalk<R, NC, ST, 0, KB>::run(ch.ncells, base, bk.lb, ch.vrb, ch.bits_lo, ch.bits_hi, sl, dv, acc);
    __syncthreads();  // the tile is free
  }
}

// partial[(blockIdx.x * C + c) * K + k] = the workgroup's sum for tap k:
// lanes -> per-wave cell sums (in `red`, kWaves * 64 floats) -> the cell of
// every tap, in a fixed order (no atomics).  A channel whose angle is not
// finite gets NaN.
template <int KB>
__device__ __forceinline__ void write_partial(const Params& P, const Prog* pg, float* red, int ncells,
                                              const float (&acc)[KB], float* __restrict__ partial) {
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
  for (int ci = 0; ci < KB; ++ci) {
    if (ci < ncells) {
      const float v = wave_sum(acc[ci]);
      if (lane == 0) red[wave * 64 + ci] = v;
    }
  }
  __syncthreads();
  for (int k = tid; k < P.K; k += kThreads) {
    const int ci = pg->tap_cell[k];
    float v = 0.f;
    if (ci >= 0 && ci < KB)
      for (int w = 0; w < kWaves; ++w) v += red[w * 64 + ci];
    partial[((size_t)blockIdx.x * P.C + c) * (size_t)P.K + k] = pg->finite ? v : __builtin_nanf("");
  }
}

// Weight gradient: partial[(blockIdx.x * C + c) * K + k] = sum over the
// workgroup's images of dy * x[tap k + output] (Eq. 1 differentiated in w),
// reduced over lanes and waves in a fixed order (no atomics).
template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads, 2) void strip_wgrad(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                        const float* __restrict__ theta, float* __restrict__ partial) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tiles = smem + kProgWords;
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t HW = (size_t)P.H * P.W;
  const size_t img = (size_t)P.C * HW;
  const int n_begin = blockIdx.x * P.npw;
  const int n_end = min(P.N, n_begin + P.npw);
  const T* xc = x + (size_t)c * HW;
  const T* dc = dy + (size_t)c * HW;

  Stage<T> stg;
  stg.init_global(P);
  uint32_t xpre[Stage<T>::kWords];
  stg.load(P, xc + (size_t)n_begin * img, min(P.G, n_end - n_begin), xpre);
  zero_tiles(P, tiles);  // margins and guards stay zero
  if (wave == 0) build_prog<T>(pg, static_cast<const T*>(nullptr), theta[c], c, P.K, 1, P.H, P.W, S);
  __syncthreads();
  Chan ch;
  ch.tr = __builtin_amdgcn_readfirstlane(pg->tr);
  ch.s = __builtin_amdgcn_readfirstlane(pg->s);
  ch.ncells = min(__builtin_amdgcn_readfirstlane(pg->ncells), KB);
  ch.bits_lo = __builtin_amdgcn_readfirstlane(pg->brk[0]);
  ch.bits_hi = __builtin_amdgcn_readfirstlane(pg->brk[1]);
  ch.vrb = (uint32_t)pg->rbase[lane];
  ch.vw = 0u;
  ch.Hs = ch.tr ? P.W : P.H;
  ch.Ws = ch.tr ? P.H : P.W;
  stg.init_lds(P, S, ch.tr != 0, lds_addr(tiles), lds_addr(smem + P.trash));
  float acc[KB];
#pragma unroll
  for (int i = 0; i < KB; ++i) acc[i] = 0.f;
  if (ch.s == 0)
    wgrad_groups<T, S, KB, kRv, kNv, 0>(P, ch, smem, xc, dc, n_begin, n_end, stg, xpre, acc);
  else if (ch.s > 0)
    wgrad_groups<T, S, KB, kRd, kNd, 1>(P, ch, smem, xc, dc, n_begin, n_end, stg, xpre, acc);
  else
    wgrad_groups<T, S, KB, kRd, kNd, -1>(P, ch, smem, xc, dc, n_begin, n_end, stg, xpre, acc);
  write_partial<KB>(P, pg, smem + P.trash - kWaves * 64, ch.ncells, acc, partial);
}

// ---------------------------------------------------------------- fused backward

// The group loop of the fused backward.  Per group the tile holds x first
// (every lane copies the x of its block into registers; the margins give
// zeros outside the plane), then dy, which the lanes walk with the mirrored
// program: the walk accumulates the lane's input-gradient block and, per
// cell, the dot product of the lane's x with the cell's dy values, which is
// the weight gradient of the cell's taps (Eq. 1 differentiated in w, with
// the output position moved onto x).  The input gradient leaves through
// the tile as in gather_groups.  A group's dy is loaded while the lanes
// copy its x, the next group's x once the lanes have written their input
// gradient blocks (no staging registers stay live through the walk).
template <typename T, int S, int KB, int R, int NC, int SD>
__device__ __forceinline__ void bwd_groups(const Params& P, const Chan& ch, float* smem, const T* xc, const T* dc,
                                           T* dxc, int n_begin, int n_end, Stage<T>& stg,
                                           uint32_t (&pre)[Stage<T>::kWords], float (&acc)[KB]) {
  constexpr int ST = S + SD;
  const size_t img = (size_t)P.C * P.H * P.W;
  float* tiles = smem + kProgWords;
  const Block bk = block_of<S, R, NC, SD>(P, ch, tiles);
  for (int n0 = n_begin; n0 < n_end; n0 += P.G) {
    const int ng = min(P.G, n_end - n0);
    // dy of the group, in flight while the lanes copy x
    stg.load(P, dc + (size_t)n0 * img, ng, pre);
    // the tile holds x of the group
    float xv[R][NC];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) xv[i][k] = bk.task ? lds_load(bk.lb + 4 * (i * ST + k)) : 0.f;
    __syncthreads();  // every lane has its x
    stg.template store_lds<S>(ch.tr != 0, pre);
    __syncthreads();  // dy of the group is in the tile
    // the next group's x (past the end: an empty range, see gather_groups)
    const int nn = max(0, min(P.G, n_end - n0 - P.G));
    const size_t next = (size_t)(nn > 0 ? n0 + P.G : n_begin) * img;
    float out[R][NC];
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int k = 0; k < NC; ++k) out[i][k] = 0.f;
    float sl[R + 1][NC];
    uint32_t base = bk.lb;
    BwdWalk<R, NC, ST, 0, KB - 1, KB>::run(ch.ncells, base, bk.lb, ch.vrb, ch.bits_lo, ch.bits_hi, ch.vw, sl, xv, out,
                                          acc);
    __syncthreads();  // every lane has finished reading the tile
    if (bk.task && bk.g < ng) put_block<R, NC, ST, SD>(bk, ch, out);
    // issued once the block is out of registers (in flight next to the
    // block, the loads would set the kernel's register peak)
    stg.load(P, xc + next, nn, pre);
    __syncthreads();  // the group's input gradient is in the tile
    float e[Stage<T>::kQ][4];
    stg.template read_lds<S>(ch.tr != 0, e);
    __syncthreads();  // the tile is free
    stg.template store_lds<S>(ch.tr != 0, pre);  // past the end: zeros into a tile nobody reads
    stg.store(P, dxc + (size_t)n0 * img, ng, e);
    __syncthreads();  // x of the next group is in the tile
  }
}

// Fused backward: dx (the input gradient, stored like the gather's output)
// and partial[(blockIdx.x * C + c) * K + k] (the workgroup's weight-gradient
// sum of tap k) from one staging of x and dy per plane and one walk.
template <typename T, int S, int KB>
__global__ __launch_bounds__(kThreads) void strip_bwd(Params P, const T* __restrict__ x, const T* __restrict__ dy,
                                                      const T* __restrict__ wgt, const float* __restrict__ theta,
                                                      T* __restrict__ dx, float* __restrict__ partial) {
  extern __shared__ float smem[];
  Prog* pg = reinterpret_cast<Prog*>(smem);
  float* tiles = smem + kProgWords;
  const int c = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t HW = (size_t)P.H * P.W;
  const size_t img = (size_t)P.C * HW;
  const int n_begin = blockIdx.x * P.npw;
  const int n_end = min(P.N, n_begin + P.npw);
  const T* xc = x + (size_t)c * HW;
  const T* dc = dy + (size_t)c * HW;
  T* dxc = dx + (size_t)c * HW;

  Stage<T> stg;
  stg.init_global(P);
  uint32_t pre[Stage<T>::kWords];
  stg.load(P, xc + (size_t)n_begin * img, min(P.G, n_end - n_begin), pre);
  zero_tiles(P, tiles);  // margins and guards stay zero
  if (wave == 0) build_prog<T>(pg, wgt, theta[c], c, P.K, -1, P.H, P.W, S);
  __syncthreads();
  Chan ch;
  ch.tr = __builtin_amdgcn_readfirstlane(pg->tr);
  ch.s = __builtin_amdgcn_readfirstlane(pg->s);
  // odd K <= KB: at most KB - 1 cells
  ch.ncells = min(__builtin_amdgcn_readfirstlane(pg->ncells), KB - 1);
  ch.bits_lo = __builtin_amdgcn_readfirstlane(pg->brk[0]);
  ch.bits_hi = __builtin_amdgcn_readfirstlane(pg->brk[1]);
  ch.vrb = (uint32_t)pg->rbase[lane];
  ch.vw = __float_as_uint(pg->w[lane]);
  ch.Hs = ch.tr ? P.W : P.H;
  ch.Ws = ch.tr ? P.H : P.W;
  stg.init_lds(P, S, ch.tr != 0, lds_addr(tiles), lds_addr(smem + P.trash));
  stg.template store_lds<S>(ch.tr != 0, pre);
  __syncthreads();  // x of the first group is in the tile
  float acc[KB];
#pragma unroll
  for (int i = 0; i < KB; ++i) acc[i] = 0.f;
  if (ch.s == 0)
    bwd_groups<T, S, KB, kRv, kNv, 0>(P, ch, smem, xc, dc, dxc, n_begin, n_end, stg, pre, acc);
  else if (ch.s > 0)
    bwd_groups<T, S, KB, kRd, kNd, 1>(P, ch, smem, xc, dc, dxc, n_begin, n_end, stg, pre, acc);
  else
    bwd_groups<T, S, KB, kRd, kNd, -1>(P, ch, smem, xc, dc, dxc, n_begin, n_end, stg, pre, acc);
  write_partial<KB>(P, pg, smem + P.trash - kWaves * 64, ch.ncells, acc, partial);
}

// ---------------------------------------------------------------- launch

// Fits the grid to `per_cu` resident workgroups on every CU of the device.
inline void fit_grid(Plan& pl, int per_cu) {
  static std::atomic<int> cu_count{0};
  int cus = cu_count.load(std::memory_order_relaxed);
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) ==
                                                 hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
    cu_count.store(cus, std::memory_order_relaxed);
  }
  pl.p.npw = fit_npw(pl.p.N, pl.p.C, pl.p.G, (long long)cus * (per_cu < 1 ? 1 : per_cu));
  pl.blocks_n = cdiv(pl.p.N, pl.p.npw);
}

// Resident workgroups per CU of strip_gather<T, S, KB> for a dynamic LDS
// size.  The answer is cached per instantiation (the queries cost more host
// time than a launch), packed with its LDS size into one atomic word.
template <typename T, int S, int KB>
hipError_t resident_per_cu(size_t lds_bytes, int* per_cu) {
  static std::atomic<unsigned long long> cache{0};
  const unsigned long long c = cache.load(std::memory_order_relaxed);
  if (c != 0 && (c >> 8) == lds_bytes) {
    *per_cu = (int)(c & 0xff);
    return hipSuccess;
  }
  const void* fn = reinterpret_cast<const void*>(strip_gather<T, S, KB>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLdsBytes);
  if (e != hipSuccess) return e;
  hipFuncAttributes fa;
  e = hipFuncGetAttributes(&fa, fn);
  if (e != hipSuccess) return e;
  // Residency from the kernel's resources: waves per SIMD from its VGPRs
  // (512 per lane, granules of 8, at most 8 waves), and the LDS rule of
  // lds_resident.
  const int vg = ((fa.numRegs > 0 ? fa.numRegs : 1) + 7) / 8 * 8;
  int waves = 512 / vg;
  if (waves > 8) waves = 8;
  int n = 4 * waves / kWaves;
  const int by_lds = lds_resident(lds_bytes);
  if (by_lds < n) n = by_lds;
  n = n < 1 ? 1 : (n > 255 ? 255 : n);
  cache.store(((unsigned long long)lds_bytes << 8) | (unsigned long long)n, std::memory_order_relaxed);
  *per_cu = n;
  return hipSuccess;
}

// Raises a kernel's dynamic LDS limit to the whole LDS once per process
// (the first launch of each instantiation pays for the runtime call).
template <const void* (*Fn)()>
hipError_t allow_full_lds() {
  static std::atomic<int> done{0};
  if (done.load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(Fn(), hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLdsBytes);
  if (e == hipSuccess) done.store(1, std::memory_order_release);
  return e;
}
template <typename T, int S, int KB>
const void* wgrad_fn() { return reinterpret_cast<const void*>(strip_wgrad<T, S, KB>); }
template <typename T, int S, int KB>
const void* bwd_fn() { return reinterpret_cast<const void*>(strip_bwd<T, S, KB>); }

template <typename T, int S, int KB>
hipError_t gather_launch(const Plan& plan, const void* in, const void* w, const float* theta, void* out,
                         hipStream_t stream) {
  int per_cu = 0;
  hipError_t e = resident_per_cu<T, S, KB>(plan.lds_bytes, &per_cu);
  if (e != hipSuccess) return e;
  Plan pl = plan;
  fit_grid(pl, per_cu);
  hipLaunchKernelGGL((strip_gather<T, S, KB>), dim3((unsigned)pl.blocks_n, (unsigned)pl.p.C, 1), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(in), static_cast<const T*>(w), theta,
                     static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int S, int KB>
hipError_t wgrad_launch(const Plan& pl, const void* x, const void* dy, const float* theta, float* partial,
                        hipStream_t stream) {
  const hipError_t e = allow_full_lds<wgrad_fn<T, S, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((strip_wgrad<T, S, KB>), dim3((unsigned)pl.blocks_n, (unsigned)pl.p.C, 1), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(x), static_cast<const T*>(dy), theta, partial);
  return hipGetLastError();
}

template <typename T, int KB>
hipError_t wgrad_t(const Plan& pl, const void* x, const void* dy, const float* theta, void* dw, float* partial,
                   hipStream_t stream) {
  hipError_t e = hipErrorInvalidValue;
#define O1D_CASE(SV) \
  if (pl.S == SV) e = wgrad_launch<T, SV, KB>(pl, x, dy, theta, partial, stream);
  O1D_STRIP_STRIDES(O1D_CASE)
#undef O1D_CASE
  if (e != hipSuccess) return e;
  return launch_partial_sum(std::is_same<T, float>::value ? Dtype::F32 : Dtype::BF16, partial, dw, pl.p.C * pl.p.K,
                            pl.blocks_n, stream);
}

template <typename T, int S, int KB>
hipError_t bwd_launch(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx,
                      float* partial, hipStream_t stream) {
  const hipError_t e = allow_full_lds<bwd_fn<T, S, KB>>();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((strip_bwd<T, S, KB>), dim3((unsigned)pl.blocks_n, (unsigned)pl.p.C, 1), dim3(kThreads),
                     pl.lds_bytes, stream, pl.p, static_cast<const T*>(x), static_cast<const T*>(dy),
                     static_cast<const T*>(w), theta, static_cast<T*>(dx), partial);
  return hipGetLastError();
}

template <typename T, int KB>
hipError_t bwd_t(const Plan& pl, const void* x, const void* dy, const void* w, const float* theta, void* dx,
                 void* dw, float* partial, hipStream_t stream) {
  hipError_t e = hipErrorInvalidValue;
#define O1D_CASE(SV) \
  if (pl.S == SV) e = bwd_launch<T, SV, KB>(pl, x, dy, w, theta, dx, partial, stream);
  O1D_STRIP_STRIDES(O1D_CASE)
#undef O1D_CASE
  if (e != hipSuccess) return e;
  return launch_partial_sum(std::is_same<T, float>::value ? Dtype::F32 : Dtype::BF16, partial, dw, pl.p.C * pl.p.K,
                            pl.blocks_n, stream);
}

template <typename T, int KB>
hipError_t gather_t(const Plan& pl, const void* in, const void* w, const float* theta, void* out,
                    hipStream_t stream) {
#define O1D_CASE(SV) \
  if (pl.S == SV) return gather_launch<T, SV, KB>(pl, in, w, theta, out, stream);
  O1D_STRIP_STRIDES(O1D_CASE)
#undef O1D_CASE
  return hipErrorInvalidValue;
}

}  // namespace
}  // namespace strip
}  // namespace o1d
