// Host-side launch planning shared by the C ABI and the kernel launchers.
// Everything here depends only on (N, C, H, W, K, dtype), never on device
// data, so the workspace size reported to callers always matches what the
// launch uses.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace o1d {

constexpr int kThreads = 256;
constexpr size_t kMaxLdsBytes = 160 * 1024;  // gfx950 LDS per workgroup

// Tiled gather / weight-gradient plan: the plane is cut into BH x BW output
// tiles; a tile stages (BH + 2 pad) x (BW + 2 pad) inputs in LDS.
struct TilePlan {
  int BH = 0, BW = 0;
  int tiles_x = 0, tiles_y = 0;
  size_t lds_bytes = 0;
  int tiles() const { return tiles_x * tiles_y; }
};

inline size_t tile_lds_bytes(int BH, int BW, int K, int extra_floats) {
  const int pad = K / 2;
  return ((size_t)(BH + 2 * pad) * (size_t)(BW + 2 * pad) + 2 * (size_t)K + (size_t)extra_floats) * 4u;
}

inline TilePlan plan_tiles(int H, int W, int K, int extra_floats) {
  TilePlan p;
  p.BH = H < 64 ? H : 64;
  p.BW = W < 64 ? W : 64;
  while (tile_lds_bytes(p.BH, p.BW, K, extra_floats) > kMaxLdsBytes && (p.BH > 1 || p.BW > 1)) {
    if (p.BH >= p.BW && p.BH > 1)
      p.BH = (p.BH + 1) / 2;
    else
      p.BW = (p.BW + 1) / 2;
  }
  p.tiles_x = (W + p.BW - 1) / p.BW;
  p.tiles_y = (H + p.BH - 1) / p.BH;
  p.lds_bytes = tile_lds_bytes(p.BH, p.BW, K, extra_floats);
  return p;
}

// Weight-gradient split: every (tile, n-chunk) of a channel writes one row
// of K float32 partial sums; a second kernel sums them in a fixed order.
struct WgradPlan {
  TilePlan tile;
  int kb = 0;       // taps accumulated per pass (register block)
  int nchunk = 0;   // number of batch chunks
  int npc = 0;      // images per chunk
  size_t parts() const { return (size_t)nchunk * (size_t)tile.tiles(); }
};

inline int wgrad_tap_block(int K) { return K <= 16 ? 16 : (K <= 32 ? 32 : 64); }

inline WgradPlan plan_wgrad(int N, int C, int H, int W, int K) {
  WgradPlan p;
  p.kb = wgrad_tap_block(K);
  p.tile = plan_tiles(H, W, K, 4 * p.kb);
  const long long blocks_per_chunk = (long long)p.tile.tiles() * (long long)C;
  long long want = (2048 + blocks_per_chunk - 1) / blocks_per_chunk;
  if (want < 1) want = 1;
  if (want > N) want = N;
  p.npc = (int)((N + want - 1) / want);
  p.nchunk = (N + p.npc - 1) / p.npc;
  return p;
}

}  // namespace o1d
