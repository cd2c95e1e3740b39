// Tile geometry shared by the host launchers and the gfx950 kernels.
//
// A block is a bt x bh x bw box of the T x H x W latent grid, boxes anchored
// at the origin; block ids are raster order over the box grid. Inside a block
// the real tokens are packed in local raster order (lt, ly, lx), so local
// index r < n_i maps to global token ((t0+lt)*H + y0+ly)*W + x0+lx. Kernels
// never touch padding tokens.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fva {

constexpr int kHeadDim = 128;
constexpr int kMaxBlocks = 1024;
constexpr int kMaxTile = 128;
constexpr int kV8TileBytes = 128 * 128;  // one block of E4M3 V^T: 128 channels x 128 key positions

struct Geometry {
  int T, H, W;
  int bt, bh, bw;
  int nbt, nby, nbx, nb;
};

struct BlockBox {
  int t0, y0, x0;   // origin of the box
  int et, ey, ex;   // in-grid extents
  int n;            // real tokens = et*ey*ex
};

__host__ __device__ inline Geometry make_geometry(int T, int H, int W, int bt, int bh, int bw) {
  Geometry g;
  g.T = T; g.H = H; g.W = W; g.bt = bt; g.bh = bh; g.bw = bw;
  g.nbt = (T + bt - 1) / bt;
  g.nby = (H + bh - 1) / bh;
  g.nbx = (W + bw - 1) / bw;
  g.nb = g.nbt * g.nby * g.nbx;
  return g;
}

__host__ __device__ inline BlockBox block_box(const Geometry& g, int i) {
  BlockBox b;
  const int it = i / (g.nby * g.nbx);
  const int rem = i - it * (g.nby * g.nbx);
  const int iy = rem / g.nbx;
  const int ix = rem - iy * g.nbx;
  b.t0 = it * g.bt; b.y0 = iy * g.bh; b.x0 = ix * g.bw;
  b.et = min(g.bt, g.T - b.t0);
  b.ey = min(g.bh, g.H - b.y0);
  b.ex = min(g.bw, g.W - b.x0);
  b.n = b.et * b.ey * b.ex;
  return b;
}

// Query-block pairs: two neighbouring blocks that both hold at most 64 real
// tokens, run by the attention as one 128-row work item (each block on two
// waves) that stages every key block kept by either once.
//  * x-pairs: (ix, ix + 1), ix even, of one (t, y) line. Block ix is not the
//    last of its line, so its x extent is bw and block ix + 1 is no larger:
//    a line pairs all its floor(nbx / 2) pairs or none (et * ey * bw <= 64).
//  * y-pairs, among the blocks no x-pair holds (the lines that do not pair,
//    and the last block of a pairing line when nbx is odd): (iy, iy + 1),
//    iy even, of one (t, x) column, both holding at most 64 tokens.
// pair_partner(g, i) is the block-id offset of i's partner: +1 or +nbx when
// i starts a pair, -1 or -nbx when it is the second block, 0 otherwise.
// Pairs are numbered per head in the order of their first block.
__host__ __device__ inline int block_tokens(const Geometry& g, int it, int iy, int ix) {
  return min(g.bt, g.T - it * g.bt) * min(g.bh, g.H - iy * g.bh) * min(g.bw, g.W - ix * g.bw);
}

// Block (it, iy, ix) belongs to an x-pair.
__host__ __device__ inline bool in_x_pair(const Geometry& g, int it, int iy, int ix) {
  const int et = min(g.bt, g.T - it * g.bt);
  const int ey = min(g.bh, g.H - iy * g.bh);
  return et * ey * g.bw <= 64 && ix < 2 * (g.nbx / 2);
}

// y-pair (iy, iy + 1) starting at (it, iy, ix), iy even.
__host__ __device__ inline bool y_pair_at(const Geometry& g, int it, int iy, int ix) {
  return iy + 1 < g.nby && !in_x_pair(g, it, iy, ix) && !in_x_pair(g, it, iy + 1, ix) &&
         block_tokens(g, it, iy, ix) <= 64 && block_tokens(g, it, iy + 1, ix) <= 64;
}

__host__ __device__ inline int pair_partner(const Geometry& g, int i) {
  const int it = i / (g.nby * g.nbx);
  const int rem = i - it * (g.nby * g.nbx);
  const int iy = rem / g.nbx;
  const int ix = rem - iy * g.nbx;
  if (in_x_pair(g, it, iy, ix)) return (ix & 1) ? -1 : 1;
  if (!(iy & 1) && y_pair_at(g, it, iy, ix)) return g.nbx;
  if ((iy & 1) && y_pair_at(g, it, iy - 1, ix)) return -g.nbx;
  return 0;
}

// Pairs in one head (every head has the same).
__host__ __device__ inline int pairs_per_head(const Geometry& g) {
  int n = 0;
  for (int i = 0; i < g.nb; ++i) n += pair_partner(g, i) > 0 ? 1 : 0;
  return n;
}

// Global token index of the r-th real token (local raster order) of a box.
__host__ __device__ inline int box_token(const Geometry& g, const BlockBox& b, int r) {
  const int plane = b.ey * b.ex;
  const int lt = r / plane;
  const int rem = r - lt * plane;
  const int ly = rem / b.ex;
  const int lx = rem - ly * b.ex;
  return ((b.t0 + lt) * g.H + (b.y0 + ly)) * g.W + (b.x0 + lx);
}

}  // namespace fva
