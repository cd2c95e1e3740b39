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

// Query-block pairs. Two x-neighbouring blocks (ix, ix + 1), ix even, of the
// same (t, y) line are one pair when both hold at most 64 real tokens; the
// attention then runs them as one 128-row work item (each block on two
// waves) that stages every key block kept by either once. Block ix is not the
// last of its line, so its x extent is bw and block ix + 1 is no larger: a
// line pairs all its floor(nbx / 2) pairs or none, decided by et * ey * bw.
__host__ __device__ inline bool line_pairs(const Geometry& g, int et, int ey) { return et * ey * g.bw <= 64; }

// Lines of t-row it (extent et) that pair.
__host__ __device__ inline int paired_lines_of_row(const Geometry& g, int et) {
  const int ey_last = g.H - (g.nby - 1) * g.bh;
  return (g.nby - 1) * (line_pairs(g, et, g.bh) ? 1 : 0) + (line_pairs(g, et, ey_last) ? 1 : 0);
}

// Pairs in one head (every head has the same).
__host__ __device__ inline int pairs_per_head(const Geometry& g) {
  const int et_last = g.T - (g.nbt - 1) * g.bt;
  const int lines = (g.nbt - 1) * paired_lines_of_row(g, g.bt) + paired_lines_of_row(g, et_last);
  return lines * (g.nbx / 2);
}

// Slot of the pair whose first block is i within its head (pairs numbered in
// raster order of their first block), or -1 when i does not start a pair.
__host__ __device__ inline int pair_slot(const Geometry& g, int i) {
  const int it = i / (g.nby * g.nbx);
  const int rem = i - it * (g.nby * g.nbx);
  const int iy = rem / g.nbx;
  const int ix = rem - iy * g.nbx;
  const int et = min(g.bt, g.T - it * g.bt);
  const int ey = min(g.bh, g.H - iy * g.bh);
  if ((ix & 1) || ix + 1 >= g.nbx || !line_pairs(g, et, ey)) return -1;
  // t-rows before it are full in t, lines before iy in this row full in y
  const int lines_before = it * paired_lines_of_row(g, g.bt) + iy * (line_pairs(g, et, g.bh) ? 1 : 0);
  return lines_before * (g.nbx / 2) + ix / 2;
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
