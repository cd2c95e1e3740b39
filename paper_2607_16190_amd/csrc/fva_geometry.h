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
