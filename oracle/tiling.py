"""Video-aware 3D block tiling (oracle side).

The paper groups spatially and temporally adjacent latent tokens into blocks
(§3.1, routing frontend; the abstract calls it video-aware block
organisation). The reading used here:

* tokens of a T x H x W latent grid are flattened in raster order,
  n = (t*H + y)*W + x;
* a block is a bt x bh x bw box of the grid, boxes anchored at the origin,
  so a partial box can only be the last one along an axis;
* block ids are raster order over the box grid (nbt, nby, nbx);
* a block holds only real tokens: n_i is the product of the box's
  in-grid extents, never the full box volume.

Written from those definitions with per-axis floor division; nothing here is
shared with the GPU library.
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class TileGeometry:
    T: int
    H: int
    W: int
    bt: int
    bh: int
    bw: int
    nbt: int
    nby: int
    nbx: int
    block_of_token: np.ndarray  # int64 [N]: block id of every token
    block_sizes: np.ndarray  # int64 [nb]: real tokens per block
    block_tokens: tuple  # nb arrays of token ids (ascending for boxes, curve order otherwise)
    order: str = "box"  # "box": 3D boxes; "hilbert": runs of a Hilbert curve (oracle.curve)

    @property
    def N(self) -> int:
        return self.T * self.H * self.W

    @property
    def nb(self) -> int:
        return self.nbt * self.nby * self.nbx


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def tile_geometry(T: int, H: int, W: int, bt: int, bh: int, bw: int) -> TileGeometry:
    """Assign every token of a T x H x W grid to its bt x bh x bw block."""
    for v in (T, H, W, bt, bh, bw):
        if int(v) <= 0:
            raise ValueError("grid and tile extents must be positive")
    nbt, nby, nbx = _ceil_div(T, bt), _ceil_div(H, bh), _ceil_div(W, bw)
    t = np.arange(T).reshape(T, 1, 1)
    y = np.arange(H).reshape(1, H, 1)
    x = np.arange(W).reshape(1, 1, W)
    blk = ((t // bt) * nby + (y // bh)) * nbx + (x // bw)
    block_of_token = np.broadcast_to(blk, (T, H, W)).reshape(-1).astype(np.int64)
    nb = nbt * nby * nbx
    sizes = np.bincount(block_of_token, minlength=nb).astype(np.int64)
    order = np.argsort(block_of_token, kind="stable")  # ascending token ids per block
    bounds = np.concatenate([[0], np.cumsum(sizes)])
    tokens = tuple(order[bounds[i] : bounds[i + 1]] for i in range(nb))
    return TileGeometry(T, H, W, bt, bh, bw, nbt, nby, nbx, block_of_token, sizes, tokens)
