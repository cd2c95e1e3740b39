"""Hilbert-curve block organisation (oracle side; test infrastructure).

The routing frontend of §3.1 may reorder blocks along a Hilbert curve, so
that tokens that are close in the latent video land in blocks that are
close too, at every scale of the curve. The reading taken here:

* the curve is the 3D Hilbert curve of J. Skilling ("Programming the
  Hilbert curve", AIP Conf. Proc. 707, 2004) on the cube of side 2^k, k the
  smallest integer with 2^k >= max(T, H, W); a token (t, y, x) is the
  point with coordinates (X0, X1, X2) = (t, y, x), and X0 contributes the
  most significant bit of every 3-bit digit of the curve index;
* the tokens of the T x H x W grid are ranked by their curve index (points
  of the cube outside the grid are skipped), and the sequence of ranked
  tokens is cut into consecutive runs of B tokens: block i holds ranks
  [iB, min((i+1)B, N)), so only the last block can be partial.

Skilling's method turns the coordinates into the "transposed" form of the
index in two passes, an inverse undo over the bit levels from the top and a
Gray encoding, and the index is then the bit interleave of that form. The
steps below follow that description; they are vectorised over points with
numpy and share nothing with the GPU library.
"""

import numpy as np

from .tiling import TileGeometry


def curve_bits(T: int, H: int, W: int) -> int:
    """Smallest k with 2^k >= max(T, H, W) (0 for a single token)."""
    m = max(int(T), int(H), int(W))
    if m <= 0:
        raise ValueError("grid extents must be positive")
    return int(m - 1).bit_length()


def hilbert_index(coords, bits: int) -> np.ndarray:
    """Curve index of every point of `coords` (int array [..., 3], each in [0, 2^bits))."""
    X = np.array(coords, dtype=np.int64, copy=True)
    if X.shape[-1] != 3:
        raise ValueError("points must have three coordinates")
    if bits == 0:
        return np.zeros(X.shape[:-1], dtype=np.int64)
    if X.min(initial=0) < 0 or X.max(initial=0) >= (1 << bits):
        raise ValueError("coordinate outside the cube")
    top = 1 << (bits - 1)
    # Inverse undo, from the top bit level down to level 1: where axis i has
    # the level's bit set, the lower bits of X0 are inverted; otherwise the
    # lower bits of X0 and Xi are exchanged.
    q = top
    while q > 1:
        low = q - 1
        for i in range(3):
            bit_set = (X[..., i] & q) != 0
            if i == 0:
                X[..., 0] = np.where(bit_set, X[..., 0] ^ low, X[..., 0])
                continue
            swap = (X[..., 0] ^ X[..., i]) & low
            swap = np.where(bit_set, 0, swap)
            x0 = np.where(bit_set, X[..., 0] ^ low, X[..., 0] ^ swap)
            X[..., i] = X[..., i] ^ swap
            X[..., 0] = x0
        q >>= 1
    # Gray encode: prefix XOR over the axes, then the correction taken from
    # the last axis's bits above level 0.
    X[..., 1] ^= X[..., 0]
    X[..., 2] ^= X[..., 1]
    fix = np.zeros(X.shape[:-1], dtype=np.int64)
    q = top
    while q > 1:
        fix ^= np.where((X[..., 2] & q) != 0, q - 1, 0)
        q >>= 1
    X ^= fix[..., None]
    # Interleave: for every level from the top, bits of X0, X1, X2.
    h = np.zeros(X.shape[:-1], dtype=np.int64)
    for b in range(bits - 1, -1, -1):
        for i in range(3):
            h = (h << 1) | ((X[..., i] >> b) & 1)
    return h


def curve_order(T: int, H: int, W: int) -> np.ndarray:
    """perm[r] = raster token id (t*H + y)*W + x of the token of curve rank r."""
    bits = curve_bits(T, H, W)
    t, y, x = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    pts = np.stack([t.ravel(), y.ravel(), x.ravel()], axis=-1)
    key = hilbert_index(pts, bits)
    return np.argsort(key, kind="stable").astype(np.int64)


def curve_geometry(T: int, H: int, W: int, B: int) -> TileGeometry:
    """Blocks of B consecutive curve ranks over a T x H x W grid.

    block_tokens[i] lists raster token ids in curve order. The box fields
    describe the one-dimensional tiling of the curve-ordered sequence:
    (bt, bh, bw) = (1, 1, B) and (nbt, nby, nbx) = (1, 1, nb).
    """
    for v in (T, H, W, B):
        if int(v) <= 0:
            raise ValueError("grid extents and block size must be positive")
    perm = curve_order(T, H, W)
    N = T * H * W
    nb = -(-N // B)
    rank_block = np.arange(N, dtype=np.int64) // B
    block_of_token = np.empty(N, dtype=np.int64)
    block_of_token[perm] = rank_block
    sizes = np.bincount(rank_block, minlength=nb).astype(np.int64)
    tokens = tuple(perm[i * B : min((i + 1) * B, N)] for i in range(nb))
    return TileGeometry(T, H, W, 1, 1, B, 1, 1, nb, block_of_token, sizes, tokens, order="hilbert")
