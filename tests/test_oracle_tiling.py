"""Pins of the oracle's 3D block tiling (video-aware block organisation, §3.1).

Checked against closed forms that do not use the oracle's own code path:
block counts from per-axis ceilings, the set of block sizes from per-axis
extents, per-size multiplicities, and brute-force coordinate checks.
"""

import itertools

import numpy as np
import pytest

from oracle import tile_geometry

WORKLOADS = {
    # name: (grid, tile, nb, padded N, block-size set)
    "tiny": ((3, 16, 16), (1, 8, 8), 12, 768, {64}),
    "480p": ((21, 30, 52), (2, 8, 8), 308, 39424, {24, 32, 48, 64, 96, 128}),
    "720p": ((21, 45, 80), (2, 8, 8), 660, 84480, {40, 64, 80, 128}),
    "long": ((31, 45, 80), (2, 8, 8), 960, 122880, {40, 64, 80, 128}),
}


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_block_counts_and_sizes(name):
    grid, tile, nb, n_pad, sizes = WORKLOADS[name]
    geo = tile_geometry(*grid, *tile)
    assert geo.nb == nb
    assert geo.nb * int(np.prod(tile)) == n_pad
    assert set(geo.block_sizes.tolist()) == sizes
    assert int(geo.block_sizes.sum()) == int(np.prod(grid))
    # every token in exactly one block
    allt = np.concatenate(geo.block_tokens)
    assert np.array_equal(np.sort(allt), np.arange(geo.N))


def test_720p_size_multiplicities():
    # 21 frames -> 10 full time-slabs + 1 single frame; 45 rows -> 5 full + 1 of 5; 80 cols -> 10 full.
    geo = tile_geometry(21, 45, 80, 2, 8, 8)
    counts = {s: int((geo.block_sizes == s).sum()) for s in (128, 80, 64, 40)}
    assert counts == {128: 10 * 5 * 10, 80: 10 * 1 * 10, 64: 1 * 5 * 10, 40: 1 * 1 * 10}


def test_partial_tiles_brute_force():
    T, H, W, bt, bh, bw = 3, 5, 7, 2, 2, 4
    geo = tile_geometry(T, H, W, bt, bh, bw)
    assert (geo.nbt, geo.nby, geo.nbx) == (2, 3, 2)
    for t, y, x in itertools.product(range(T), range(H), range(W)):
        n = (t * H + y) * W + x
        blk = ((t // bt) * 3 + y // bh) * 2 + x // bw
        assert geo.block_of_token[n] == blk
    for i, toks in enumerate(geo.block_tokens):
        it, iy, ix = i // 6, (i // 2) % 3, i % 2
        et = min(bt, T - it * bt)
        ey = min(bh, H - iy * bh)
        ex = min(bw, W - ix * bw)
        assert len(toks) == et * ey * ex
        assert np.all(np.diff(toks) > 0)  # ascending token order


def test_rejects_bad_extents():
    with pytest.raises(ValueError):
        tile_geometry(0, 4, 4, 1, 2, 2)
