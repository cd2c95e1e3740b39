"""Pins of the oracle's Hilbert-curve block organisation (§3.1, routing frontend).

The curve index is checked against what defines a Hilbert curve rather than
against its own formula: on every cube up to 16^3 it is a bijection onto
0 .. 8^k - 1, consecutive indices are unit steps (the curve is continuous),
and every aligned run of 8^m indices fills an aligned cube of side 2^m (the
self-similarity that keeps neighbours together at every scale). The block
partition is checked by counting, and on a cube grid whose blocks are whole
sub-cubes the routing and attention results must equal those of the 3D box
tiling with the same sub-cubes, up to the numbering of the blocks.
"""

import itertools

import numpy as np
import pytest

from oracle import (
    attn_ref_head,
    curve_bits,
    curve_geometry,
    curve_order,
    hilbert_index,
    route_ref,
    tile_geometry,
)


def cube_path(bits):
    n = 1 << bits
    pts = np.array(list(itertools.product(range(n), repeat=3)), dtype=np.int64)
    h = hilbert_index(pts, bits)
    path = np.empty_like(pts)
    path[h] = pts
    return h, path


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_curve_is_a_bijection(bits):
    h, _ = cube_path(bits)
    assert np.array_equal(np.sort(h), np.arange(8**bits))


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_curve_moves_by_unit_steps(bits):
    _, path = cube_path(bits)
    step = np.abs(np.diff(path, axis=0))
    assert np.all(step.sum(axis=1) == 1)  # one axis changes, by one
    assert np.array_equal(path[0], [0, 0, 0])


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_curve_fills_aligned_cubes_at_every_scale(bits):
    _, path = cube_path(bits)
    for m in range(1, bits):
        s = 1 << m
        seg = path.reshape(-1, s**3, 3)
        lo, hi = seg.min(axis=1), seg.max(axis=1)
        assert np.all(lo % s == 0), m
        assert np.all(hi - lo == s - 1), m


def test_curve_bits():
    assert curve_bits(1, 1, 1) == 0
    assert curve_bits(3, 16, 16) == 4
    assert curve_bits(21, 45, 80) == 7
    assert curve_bits(2, 129, 3) == 8
    assert hilbert_index(np.zeros((4, 3), dtype=np.int64), 0).tolist() == [0, 0, 0, 0]


def test_order_of_a_partial_grid_follows_the_cube_path():
    # Walk the whole 8^3 path and keep the points inside a 3 x 5 x 7 grid.
    T, H, W = 3, 5, 7
    _, path = cube_path(3)
    inside = (path[:, 0] < T) & (path[:, 1] < H) & (path[:, 2] < W)
    expect = [(t * H + y) * W + x for t, y, x in path[inside]]
    assert curve_order(T, H, W).tolist() == expect


@pytest.mark.parametrize("grid,B", [((21, 45, 80), 128), ((21, 30, 52), 128), ((3, 16, 16), 64), ((2, 3, 5), 7)])
def test_curve_blocks_partition_the_tokens(grid, B):
    geo = curve_geometry(*grid, B)
    N = int(np.prod(grid))
    assert geo.nb == -(-N // B)
    assert np.all(geo.block_sizes[:-1] == B)
    assert geo.block_sizes[-1] == N - (geo.nb - 1) * B
    allt = np.concatenate(geo.block_tokens)
    assert np.array_equal(np.sort(allt), np.arange(N))
    for i, toks in enumerate(geo.block_tokens):
        assert np.all(geo.block_of_token[toks] == i)


def test_cube_blocks_equal_box_tiling():
    # On an 8^3 grid with 64-token blocks every block is an aligned 4^3 cube,
    # so the curve blocks are the 4x4x4 boxes in another order.
    cg = curve_geometry(8, 8, 8, 64)
    bg = tile_geometry(8, 8, 8, 4, 4, 4)
    box_of = {tuple(np.sort(t)): j for j, t in enumerate(bg.block_tokens)}
    perm = np.array([box_of[tuple(np.sort(t))] for t in cg.block_tokens])
    assert np.array_equal(np.sort(perm), np.arange(8))

    rng = np.random.default_rng(7)
    d = 16
    emb = rng.standard_normal((512, d))
    Q = rng.standard_normal((512, d)) + 2.0 * emb
    K = rng.standard_normal((512, d)) + 2.0 * emb
    V = rng.standard_normal((512, d))
    for p, k_min in ((0.6, 1), (0.9, 2), (1.0, 0)):
        rc = route_ref(Q[None], K[None], p, k_min, cg)
        rb = route_ref(Q[None], K[None], p, k_min, bg)
        # curve block i is box perm[i]: rows and columns renumbered
        assert np.array_equal(rc["mask"][0], rb["mask"][0][np.ix_(perm, perm)])
        assert np.array_equal(rc["counts"][0], rb["counts"][0][perm])
        oc = attn_ref_head(Q, K, V, rc["mask"][0], cg)
        ob = attn_ref_head(Q, K, V, rb["mask"][0], bg)
        np.testing.assert_allclose(oc, ob, rtol=0, atol=1e-12)
