"""GPU parity of fva_route against the fp64 oracle.

Mask rule (oracle/compare.py): bit-exact except blocks whose oracle running
sum before them lies within 1e-5 of p (band) or whose score ties the cut
block's to 1e-12 (tie); both are counted and reported, mismatches must be 0.
counts and kv_idx must describe the GPU mask exactly.
"""

import math

import numpy as np
import pytest

import synth
from oracle import route_ref
from oracle.compare import compare_mask_rows

from _gpu_util import custom_config, f64, geometry_of, lib, log, tiling_of, to_dev, torch_mod, workload

pytestmark = pytest.mark.gpu


def gpu_route(Qb, Kb, cfg, p, k_min):
    fva = lib()
    q, k = to_dev(Qb), to_dev(Kb)
    mask, counts, kv = fva.fva_route(q, k, p, k_min, tiling_of(cfg))
    torch_mod().cuda.synchronize()
    return mask.cpu().numpy(), counts.cpu().numpy(), kv.cpu().numpy()


def check_route(name, Qb, Kb, cfg, p, k_min, heads=None):
    """Route on the GPU (all heads) and compare the given heads with the oracle."""
    geo = geometry_of(cfg)
    nb = geo.nb
    mask, counts, kv = gpu_route(Qb, Kb, cfg, p, k_min)
    B, H = Qb.shape[:2]
    heads = list(range(H)) if heads is None else list(heads)
    # internal consistency of every row
    assert np.array_equal(mask.sum(axis=-1), counts), "counts must equal mask row sums"
    kf = min(k_min, nb)
    assert counts.min() >= kf
    for b in range(B):
        for h in heads:
            for i in range(nb):
                c = counts[b, h, i]
                assert np.array_equal(kv[b, h, i, :c], np.nonzero(mask[b, h, i])[0]), (name, b, h, i)
    totals = dict(mismatch=0, band=0, tie=0)
    for b in range(B):
        ref = route_ref(f64(Qb[b, heads]), f64(Kb[b, heads]), p, k_min, geo)
        cmp = compare_mask_rows(
            mask[b, heads].reshape(-1, nb), ref["mask"].reshape(-1, nb), ref["order"].reshape(-1, nb),
            ref["cum"].reshape(-1, nb), ref["scores"].reshape(-1, nb), ref["counts"].reshape(-1), p, k_min,
        )
        for key in totals:
            totals[key] += cmp[key]
        diff_rows = (mask[b, heads] != ref["mask"]).any(axis=-1)
        same = ~diff_rows
        assert np.array_equal(counts[b, heads][same], ref["counts"][same])
    log(f"[route] {name} p={p} k_min={k_min} heads={len(heads)}: mismatches={totals['mismatch']} "
        f"band-tolerated={totals['band']} tie-tolerated={totals['tie']} "
        f"density={counts[:, heads].mean() / nb:.3f}")
    assert totals["mismatch"] == 0, totals
    return mask, counts, kv


def test_route_tiny():
    cfg = synth.get_config("tiny")
    Qb, Kb, _ = workload("tiny")
    check_route("tiny", Qb, Kb, cfg, cfg.p, cfg.k_min)


PARTIAL = [
    # (grid, tile): partial boxes on every axis, 1x8x8 and 2x8x8 boxes
    ((5, 13, 21), (2, 8, 8)),
    ((3, 9, 10), (1, 8, 8)),
    ((4, 32, 40), (1, 8, 8)),  # nb = 80 > 64: several lanes per row
    ((7, 17, 29), (2, 8, 8)),
    ((5, 24, 40), (1, 8, 8)),  # nb = 75: rows not whole words, blocks past 32 in each 64
]


@pytest.mark.parametrize("grid,tile", PARTIAL)
@pytest.mark.parametrize("p,k_min", [(0.9, 4), (0.5, 1), (0.95, 0), (0.0, 3), (1.0, 0), (0.8, 10_000)])
def test_route_partial_tiles(grid, tile, p, k_min):
    cfg = custom_config("partial", 3, grid, tile, (0.3, 1.5, 5.0), seed=11)
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check_route(f"grid{grid}tile{tile}", Qb, Kb, cfg, p, k_min)


@pytest.mark.parametrize("grid", [(3, 16, 16), (4, 32, 40), (10, 40, 48)])
@pytest.mark.parametrize("p,k_min", [(0.9037, 2), (0.5513, 0), (0.3071, 7)])  # p*nb never integral
def test_route_exact_ties(grid, p, k_min):
    # Q = 0: every score is exactly 0, P = 1/nb, the kept set is the lowest
    # m = max(ceil(p*nb), k_min) block ids (ties go to the lower id).
    cfg = custom_config("ties", 1, grid, (1, 8, 8), (1.0,), seed=12)
    _, Kb, _ = synth.gen_qkv(cfg)
    Qb = np.zeros_like(Kb)
    nb = geometry_of(cfg).nb
    if abs(p * nb - round(p * nb)) < 1e-6:
        pytest.skip("p*nb on an integer is a band case")
    mask, counts, _ = gpu_route(Qb, Kb, cfg, p, k_min)
    m = min(max(math.ceil(p * nb), k_min), nb)
    expect = np.zeros(nb, np.uint8)
    expect[:m] = 1
    assert np.all(counts == m)
    assert np.all(mask[0, 0] == expect[None, :])


@pytest.mark.parametrize("name", ["480p", "720p", "720p_stress", "long"])
def test_route_full_workloads(name):
    cfg = synth.get_config(name)
    Qb, Kb, _ = workload(name)
    check_route(name, Qb, Kb, cfg, cfg.p, cfg.k_min)


@pytest.mark.parametrize("p", [0.8, 0.95])
def test_route_long_p_sweep(p):
    cfg = synth.get_config("long")
    Qb, Kb, _ = workload("long")
    check_route("long", Qb, Kb, cfg, p, cfg.k_min)


def test_route_deterministic():
    cfg = synth.get_config("720p")
    Qb, Kb, _ = workload("720p")
    m1, c1, k1 = gpu_route(Qb, Kb, cfg, cfg.p, cfg.k_min)
    m2, c2, k2 = gpu_route(Qb, Kb, cfg, cfg.p, cfg.k_min)
    assert np.array_equal(m1, m2) and np.array_equal(c1, c2)
    valid = np.arange(k1.shape[-1])[None, None, None, :] < c1[..., None]
    assert np.array_equal(k1[valid], k2[valid])  # entries past counts are unspecified


# Block counts on both sides of every multiple of 64 that selects a
# different number of scores per lane (1..16): a row's last lane group is
# then full, holds one block, or (nb = 1) only lane 0 holds a block. One
# line of 64-token blocks with a short last block, two heads (a flat and a
# concentrated one).
WAVE_EDGE_NB = [1, 63, 64, 65, 128, 129, 256, 257, 511, 513, 768, 769, 1024]


def line_config(name, nb, seed, alphas=(0.5, 3.0)):
    n = 40 if nb == 1 else 64 * nb - 17
    return custom_config(name, len(alphas), (1, 1, n), (1, 1, 64), alphas, seed=seed)


@pytest.mark.parametrize("nb", WAVE_EDGE_NB)
def test_route_block_counts_at_wave_edges(nb):
    cfg = line_config(f"edge{nb}", nb, seed=60 + nb % 37)
    assert geometry_of(cfg).nb == nb
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check_route(f"edge nb={nb}", Qb, Kb, cfg, cfg.p, cfg.k_min)


def test_route_max_blocks():
    # nb = 1024, the largest supported block count: 16 x 128 x 64 tokens, 2x8x8 boxes.
    cfg = custom_config("max_blocks", 1, (16, 128, 64), (2, 8, 8), (1.5,), seed=11)
    assert geometry_of(cfg).nb == 1024
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check_route("max_blocks", Qb, Kb, cfg, cfg.p, cfg.k_min)


def test_route_batch_two_odd_heads():
    cfg = synth.WorkloadConfig("batch2", 3, (5, 13, 21), (2, 8, 8), 0.9, 3, 12, "fixed", (0.7, 2.5, 4.0), batch=2)
    Qb, Kb, _ = synth.gen_qkv(cfg)
    assert Qb.shape[:2] == (2, 3)
    check_route("batch2", Qb, Kb, cfg, cfg.p, cfg.k_min)


def test_route_unaligned_mask_rows():
    # Mask rows of whole 32-bit words go out as words only when the row start
    # is 4-byte aligned; a mask at an odd address takes the byte stores.
    # Both must give the same mask (nb = 80, a multiple of 4).
    cfg = custom_config("unaligned", 3, (4, 32, 40), (1, 8, 8), (0.7, 2.0, 4.0), seed=21)
    nb = geometry_of(cfg).nb
    assert nb % 4 == 0
    Qb, Kb, _ = synth.gen_qkv(cfg)
    mask, counts, kv = gpu_route(Qb, Kb, cfg, cfg.p, cfg.k_min)
    fva, torch = lib(), torch_mod()
    q, k = to_dev(Qb), to_dev(Kb)
    for offset in (1, 2, 3):
        buf = torch.zeros(mask.size + 4, dtype=torch.uint8, device="cuda:0")
        m_dev = buf[offset:offset + mask.size].view(mask.shape)
        c_dev = torch.empty(counts.shape, dtype=torch.int32, device="cuda:0")
        k_dev = torch.empty(kv.shape, dtype=torch.int32, device="cuda:0")
        fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg), out=(m_dev, c_dev, k_dev))
        torch.cuda.synchronize()
        assert np.array_equal(m_dev.cpu().numpy(), mask), offset
        assert np.array_equal(c_dev.cpu().numpy(), counts), offset
        host = buf.cpu().numpy()
        assert not host[:offset].any() and not host[offset + mask.size:].any(), offset  # nothing outside the view
    check_route("unaligned", Qb, Kb, cfg, cfg.p, cfg.k_min)


def test_route_multilevel_select():
    # One key block far below the rest stretches the score range, so the
    # first 64-bucket pass leaves the whole cluster (~150 blocks) in the
    # bucket where the running mass crosses p and the radix select takes a
    # second level before ranking. nb = 300.
    grid, tile = (10, 40, 48), (1, 8, 8)
    cfg = custom_config("multilevel", 1, grid, tile, (1.0,), seed=5)
    geo = geometry_of(cfg)
    T, H, W = grid
    rng = np.random.default_rng(5)
    u = rng.standard_normal(128)
    u /= np.linalg.norm(u)
    a = rng.uniform(0.0, 1.0, geo.nb)
    a[137] = -40.0
    t, y, x = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    blk = ((t // tile[0]) * geo.nby + y // tile[1]) * geo.nbx + x // tile[2]
    blk = blk.reshape(-1)
    q = 2.0 * u[None, :] + 0.01 * rng.standard_normal((blk.size, 128))
    k = a[blk][:, None] * u[None, :] + 0.5 * rng.standard_normal((blk.size, 128))
    Qb = synth.f32_to_bf16_bits(q.astype(np.float32)).reshape(1, 1, -1, 128)
    Kb = synth.f32_to_bf16_bits(k.astype(np.float32)).reshape(1, 1, -1, 128)
    mask, counts, _ = check_route("multilevel", Qb, Kb, cfg, 0.9, 4)
    assert mask[0, 0, :, 137].sum() == 0  # the outlier is never kept
    assert 0.5 * geo.nb < counts.mean() < geo.nb  # the cut falls inside the cluster
