"""Seeded random small configurations, routing and attention against the oracle.

Thirty cases drawn from a fixed seed: grid extents 1..4 x 1..20 x 1..20
(partial blocks on every axis), every supported kind of block box (two
planes, one plane, a wide plane, narrow boxes, a run of tokens), batch 1
or 2, one to three heads with concentrations from flat to peaked, p from 0
to 1 and k_min from 0 to 6. For each case:

* the mask by the routing rule (bit-exact except band and tie blocks,
  oracle/compare.py), counts = row sums and ascending kept lists;
* the attention output on the GPU's own mask, every element, within
  max 2e-2 / mean 1e-3 of the fp64 oracle;
* the same with E4M3 V (the bar of tests/test_gpu_fp8.py: the oracle on the
  dequantised V, P-rounding bound plus 2e-2), empty rows exactly zero;
* the same with Hilbert-curve blocks of the box volume (the checks of
  tests/test_gpu_curve.py, batch 0);
* routing with slack-aware augmentation over a random head -> rank map,
  bit-exact (tests/test_gpu_sasa.py).
"""

import numpy as np
import pytest

import synth
from oracle import attn_ref_head, route_ref
from oracle.compare import ATTN_MAX_ABS, ATTN_MEAN_ABS, compare_mask_rows

from _gpu_util import f64, geometry_of, lib, log, tiling_of, to_dev, torch_mod

pytestmark = pytest.mark.gpu

TILES = [(1, 8, 8), (2, 8, 8), (1, 8, 16), (2, 4, 8), (4, 4, 8), (1, 1, 128), (1, 2, 32)]


def draw(case):
    rng = np.random.default_rng([2024, case])
    tile = TILES[int(rng.integers(len(TILES)))]
    grid = (int(rng.integers(1, 5)), int(rng.integers(1, 21)), int(rng.integers(1, 21)))
    heads = int(rng.integers(1, 4))
    batch = int(rng.integers(1, 3))
    p = float(rng.choice([0.0, 0.3, 0.5, 0.9, 0.97, 1.0]))
    k_min = int(rng.integers(0, 7))
    alphas = tuple(float(a) for a in rng.choice([0.3, 1.0, 3.0, 5.0], size=heads))
    return synth.WorkloadConfig(f"random{case}", heads, grid, tile, p, k_min, 700 + case, "fixed", alphas, batch=batch)


@pytest.mark.parametrize("case", range(30))
def test_random_small_config(case):
    fva, torch = lib(), torch_mod()
    cfg = draw(case)
    geo = geometry_of(cfg)
    nb = geo.nb
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    tiling = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling)
    out = fva.fva_attn(q, k, v, tiling, mask, counts, kv)
    torch.cuda.synchronize()
    m, c, kvn = mask.cpu().numpy(), counts.cpu().numpy(), kv.cpu().numpy()
    O = out.float().cpu().numpy().astype(np.float64)
    assert np.array_equal(m.sum(axis=-1), c)
    band = tie = 0
    errs = []
    for b in range(cfg.batch):
        ref = route_ref(f64(Qb[b]), f64(Kb[b]), cfg.p, cfg.k_min, geo)
        cmp = compare_mask_rows(m[b].reshape(-1, nb), ref["mask"].reshape(-1, nb), ref["order"].reshape(-1, nb),
                                ref["cum"].reshape(-1, nb), ref["scores"].reshape(-1, nb), ref["counts"].reshape(-1),
                                cfg.p, cfg.k_min)
        assert cmp["mismatch"] == 0, (case, b, cmp)
        band += cmp["band"]
        tie += cmp["tie"]
        for h in range(cfg.heads):
            for i in range(nb):
                assert np.array_equal(kvn[b, h, i, : c[b, h, i]], np.nonzero(m[b, h, i])[0])
            o_ref = attn_ref_head(f64(Qb[b, h]), f64(Kb[b, h]), f64(Vb[b, h]), m[b, h], geo)
            errs.append(np.abs(O[b, h] - o_ref).ravel())
    e = np.concatenate(errs)
    log(f"[random {case}] grid {cfg.grid} tile {cfg.tile} batch {cfg.batch} heads {cfg.heads} p {cfg.p} "
        f"k_min {cfg.k_min}: nb {nb}, retained {c.mean() / nb:.3f}, band {band} tie {tie}, "
        f"attn max {e.max():.2e} mean {e.mean():.2e}")
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS


@pytest.mark.parametrize("case", range(30))
def test_random_small_config_fp8v(case):
    # The same configurations with E4M3 V: the quantiser's exponents and the
    # attention against the oracle on the dequantised V, within the
    # P-rounding bound plus the bf16 bar (tests/test_gpu_fp8.py).
    from test_gpu_fp8 import compare_rows

    fva, torch = lib(), torch_mod()
    cfg = draw(case)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    tiling = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling)
    v8, vexp = fva.fva_quantize_v(v, tiling)
    out = fva.fva_attn_fp8v(q, k, v8, vexp, tiling, mask, counts, kv)
    torch.cuda.synchronize()
    m = mask.cpu().numpy()
    O = out.float().cpu().numpy().astype(np.float64)
    rows = {h: list(range(geo.nb)) for h in range(cfg.heads)}
    for b in range(cfg.batch):
        compare_rows(f"random {case} batch {b}", Qb[b:b + 1], Kb[b:b + 1], Vb[b:b + 1], m[b], O[b], geo, rows)
        for h in range(cfg.heads):
            for i in range(geo.nb):
                if not m[b, h, i].any():
                    assert np.all(O[b, h][geo.block_tokens[i]] == 0)


@pytest.mark.parametrize("case", range(30))
def test_random_small_config_curve(case):
    # The same configurations with Hilbert-curve blocks of the box volume:
    # tokens permuted along the curve, routed and attended with the
    # one-dimensional tiling, O permuted back; checked against the oracle run
    # with curve blocks on the raster inputs (batch 0).
    from test_gpu_curve import check_mask, curve_run

    from oracle import curve_geometry

    cfg = draw(case)
    B = int(np.prod(cfg.tile))
    geo = curve_geometry(*cfg.grid, B)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    mask, counts, kv, O = curve_run(Qb, Kb, Vb, cfg.grid, B, cfg.p, cfg.k_min)
    check_mask(f"random {case}", mask, counts, kv, Qb, Kb, geo, cfg.p, cfg.k_min)
    errs = []
    for h in range(cfg.heads):
        ref = attn_ref_head(f64(Qb[0, h]), f64(Kb[0, h]), f64(Vb[0, h]), mask[0, h], geo)
        errs.append(np.abs(O[h] - ref).ravel())
    e = np.concatenate(errs)
    log(f"[random curve {case}] nb {geo.nb}: attn max {e.max():.2e} mean {e.mean():.2e}")
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS


@pytest.mark.parametrize("case", range(30))
def test_random_small_config_sasa(case):
    # The same configurations (batch 1) routed with slack-aware augmentation
    # over a random head -> rank map (ids outside [0, n_ranks) take no part)
    # and random n1, n2: mask, counts, kept lists and per-rank extra blocks
    # bit-exact against the oracle (tests/test_gpu_sasa.py).
    import dataclasses

    from test_gpu_sasa import check

    cfg = dataclasses.replace(draw(case), batch=1)
    rng = np.random.default_rng([4048, case])
    n_ranks = int(rng.integers(1, 5))
    rank_of = rng.integers(-1, n_ranks + 1, size=cfg.heads).astype(np.int32)
    n1 = float(rng.choice([0.0, 0.5, 0.8, 1.0]))
    n2 = float(rng.choice([0.0, 0.07, 0.3]))
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check(f"random {case}", Qb, Kb, cfg, rank_of, n_ranks, n1=n1, n2=n2)
