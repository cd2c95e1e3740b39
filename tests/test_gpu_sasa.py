"""GPU parity of slack-aware augmentation (fva_route_sasa) against the oracle.

Integer work end to end: the routing order and first-pass counts are those
of fva_route (bit-exact against the oracle on these workloads). The oracle
decides each rank's trigger and extra blocks in exact rational arithmetic;
the kernel's fp64 evaluation must give the same value, except at a rank
that oracle.sasa.boundary_ranks names (an exact quantity within fp64
rounding of its boundary), where either side's value is accepted and the
mask is then checked for the kernel's value. The augmented mask, counts and
kept lists must equal the oracle's bit for bit.
"""

import numpy as np
import pytest

import synth
from oracle import route_ref
from oracle.sasa import augment_with, boundary_ranks, rank_loads, sasa_extras

from _gpu_util import custom_config, f64, geometry_of, lib, log, tiling_of, to_dev, torch_mod, workload

pytestmark = pytest.mark.gpu


def run_sasa(Qb, Kb, cfg, rank_of, n_ranks, n1, n2):
    fva, torch = lib(), torch_mod()
    q, k = to_dev(Qb), to_dev(Kb)
    r = torch.from_numpy(np.asarray(rank_of, dtype=np.int32)).to("cuda:0")
    mask, counts, kv, extra = fva.fva_route_sasa(q, k, cfg.p, cfg.k_min, tiling_of(cfg), r, n_ranks, n1, n2)
    plain = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    torch.cuda.synchronize()
    return (mask.cpu().numpy()[0], counts.cpu().numpy()[0], kv.cpu().numpy()[0], extra.cpu().numpy(),
            plain[1].cpu().numpy()[0])


def accepted_extras(got, counts, rank_of, n_ranks, n1, n2):
    """The kernel's per-rank extras, checked against the oracle's exact ones.

    Equal, or (at a boundary rank) one of the values either decision gives.
    Returns the extras to build the reference mask from.
    """
    e_ref, _ = sasa_extras(counts, rank_of, n_ranks, n1, n2)
    bound = boundary_ranks(counts, rank_of, n_ranks, n1, n2)
    got = np.asarray(got, dtype=np.int64)
    for r in range(n_ranks):
        assert int(got[r]) in bound.get(r, {int(e_ref[r])}), (r, got[r], e_ref[r], bound.get(r))
    if bound:
        log(f"[sasa] boundary ranks {sorted(bound)}: kernel {[int(got[r]) for r in sorted(bound)]}, "
            f"exact {[int(e_ref[r]) for r in sorted(bound)]}")
    return got


def check(name, Qb, Kb, cfg, rank_of, n_ranks, n1=0.8, n2=0.07):
    geo = geometry_of(cfg)
    mask, counts, kv, extra, counts0 = run_sasa(Qb, Kb, cfg, rank_of, n_ranks, n1, n2)
    ref = route_ref(f64(Qb[0]), f64(Kb[0]), cfg.p, cfg.k_min, geo)
    assert np.array_equal(counts0, ref["counts"]), "first-pass counts differ from the oracle"
    rank_of = np.asarray(rank_of)
    valid = (rank_of >= 0) & (rank_of < n_ranks)
    keep = np.nonzero(valid)[0]  # heads without a rank take no part and stay as routed
    e_use = accepted_extras(extra[:n_ranks], ref["counts"][keep], rank_of[keep], n_ranks, n1, n2)
    _, c_sub = augment_with(ref["order"][keep], ref["counts"][keep], rank_of[keep], e_use)
    c_ref = ref["counts"].copy()
    c_ref[keep] = c_sub
    m_ref = np.zeros_like(mask)
    for h in range(mask.shape[0]):
        for i in range(geo.nb):
            m_ref[h, i, ref["order"][h, i, : c_ref[h, i]]] = 1
    assert np.array_equal(counts, c_ref)
    assert np.array_equal(mask, m_ref)
    for h in range(mask.shape[0]):
        for i in range(geo.nb):
            assert np.array_equal(kv[h, i, : counts[h, i]], np.nonzero(mask[h, i])[0])
    S0, _ = rank_loads(counts0, np.where(valid, rank_of, 0), n_ranks)
    S1, _ = rank_loads(counts, np.where(valid, rank_of, 0), n_ranks)
    log(f"[sasa] {name}: extra per rank {extra[:n_ranks].tolist()}; rank loads (rows) "
        f"{np.round(S0 / geo.nb, 1).tolist()} -> {np.round(S1 / geo.nb, 1).tolist()}; "
        f"retained {counts0.sum() / counts0.size / geo.nb:.3f} -> {counts.sum() / counts.size / geo.nb:.3f}")
    return counts0, counts, extra


def test_sasa_tiny_two_ranks():
    cfg = synth.get_config("tiny")
    Qb, Kb, _ = workload("tiny")
    check("tiny", Qb, Kb, cfg, [0, 1], 2, n1=0.8, n2=0.0)


@pytest.mark.parametrize("name", ["480p", "720p", "720p_stress"])
def test_sasa_full_workloads_eight_ranks(name):
    cfg = synth.get_config(name)
    Qb, Kb, _ = workload(name)
    rank_of = np.arange(cfg.heads) // (cfg.heads // 8)  # Ulysses: contiguous head groups per rank
    c0, c1, extra = check(name, Qb, Kb, cfg, rank_of, 8)
    geo = geometry_of(cfg)
    S0, _ = rank_loads(c0, rank_of, 8)
    S1, _ = rank_loads(c1, rank_of, 8)
    assert S1.max() == S0.max()  # no new straggler
    assert (extra > 0).any() or (S0.max() - S0 <= 0.07 * S0.max()).all()


@pytest.mark.parametrize("n1,n2", [(0.0, 0.07), (1.0, 0.0), (0.5, 0.3)])
def test_sasa_parameters_and_uneven_ranks(n1, n2):
    cfg = custom_config("sasa", 6, (5, 13, 21), (2, 8, 8), (0.3, 5.0, 1.0, 4.0, 0.5, 2.0), seed=41)
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check(f"n1={n1} n2={n2}", Qb, Kb, cfg, [0, 0, 0, 1, 2, 2], 3, n1=n1, n2=n2)


def test_sasa_heads_without_rank_and_empty_rank():
    cfg = custom_config("sasa2", 4, (3, 16, 16), (1, 8, 8), (0.3, 5.0, 4.0, 0.5), seed=43)
    Qb, Kb, _ = synth.gen_qkv(cfg)
    # head 1 has no rank (-1), head 3 an id past n_ranks; rank 2 holds no head
    check("no-rank", Qb, Kb, cfg, [0, -1, 1, 7], 3, n1=0.9, n2=0.0)


def test_sasa_batch_two():
    # ranks over batch * heads: rank_of[b * heads + h]
    fva, torch = lib(), torch_mod()
    cfg = synth.WorkloadConfig("sasab2", 3, (3, 16, 16), (1, 8, 8), 0.9, 2, 47, "fixed", (0.3, 5.0, 2.0), batch=2)
    Qb, Kb, _ = synth.gen_qkv(cfg)
    geo = geometry_of(cfg)
    rank_of = np.array([0, 0, 1, 1, 2, 2], dtype=np.int32)
    r = torch.from_numpy(rank_of).to("cuda:0")
    mask, counts, kv, extra = fva.fva_route_sasa(to_dev(Qb), to_dev(Kb), cfg.p, cfg.k_min, tiling_of(cfg), r, 3, 0.8, 0.0)
    torch.cuda.synchronize()
    order = np.concatenate([route_ref(f64(Qb[b]), f64(Kb[b]), cfg.p, cfg.k_min, geo)["order"] for b in range(2)])
    c0 = np.concatenate([route_ref(f64(Qb[b]), f64(Kb[b]), cfg.p, cfg.k_min, geo)["counts"] for b in range(2)])
    e_use = accepted_extras(extra.cpu().numpy(), c0, rank_of, 3, 0.8, 0.0)
    m_ref, c_ref = augment_with(order, c0, rank_of, e_use)
    assert np.array_equal(counts.cpu().numpy().reshape(6, -1), c_ref)
    assert np.array_equal(mask.cpu().numpy().reshape(6, geo.nb, geo.nb), m_ref)
    log(f"[sasa] batch 2: extra per rank {e_use.tolist()}")


@pytest.mark.parametrize("nb", [1, 64, 65, 129, 257, 513, 769, 1024])
def test_sasa_block_counts_at_wave_edges(nb):
    # a line of 64-token blocks (short last block), a flat head on rank 0
    # and a concentrated one on rank 1: rank 1 is augmented
    n = 40 if nb == 1 else 64 * nb - 17
    cfg = custom_config(f"sasa_edge{nb}", 2, (1, 1, n), (1, 1, 64), (0.5, 3.0), seed=90 + nb % 31)
    assert geometry_of(cfg).nb == nb
    Qb, Kb, _ = synth.gen_qkv(cfg)
    check(f"edge nb={nb}", Qb, Kb, cfg, [0, 1], 2, n1=0.8, n2=0.0)


def test_sasa_one_rank_per_head_and_max_ranks():
    cfg = synth.get_config("480p")
    Qb, Kb, _ = workload("480p")
    check("480p, 40 ranks", Qb, Kb, cfg, np.arange(cfg.heads), cfg.heads)
    # 1024 ranks, heads spread over a few of them, the rest empty
    rank_of = (np.arange(cfg.heads) % 4) * 255
    check("480p, 1024 ranks", Qb, Kb, cfg, rank_of, 1024)
