"""Pins of the oracle's routing frontend (pooled scores, softmax, Top-p, floor).

Each check fixes a property the paper's definitions (§2.1 Top-p and the Top-k
floor, §3.1 pooled block similarities, Eq. 1 workload) or plain mathematics
impose, independent of the oracle's own implementation:

* pooling: explicit per-token loops, constants and linearity;
* Top-p: brute-force subset enumeration (fewest blocks with mass >= p, and the
  chosen set has the largest mass among sets of that size), hand-worked rows
  (tests/golden/topp_rows.json), the uniform and one-hot closed forms;
* invariants: floor, reach, minimality, prefix property, nesting in p.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle import (
    block_scores,
    block_softmax,
    head_workload,
    pool_blocks,
    route_ref,
    tile_geometry,
    topp_select,
)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "topp_rows.json")


def test_pool_explicit_loop_partial_tiles():
    geo = tile_geometry(3, 5, 7, 2, 2, 4)
    rng = np.random.default_rng(0)
    X = rng.standard_normal((geo.N, 6))
    got = pool_blocks(X, geo)
    for i in range(geo.nb):
        acc = np.zeros(6)
        cnt = 0
        for n in range(geo.N):
            if geo.block_of_token[n] == i:
                acc += X[n]
                cnt += 1
        np.testing.assert_allclose(got[i], acc / cnt, rtol=0, atol=1e-14)


def test_pool_constant_and_linear():
    geo = tile_geometry(3, 16, 16, 1, 8, 8)
    X = np.full((geo.N, 4), 2.5)
    np.testing.assert_array_equal(pool_blocks(X, geo), np.full((geo.nb, 4), 2.5))
    rng = np.random.default_rng(1)
    A, B = rng.standard_normal((2, geo.N, 4))
    np.testing.assert_allclose(pool_blocks(3 * A - B, geo), 3 * pool_blocks(A, geo) - pool_blocks(B, geo), atol=1e-13)


def test_scores_explicit():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((2, 5, 8))
    s = block_scores(q, k)
    for i in range(5):
        for j in range(5):
            assert abs(s[i, j] - sum(q[i, c] * k[j, c] for c in range(8)) / math.sqrt(8)) < 1e-14


def test_softmax_rows_sum_to_one_and_shift_invariant():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((4, 9)) * 5
    P = block_softmax(s)
    np.testing.assert_allclose(P.sum(axis=1), 1.0, atol=1e-15)
    np.testing.assert_allclose(block_softmax(s + 100.0), P, atol=1e-15)
    np.testing.assert_allclose(P[0], np.exp(s[0]) / np.exp(s[0]).sum(), atol=1e-15)


def _golden_rows():
    with open(GOLDEN) as f:
        data = json.load(f)
    for row in data["rows"]:
        if "scores_are_log_probs" in row:
            s = np.log(np.asarray(row["scores_are_log_probs"], dtype=np.float64))
        else:
            s = np.asarray(row["scores"], dtype=np.float64)
        for case in row["cases"]:
            yield row["name"], s, case


@pytest.mark.parametrize("name,s,case", list(_golden_rows()))
def test_golden_rows(name, s, case):
    P = block_softmax(s[None, :])
    sel = topp_select(s[None, :], P, case["p"], case["k_min"])
    assert sel["kv_idx"][0].tolist() == case["kept"], name
    assert int(sel["m_p"][0]) == case["m_p"], name
    assert int(sel["counts"][0]) == len(case["kept"])


def test_brute_force_minimal_subset():
    rng = np.random.default_rng(4)
    nb = 10
    for trial in range(60):
        s = rng.standard_normal((1, nb)) * rng.uniform(0.2, 4.0)
        P = block_softmax(s)[0]
        p = float(rng.uniform(0.05, 0.999))
        sel = topp_select(s, P[None, :], p, 0)
        m = int(sel["counts"][0])
        # smallest cardinality of any subset with mass >= p
        best_card = None
        best_mass = -1.0
        for card in range(0, nb + 1):
            masses = [sum(P[list(c)]) for c in itertools.combinations(range(nb), card)]
            ok = [x for x in masses if x >= p]
            if ok:
                best_card = card
                best_mass = max(ok)
                break
        assert best_card is not None
        assert m == best_card
        kept_mass = P[sel["kv_idx"][0]].sum()
        assert kept_mass >= p
        assert abs(kept_mass - best_mass) < 1e-12  # the prefix is the heaviest set of that size


def test_uniform_closed_form():
    # Q = 0 -> every score is 0 -> P = 1/nb; m = max(ceil(p * nb), k_min); kept = lowest ids.
    geo = tile_geometry(3, 16, 16, 1, 8, 8)
    Q = np.zeros((1, geo.N, 8))
    K = np.random.default_rng(5).standard_normal((1, geo.N, 8))
    for p, k_min in ((0.9, 2), (0.55, 0), (0.3, 7), (0.62, 1)):  # p*nb kept away from integers
        r = route_ref(Q, K, p, k_min, geo)
        m = max(math.ceil(p * geo.nb), k_min)
        assert np.all(r["counts"] == m)
        expect = np.zeros(geo.nb, np.uint8)
        expect[:m] = 1
        assert np.all(r["mask"][0] == expect[None, :])
    assert max(math.ceil(0.9 * 12), 2) == 11  # the tiny workload keeps 11 of 12 blocks


def test_one_hot_closed_form():
    nb = 12
    s = np.full((3, nb), -50.0)
    s[0, 7] = 10.0
    s[1, 0] = 10.0
    s[2, 11] = 10.0
    P = block_softmax(s)
    for k_min in (0, 1, 3):
        sel = topp_select(s, P, 0.9, k_min)
        assert np.all(sel["counts"] == max(1, k_min))
        assert sel["mask"][0, 7] == 1 and sel["mask"][1, 0] == 1 and sel["mask"][2, 11] == 1


def _check_invariants(s, P, sel, p, k_min):
    nb = s.shape[1]
    kf = min(k_min, nb)
    for r in range(s.shape[0]):
        m = int(sel["counts"][r])
        kept = sel["mask"][r].astype(bool)
        assert kept.sum() == m
        assert m >= kf
        c = np.concatenate([[0.0], np.cumsum(P[r][sel["order"][r]])])
        assert c[m] >= p or m == nb
        if m > kf and m > 0:
            assert c[m - 1] < p  # minimality: one block fewer does not reach p
        if 0 < m < nb:
            assert s[r][kept].min() >= s[r][~kept].max()  # kept set is a score prefix
        assert sel["kv_idx"][r].tolist() == np.nonzero(kept)[0].tolist()


def test_invariants_and_nesting_random():
    rng = np.random.default_rng(6)
    for trial in range(20):
        nb = int(rng.integers(1, 40))
        s = rng.standard_normal((5, nb)) * rng.uniform(0.1, 6.0)
        P = block_softmax(s)
        k_min = int(rng.integers(0, 6))
        prev = None
        for p in (0.0, 0.3, 0.8, 0.9, 0.95, 1.0):
            sel = topp_select(s, P, p, k_min)
            _check_invariants(s, P, sel, p, k_min)
            if prev is not None:
                assert np.all(sel["mask"] >= prev)  # masks nest as p grows
            prev = sel["mask"]


def test_p_one_keeps_all():
    rng = np.random.default_rng(7)
    s = rng.standard_normal((4, 30)) * 8
    for k_min in (0, 4):
        sel = topp_select(s, block_softmax(s), 1.0, k_min)
        assert np.all(sel["counts"] == 30)
        assert np.all(sel["mask"] == 1)


def test_rejects_bad_parameters():
    s = np.zeros((1, 3))
    with pytest.raises(ValueError):
        topp_select(s, block_softmax(s), 1.5, 0)
    with pytest.raises(ValueError):
        topp_select(s, block_softmax(s), 0.5, -1)


def test_tiny_workload_heads_differ_in_density():
    cfg = synth.get_config("tiny")
    geo = tile_geometry(*cfg.grid, *cfg.tile)
    Q, K, _ = synth.gen_qkv(cfg)
    Qf = synth.bf16_bits_to_f32(Q[0]).astype(np.float64)
    Kf = synth.bf16_bits_to_f32(K[0]).astype(np.float64)
    r = route_ref(Qf, Kf, cfg.p, cfg.k_min, geo)
    L = head_workload(r["counts"])
    assert L.shape == (2,)
    assert L[0] < L[1]  # alpha = 3 (concentrated) keeps fewer blocks than alpha = 0.5 (flat)
    assert np.all(r["counts"] >= cfg.k_min)


def test_workload_eq1():
    counts = np.array([[1, 2, 3, 6], [4, 4, 4, 4]])
    np.testing.assert_array_equal(head_workload(counts), [3.0, 4.0])
