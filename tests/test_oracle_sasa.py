"""Pins of the oracle's slack-aware augmentation (§3.3, single-GPU reading).

A hand-worked case, then what §3.3 requires of any budget rule: the
critical rank never grows, no rank overtakes the old maximum (no new
straggler), ranks below the trigger are untouched, the augmented kept set
is the next blocks of the routing order (a superset and a prefix of it),
n1 = 0 and balanced ranks change nothing, more n1 never keeps less. The
decisions are exact rationals; an fp64 evaluation of the same rule (what a
kernel computes) may differ only at the boundaries boundary_ranks names,
and does differ at a hand-built one.
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle.sasa import augment_with, boundary_ranks, rank_loads, sasa_augment, sasa_extras


def random_case(rng, heads=12, nb=9, ranks=4):
    counts = rng.integers(1, nb + 1, size=(heads, nb))
    order = np.stack([np.stack([rng.permutation(nb) for _ in range(nb)]) for _ in range(heads)])
    rank_of = np.repeat(np.arange(ranks), heads // ranks)
    return counts, order, rank_of


def test_hand_worked_case():
    # nb = 4; heads 0, 1 on rank 0 (S = 8 + 4 = 12), head 2 on rank 1 (S = 6).
    counts = np.array([[2, 2, 2, 2], [1, 1, 1, 1], [1, 2, 1, 2]])
    order = np.tile(np.array([3, 1, 0, 2]), (3, 4, 1))
    S_r, H_r = rank_loads(counts, [0, 0, 1], 2)
    assert S_r.tolist() == [12, 6] and H_r.tolist() == [2, 1]
    # rank 1: slack 6/4 = 1.5 rows, above 0.07 * 3 = 0.21; budget 0.8 * 1.5 = 1.2 -> one more block per row
    mask, new_counts, extra, info = sasa_augment(order, counts, [0, 0, 1], 2, 0.8, 0.07)
    assert extra.tolist() == [0, 1]
    assert new_counts.tolist() == [[2, 2, 2, 2], [1, 1, 1, 1], [2, 3, 2, 3]]
    assert info["fired"].tolist() == [False, True]
    assert np.allclose(info["L_r"], [3.0, 1.5]) and np.allclose(info["dL_r"], [0.0, 1.5])
    assert np.allclose(info["B_r"], [0.0, 1.2])
    assert mask[2, 0].tolist() == [0, 1, 0, 1]  # blocks 3 and 1, the first two of the order
    assert mask[2, 1].tolist() == [1, 1, 0, 1]  # and block 0, the third
    # a trigger above the slack turns it off
    _, nc2, extra2, _ = sasa_augment(order, counts, [0, 0, 1], 2, 0.8, 0.6)
    assert extra2.tolist() == [0, 0] and np.array_equal(nc2, counts)


@pytest.mark.parametrize("seed", range(20))
def test_budget_invariants(seed):
    rng = np.random.default_rng(seed)
    counts, order, rank_of = random_case(rng)
    nb = counts.shape[1]
    n1, n2 = 0.8, 0.07
    mask, nc, extra, info = sasa_augment(order, counts, rank_of, 4, n1, n2)
    S_r, H_r = rank_loads(counts, rank_of, 4)
    S_aug, _ = rank_loads(nc, rank_of, 4)
    crit = np.argmax(S_r)
    assert S_aug[crit] == S_r[crit]
    assert np.all(S_aug <= S_r.max())  # no new straggler
    assert np.all(S_aug >= S_r)
    assert np.all((S_aug - S_r) <= n1 * (S_r.max() - S_r) + 1e-9)  # within the budget
    low = (S_r.max() - S_r) <= n2 * S_r.max()
    assert np.all(S_aug[low] == S_r[low])
    for h in range(counts.shape[0]):
        for i in range(nb):
            kept = np.nonzero(mask[h, i])[0]
            assert set(kept) == set(order[h, i, : nc[h, i]].tolist())
            assert set(order[h, i, : counts[h, i]].tolist()) <= set(kept.tolist())
            assert nc[h, i] == min(nb, counts[h, i] + extra[rank_of[h]])


def test_identity_cases_and_monotonicity():
    rng = np.random.default_rng(3)
    counts, order, rank_of = random_case(rng)
    _, nc0, e0, _ = sasa_augment(order, counts, rank_of, 4, 0.0, 0.07)
    assert np.array_equal(nc0, counts) and not e0.any()
    balanced = np.full_like(counts, 4)
    _, ncb, eb, _ = sasa_augment(order, balanced, rank_of, 4, 0.8, 0.0)
    assert np.array_equal(ncb, balanced) and not eb.any()
    prev = counts
    for n1 in (0.2, 0.5, 0.8, 1.0):
        _, nc, _, _ = sasa_augment(order, counts, rank_of, 4, n1, 0.07)
        assert np.all(nc >= prev)
        prev = nc


def fp64_extras(counts, rank_of, ranks, n1, n2):
    """The rule evaluated in fp64, as a floating-point kernel would."""
    S_r, H_r = rank_loads(counts, rank_of, ranks)
    S_max = float(S_r.max())
    nb = counts.shape[1]
    out = np.zeros(ranks, dtype=np.int64)
    for r in range(ranks):
        D = S_max - float(S_r[r])
        if H_r[r] > 0 and D > n2 * S_max:
            out[r] = int(np.floor((n1 * D) / float(nb * int(H_r[r]))))
    return out


def test_exact_decision_where_fp64_rounds_up():
    # D = 10 on rank 1, nb * H = 7, n1 = 0.7: the double 0.7 is below 7/10, so
    # n1 * D / 7 is just below 1 (no extra block), while fp64 rounds 0.7 * 10
    # to exactly 7 and gives one. The oracle keeps the exact answer and names
    # the rank as a boundary that accepts both.
    counts = np.array([[7] * 7, [7, 7, 7, 7, 7, 2, 2]])
    extra, info = sasa_extras(counts, [0, 1], 2, 0.7, 0.0)
    assert extra.tolist() == [0, 0] and info["fired"].tolist() == [False, True]
    assert fp64_extras(counts, [0, 1], 2, 0.7, 0.0).tolist() == [0, 1]
    assert boundary_ranks(counts, [0, 1], 2, 0.7, 0.0) == {1: {0, 1}}
    mask, nc = augment_with(np.tile(np.arange(7), (2, 7, 1)), counts, [0, 1], [0, 1])
    assert nc[1].tolist() == [7, 7, 7, 7, 7, 3, 3] and mask[1, 5].tolist() == [1, 1, 1, 0, 0, 0, 0]
    # the trigger boundary: D = n2 * S_max exactly does not fire (strict >)
    counts = np.array([[4, 4], [2, 4]])  # S = 8, 6; D = 2 = 0.25 * 8
    extra, info = sasa_extras(counts, [0, 1], 2, 1.0, 0.25)
    assert extra.tolist() == [0, 0] and not info["fired"].any()
    assert boundary_ranks(counts, [0, 1], 2, 1.0, 0.25) == {1: {0, 1}}


@pytest.mark.parametrize("seed", range(30))
def test_fp64_decisions_stay_within_the_boundary_sets(seed):
    rng = np.random.default_rng(100 + seed)
    ranks = int(rng.integers(2, 6))
    heads = ranks * int(rng.integers(1, 4))
    nb = int(rng.integers(3, 40))
    counts = rng.integers(0, nb + 1, size=(heads, nb))
    rank_of = rng.integers(0, ranks, size=heads)
    # short decimals make exact boundaries common (0.5 * 8 / 4 = 1, 0.25 of S_max ...)
    n1 = float(rng.choice([0.1, 0.25, 0.5, 0.7, 0.8, 1.0, rng.uniform(0, 1)]))
    n2 = float(rng.choice([0.0, 0.05, 0.07, 0.1, 0.25, rng.uniform(0, 0.3)]))
    extra, _ = sasa_extras(counts, rank_of, ranks, n1, n2)
    bound = boundary_ranks(counts, rank_of, ranks, n1, n2)
    got = fp64_extras(counts, rank_of, ranks, n1, n2)
    S_r, H_r = rank_loads(counts, rank_of, ranks)
    for r in range(ranks):
        assert got[r] in bound.get(r, {int(extra[r])}), (r, got[r], extra[r], bound)
        if r in bound:
            assert int(extra[r]) in bound[r]
            continue
        # away from the boundaries, the exact rule by hand
        D = int(S_r.max()) - int(S_r[r])
        if H_r[r] == 0 or not Fraction(D) > Fraction(n2) * int(S_r.max()):
            assert extra[r] == 0
        else:
            assert extra[r] == (Fraction(n1) * D / (nb * int(H_r[r]))) // 1
