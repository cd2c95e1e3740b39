"""Pins of the GPU-vs-oracle mask classifier (oracle/compare.py).

Every GPU mask verdict goes through compare_mask_rows, so it is pinned here
on hand-built rows whose band, tie and mismatch counts follow from the rule
(Top-p with a floor, §2.1) by inspection. Each case is chosen so that a
plausible slip in the classifier changes a count:

* reading the inclusive sum c_r instead of c_{r-1} for rank r;
* letting the floor rank itself (r == min(k_min, nb)) into the band;
* tolerating a block that is not a tie and not at a moved cut;
* accepting a GPU set that is not a prefix of the oracle order (skipping a
  band rank and keeping a later one), even when every running sum involved
  lies in the band.
"""

import numpy as np
import pytest

from oracle.compare import BAND, compare_mask_rows
from oracle.route import topp_select

# One row, scores strictly decreasing with the block id, so the order pi is
# the identity and rank r is block r - 1. The probabilities are given
# directly (topp_select takes them as inputs), which makes every running sum
# a chosen number.
S_DESC = np.array([8.0, 7.0, 6.0, 5.0, 4.0, 3.0, 2.0, 1.0])
P_ROW = np.array([0.5, 0.3, 0.1, 0.05, 0.03, 0.01, 0.005, 0.005])


def classify(gpu_kept, s, P, p, k_min):
    s = np.asarray(s, dtype=np.float64)[None, :]
    P = np.asarray(P, dtype=np.float64)[None, :]
    ref = topp_select(s, P, p, k_min)
    g = np.zeros_like(ref["mask"])
    g[0, list(gpu_kept)] = 1
    res = compare_mask_rows(g, ref["mask"], ref["order"], ref["cum"], s, ref["counts"], p, k_min)
    return ref, res


def counts_of(res):
    return res["band"], res["tie"], res["mismatch"]


def c(r):
    """Running sum c_r of P_ROW in rank order (c_0 = 0)."""
    return float(np.cumsum(P_ROW)[r - 1]) if r > 0 else 0.0


def test_identical_masks_have_no_disagreement():
    ref, res = classify(range(3), S_DESC, P_ROW, 0.85, 2)
    assert int(ref["counts"][0]) == 3
    assert counts_of(res) == (0, 0, 0) and res["rows_with_diff"] == 0


def test_band_block_dropped_at_the_cut():
    # p sits 3e-6 above c_3, so the oracle keeps rank 4 (c_4 >= p, c_3 < p);
    # the decision on rank 4 is c_3 >= p, within the band: a GPU that stops at
    # 3 blocks is band-tolerated.
    p = c(3) + 3e-6
    ref, res = classify(range(3), S_DESC, P_ROW, p, 2)
    assert int(ref["counts"][0]) == 4
    assert counts_of(res) == (1, 0, 0)


def test_exclusive_sum_decides_not_the_inclusive_one():
    # p sits 3e-6 below c_4 (far from c_3): the oracle keeps 4 blocks.
    p = c(4) - 3e-6
    ref, _ = classify(range(4), S_DESC, P_ROW, p, 2)
    assert int(ref["counts"][0]) == 4
    # dropping rank 4 hinges on c_3 >= p, far from p: a mismatch (a slip
    # reading c_4 here would call it band)
    _, res = classify(range(3), S_DESC, P_ROW, p, 2)
    assert counts_of(res) == (0, 0, 1)
    # keeping rank 5 as well hinges on c_4 >= p, within the band: tolerated
    # (a slip reading c_5 here would call it a mismatch)
    _, res = classify(range(5), S_DESC, P_ROW, p, 2)
    assert counts_of(res) == (1, 0, 0)


def test_block_inside_the_floor_is_a_mismatch_even_in_band():
    # Same p as the first band case, but k_min = 4: rank 4 is the floor's
    # own last rank, kept whatever the sums say.
    p = c(3) + 3e-6
    ref, res = classify(range(3), S_DESC, P_ROW, p, 4)
    assert int(ref["counts"][0]) == 4
    assert counts_of(res) == (0, 0, 1)
    # one rank above the floor the same band decision is tolerated
    p5 = c(4) + 3e-6
    ref, res = classify(range(4), S_DESC, P_ROW, p5, 4)
    assert int(ref["counts"][0]) == 5
    assert counts_of(res) == (1, 0, 0)


def test_plain_extra_block_is_a_mismatch():
    p = 0.85  # c_2 = 0.8 < p <= c_3 = 0.9: three blocks, no sum near p
    ref, res = classify([0, 1, 2, 7], S_DESC, P_ROW, p, 2)
    assert int(ref["counts"][0]) == 3
    # block 7 (rank 8) is not the next rank and not tied: mismatch; the GPU's
    # count 4 also moves the cut over rank 4, whose c_3 = 0.9 is far from p
    band, tie, mis = counts_of(res)
    assert band == 0 and tie == 0 and mis == 2


def test_extra_block_at_the_cut_outside_the_band_is_a_mismatch():
    _, res = classify(range(4), S_DESC, P_ROW, 0.85, 2)
    assert counts_of(res) == (0, 0, 1)


def test_exact_tie_swap_at_the_cut():
    s = S_DESC.copy()
    s[4] = s[3]  # blocks 3 and 4 tie; the oracle takes the lower id first
    P = P_ROW
    ref, res = classify([0, 1, 2, 4], s, P, 0.92, 2)
    assert int(ref["counts"][0]) == 4 and list(ref["kv_idx"][0]) == [0, 1, 2, 3]
    assert counts_of(res) == (0, 2, 0)


def test_swap_with_an_untied_block_is_a_mismatch():
    # keep rank 5 instead of rank 4 without a tie: the dropped block is the
    # GPU prefix's own cut (its score is s_cut), the kept one is not tied
    ref, res = classify([0, 1, 2, 4], S_DESC, P_ROW, 0.92, 2)
    assert int(ref["counts"][0]) == 4
    _, _, mis = counts_of(res)
    assert mis >= 1 and res["mismatch_rows"] == [0]


def test_non_prefix_set_is_a_mismatch_even_when_every_sum_is_in_band():
    # rank 4 carries almost no mass: c_3 and c_4 are both within 1e-5 of p.
    P = np.array([0.5, 0.3, 0.1, 2e-6, 0.05, 0.03, 0.01, 0.009998])
    cs = np.cumsum(P)
    p = float(cs[2]) + 1.5e-6  # c_3 < p <= c_4
    assert abs(cs[2] - p) <= BAND and abs(cs[3] - p) <= BAND
    ref, _ = classify(range(4), S_DESC, P, p, 2)
    assert int(ref["counts"][0]) == 4
    # a moved cut either way is fine: 3 blocks or 5 blocks
    _, res = classify(range(3), S_DESC, P, p, 2)
    assert counts_of(res) == (1, 0, 0)
    _, res = classify(range(5), S_DESC, P, p, 2)
    assert counts_of(res) == (1, 0, 0)
    # skipping rank 4 and keeping rank 5 is no rounding of the running sums
    _, res = classify([0, 1, 2, 4], S_DESC, P, p, 2)
    assert res["mismatch"] >= 1 and res["mismatch_rows"] == [0]
    # nor is keeping rank 6 without rank 5
    _, res = classify([0, 1, 2, 3, 5], S_DESC, P, p, 2)
    assert res["mismatch"] >= 1


def test_moved_cut_over_a_tie_swap_still_needs_the_band():
    # The GPU keeps five blocks, taking block 5 (tied with block 4) in place
    # of block 4. Rank 5's decision (c_4 >= p) is far from p = 0.85, so the
    # set is wrong although block 4 itself shows no disagreement with the
    # oracle's four-block set.
    s = S_DESC.copy()
    s[5] = s[4]
    ref, res = classify([0, 1, 2, 3, 5], s, P_ROW, 0.93, 2)
    assert int(ref["counts"][0]) == 4
    assert res["tie"] == 1 and res["mismatch"] == 1


@pytest.mark.parametrize("p", [0.0, 1.0])
def test_edges_p_zero_and_one(p):
    # p = 0 keeps the floor only; p = 1 keeps every block. Any other count
    # is a mismatch (no running sum is within the band of 0, and at p = 1 the
    # sums before the last rank are all at least 0.005 below p).
    ref, res = classify(range(2 if p == 0.0 else 8), S_DESC, P_ROW, p, 2)
    assert int(ref["counts"][0]) == (2 if p == 0.0 else 8)
    assert counts_of(res) == (0, 0, 0)
    _, res = classify(range(3 if p == 0.0 else 7), S_DESC, P_ROW, p, 2)
    assert counts_of(res) == (0, 0, 1)


def test_several_rows_are_counted_separately():
    s = np.stack([S_DESC, S_DESC])
    P = np.stack([P_ROW, P_ROW])
    p = c(3) + 3e-6
    ref = topp_select(s, P, p, 2)
    g = ref["mask"].copy()
    g[0, 3] = 0  # band
    g[1, 6] = 1  # plain mismatch (rank 7 out of order)
    res = compare_mask_rows(g, ref["mask"], ref["order"], ref["cum"], s, ref["counts"], p, 2)
    assert res["rows_with_diff"] == 2 and res["band"] == 1 and res["mismatch_rows"] == [1]
