"""Slack-aware sparse augmentation, single-GPU reading (oracle side).

§3.3 adds key blocks to the masks of ranks that would otherwise wait for the
slowest rank. With L_r the workload of rank r (the sum of Eq. 1's L_h over
its heads), L_max = max_r L_r and the slack dL_r = L_max - L_r (the slack
equation), a rank with dL_r > n2 * L_max (the trigger) receives the budget
B_r = n1 * dL_r (the budget equation) and spends it on not-yet-selected key
blocks in the routing's importance order, so L_r^aug = L_r + B_r.

Readings taken here (the paper leaves them open):

* the ranks are given by a head -> rank map over the heads one GPU holds
  (on R GPUs, each GPU would apply the same rule to its own rank);
* the budget is spread evenly over the rank's query-block rows: every row
  of every head of rank r keeps e_r = floor(B_r / H_r) more key blocks
  (H_r heads in the rank; a row with every block kept stays as it is), so
  the rank's workload grows by at most B_r;
* the added blocks are the next ones of the routing order (score
  descending, ties to the lower block id): a row keeps its first
  min(nb, m + e_r) blocks of that order;
* workloads are computed from exact integer sums: with S_h the sum of
  counts over the head's rows, L_h = S_h / nb, S_r = sum of S_h over the
  rank, and D_r = S_max - S_r. The trigger and the budget are decided in
  exact rational arithmetic on the values n1 and n2 hold:
      D_r > n2 * S_max,
      e_r = floor(n1 * D_r / (nb * H_r)).
  A kernel that evaluates them in floating point can decide otherwise only
  when one of the two exact quantities lies within its rounding of the
  boundary (D_r = n2 * S_max, or an integer quotient); boundary_ranks names
  those ranks and the values either decision gives.

Test infrastructure only; nothing here is shared with the GPU library.
"""

from fractions import Fraction

import numpy as np


def rank_loads(counts: np.ndarray, rank_of: np.ndarray, n_ranks: int):
    """S_r (integer sums of kept blocks over the rank's rows) and H_r per rank."""
    counts = np.asarray(counts, dtype=np.int64)  # [heads, nb]
    rank_of = np.asarray(rank_of, dtype=np.int64)
    S_h = counts.sum(axis=1)
    S_r = np.zeros(n_ranks, dtype=np.int64)
    H_r = np.zeros(n_ranks, dtype=np.int64)
    for h, r in enumerate(rank_of):
        S_r[r] += S_h[h]
        H_r[r] += 1
    return S_r, H_r


def _exact_decision(D: int, S_max: int, H: int, nb: int, n1: float, n2: float):
    """(trigger fired, floor quotient, trigger margin, quotient) of one rank, exact."""
    margin = Fraction(D) - Fraction(n2) * S_max
    q = Fraction(n1) * D / (nb * H)
    return margin > 0, int(q // 1), margin, q


def sasa_extras(counts, rank_of, n_ranks: int, n1: float, n2: float):
    """Extra blocks per row for every rank (int64 [n_ranks]) and the per-rank figures.

    Returns (extra_r, info) with info holding L_r, dL_r, B_r (as fractions of
    a row, i.e. in the units of Eq. 1) and whether the trigger fired.
    """
    counts = np.asarray(counts, dtype=np.int64)
    nb = counts.shape[1]
    S_r, H_r = rank_loads(counts, rank_of, n_ranks)
    S_max = int(S_r.max()) if n_ranks > 0 else 0
    extra = np.zeros(n_ranks, dtype=np.int64)
    fired = np.zeros(n_ranks, dtype=bool)
    for r in range(n_ranks):
        if H_r[r] == 0:
            continue
        fire, e, _, _ = _exact_decision(S_max - int(S_r[r]), S_max, int(H_r[r]), nb, n1, n2)
        fired[r] = fire
        extra[r] = e if fire else 0
    info = {
        "L_r": S_r / nb,
        "dL_r": (S_max - S_r) / nb,
        "B_r": np.where(fired, float(n1) * (S_max - S_r) / nb, 0.0),
        "fired": fired,
        "H_r": H_r,
    }
    return extra, info


def boundary_ranks(counts, rank_of, n_ranks: int, n1: float, n2: float, rel: float = 2.0**-48):
    """Ranks whose decision sits at a boundary, and the extras either side gives.

    A rank is at a boundary when its trigger margin D_r - n2 * S_max, or the
    distance of its quotient n1 * D_r / (nb * H_r) to the nearest integer,
    is within `rel` of the quantities involved (a few units of fp64
    rounding). Returns {rank: set of acceptable extra values}; ranks not in
    the dict have exactly one acceptable value, the exact one.
    """
    counts = np.asarray(counts, dtype=np.int64)
    nb = counts.shape[1]
    S_r, H_r = rank_loads(counts, rank_of, n_ranks)
    S_max = int(S_r.max()) if n_ranks > 0 else 0
    out = {}
    for r in range(n_ranks):
        if H_r[r] == 0:
            continue
        D = S_max - int(S_r[r])
        fire, e, margin, q = _exact_decision(D, S_max, int(H_r[r]), nb, n1, n2)
        fires = {fire}
        if abs(margin) <= Fraction(rel) * max(D, Fraction(n2) * S_max, 1):
            fires = {True, False}
        floors = {e}
        near = round(q)
        if abs(q - near) <= Fraction(rel) * max(q, 1):
            floors = {max(near - 1, 0), near}
        ok = {f if fr else 0 for fr in fires for f in floors}
        if len(ok) > 1:
            out[r] = ok
    return out


def augment_with(order: np.ndarray, counts: np.ndarray, rank_of, extra):
    """(mask, counts) when every row of rank r keeps min(nb, m + extra[r]) blocks of its order."""
    order = np.asarray(order)
    counts = np.asarray(counts, dtype=np.int64)
    heads, nb = counts.shape
    rank_of = np.asarray(rank_of, dtype=np.int64)
    new_counts = np.minimum(nb, counts + np.asarray(extra, dtype=np.int64)[rank_of][:, None])
    mask = np.zeros((heads, nb, nb), dtype=np.uint8)
    for h in range(heads):
        for i in range(nb):
            mask[h, i, order[h, i, : new_counts[h, i]]] = 1
    return mask, new_counts


def sasa_augment(order: np.ndarray, counts: np.ndarray, rank_of, n_ranks: int, n1: float, n2: float):
    """Augmented (mask, counts) of every head: first min(nb, m + e_r) blocks of each row's order.

    order: int [heads, nb, nb], the routing order of every row (score
    descending, ties to the lower id), as route_ref returns it.
    """
    extra, info = sasa_extras(counts, rank_of, n_ranks, n1, n2)
    mask, new_counts = augment_with(order, counts, rank_of, extra)
    return mask, new_counts, extra, info
