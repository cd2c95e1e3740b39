"""Comparison rules between a GPU result and the oracle (test infrastructure).

Mask rule. For row (b, h, i) take the oracle's order pi and running sums c_r.
A key block that the GPU and the oracle disagree on is
  * band-tolerated when its oracle rank r exceeds min(k_min, nb) and the
    running sum before it, c_{r-1}, lies within 1e-5 of p: whether it is kept
    hinges on the comparison c_{r-1} >= p, which rounding can flip;
  * tie-tolerated when its score is within 1e-12 * max(1, |s_cut|) of the
    score of the oracle's last kept block: it may swap with that block.
Every other disagreement is a mismatch; the required count is zero.

Attention rule: on the same mask, max |O_gpu - O_ref| <= 2e-2 and
mean |O_gpu - O_ref| <= 1e-3 over the compared real-token elements.
"""

import numpy as np

BAND = 1e-5
TIE_REL = 1e-12
ATTN_MAX_ABS = 2e-2
ATTN_MEAN_ABS = 1e-3


def compare_mask_rows(gpu_mask, ref_mask, order, cum, scores, counts_ref, p, k_min):
    """Classify GPU/oracle mask disagreements for a stack of rows (rows x nb).

    Returns dict(mismatch, band, tie, rows_with_diff, mismatch_rows).
    """
    gpu_mask = np.asarray(gpu_mask).astype(bool)
    ref_mask = np.asarray(ref_mask).astype(bool)
    rows, nb = ref_mask.shape
    kf = min(int(k_min), nb)
    diff_rows = np.nonzero((gpu_mask != ref_mask).any(axis=1))[0]
    out = dict(mismatch=0, band=0, tie=0, rows_with_diff=int(diff_rows.size), mismatch_rows=[])
    for r in diff_rows:
        rank = np.empty(nb, dtype=np.int64)
        rank[order[r]] = np.arange(1, nb + 1)
        c = np.concatenate([[0.0], cum[r]])
        m = int(counts_ref[r])
        s_cut = scores[r][order[r][m - 1]] if m > 0 else None
        bad = False
        for j in np.nonzero(gpu_mask[r] != ref_mask[r])[0]:
            rj = int(rank[j])
            if rj > kf and abs(c[rj - 1] - p) <= BAND:
                out["band"] += 1
            elif s_cut is not None and abs(scores[r][j] - s_cut) <= TIE_REL * max(1.0, abs(s_cut)):
                out["tie"] += 1
            else:
                out["mismatch"] += 1
                bad = True
        if bad:
            out["mismatch_rows"].append(int(r))
    return out


def attn_errors(o_gpu, o_ref):
    """(max abs, mean abs) error between two arrays of compared elements."""
    e = np.abs(np.asarray(o_gpu, dtype=np.float64) - np.asarray(o_ref, dtype=np.float64))
    if e.size == 0:
        return 0.0, 0.0
    return float(e.max()), float(e.mean())
