"""Comparison rules between a GPU result and the oracle (test infrastructure).

Mask rule (the band rule for Top-p, §2.1, made operational). For row
(b, h, i) take the oracle's order pi (score descending, ties to the lower
block id), its running sums c_r (c_0 = 0) and its kept count m. Let m' be the
number of blocks the GPU kept and pi_1 .. pi_m' the oracle's prefix of that
length. Every key block on which the GPU and the oracle disagree is then
exactly one of:

  * band-tolerated: its rank r lies between the two counts
    (min(m, m') < r <= max(m, m')), the GPU's choice for it agrees with the
    prefix of length m' (kept iff r <= m'), r exceeds the floor min(k_min, nb),
    and the running sum before it, c_{r-1}, lies within 1e-5 of p. Whether
    rank r joins the set hinges on the comparison c_{r-1} >= p, which
    rounding near p can flip; it cannot make the GPU skip a rank and keep a
    later one, nor reach inside the floor;
  * tie-tolerated: the GPU's choice for it disagrees with the prefix of
    length m' (the GPU's set is not that prefix there), and its score is
    within 1e-12 * max(1, |s_cut|) of s_cut, the score at rank m' (the cut of
    the GPU's own count): it swapped places with an equal-scored block;
  * a mismatch: anything else (required count: zero).

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

    gpu_mask, ref_mask: 0/1 [rows, nb]; order: the oracle's pi [rows, nb];
    cum: c_1 .. c_nb [rows, nb]; scores: s [rows, nb]; counts_ref: m [rows].
    Returns dict(mismatch, band, tie, rows_with_diff, mismatch_rows).
    """
    gpu_mask = np.asarray(gpu_mask).astype(bool)
    ref_mask = np.asarray(ref_mask).astype(bool)
    order = np.asarray(order)
    cum = np.asarray(cum, dtype=np.float64)
    scores = np.asarray(scores, dtype=np.float64)
    rows, nb = ref_mask.shape
    kf = min(int(k_min), nb)
    diff_rows = np.nonzero((gpu_mask != ref_mask).any(axis=1))[0]
    out = dict(mismatch=0, band=0, tie=0, rows_with_diff=int(diff_rows.size), mismatch_rows=[])
    for r in diff_rows:
        rank = np.empty(nb, dtype=np.int64)
        rank[order[r]] = np.arange(1, nb + 1)
        c = np.concatenate([[0.0], cum[r]])  # c[t] = c_t
        m = int(counts_ref[r])
        m_gpu = int(gpu_mask[r].sum())
        lo, hi = min(m, m_gpu), max(m, m_gpu)
        s_cut = scores[r][order[r][m_gpu - 1]] if m_gpu > 0 else None

        def band_ok(t):
            return t > kf and abs(c[t - 1] - p) <= BAND

        bad = False
        diffs = np.nonzero(gpu_mask[r] != ref_mask[r])[0]
        for j in diffs:
            rj = int(rank[j])
            in_prefix = rj <= m_gpu  # kept by the oracle's prefix of the GPU's length
            if gpu_mask[r][j] == in_prefix:
                # a moved cut: rank rj lies in (lo, hi] by construction
                if band_ok(rj):
                    out["band"] += 1
                    continue
            elif s_cut is not None and abs(scores[r][j] - s_cut) <= TIE_REL * max(1.0, abs(s_cut)):
                out["tie"] += 1
                continue
            out["mismatch"] += 1
            bad = True
        # A rank of the moved cut whose block took part in a tie swap is no
        # disagreement of its own; the decision at that rank still needs the band.
        diff_set = set(int(j) for j in diffs)
        for t in range(lo + 1, hi + 1):
            if int(order[r][t - 1]) not in diff_set and not band_ok(t):
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
