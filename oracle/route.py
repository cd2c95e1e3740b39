"""Routing frontend (oracle side): pooled block scores, softmax, Top-p + floor.

Follows, in the paper's order:

1. block-level similarities from pooled Q/K (§3.1, routing frontend):
   qbar_i, kbar_j are the means of Q and K over the real tokens of block i / j;
   s_ij = qbar_i . kbar_j / sqrt(d) (the scale is not printed; 1/sqrt(d) is the
   reading taken here, the usual attention scale);
2. normalised importance (§2.1): P_ij = softmax_j(s_ij) over all key blocks of
   the row;
3. Top-p (§2.1): keep key blocks in decreasing score order until their
   summed softmax mass is at least p. The blocks are taken in that order (ties
   to the lower block id), c_r is the running sum of their P, and
   m_p = min{r : c_r >= p}, or nb when no prefix reaches p; p = 1 keeps all
   blocks, as it does in exact arithmetic;
4. Top-k safety floor (§2.1, §3.1): m = max(m_p, min(k_min, nb));
5. the block mask M_ij (§2.1) keeps the first m blocks of that order;
   L_h = mean_i sum_j M_ij (§2.2, Eq. 1).

All arithmetic is fp64; bf16 inputs convert to fp64 exactly.
"""

import numpy as np

from .tiling import TileGeometry


def pool_blocks(X: np.ndarray, geo: TileGeometry) -> np.ndarray:
    """Mean of X (N x d) over the real tokens of every block -> (nb x d) fp64.

    Padding never enters the mean: a partial block divides by its own n_i.
    """
    X = np.asarray(X, dtype=np.float64)
    if X.shape[0] != geo.N:
        raise ValueError("token count does not match the grid")
    out = np.empty((geo.nb, X.shape[1]), dtype=np.float64)
    for i, toks in enumerate(geo.block_tokens):
        out[i] = X[toks].sum(axis=0) / len(toks)
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray) -> np.ndarray:
    """s_ij = qbar_i . kbar_j / sqrt(d), fp64."""
    d = qbar.shape[-1]
    return (qbar @ kbar.T) / np.sqrt(np.float64(d))


def block_softmax(s: np.ndarray) -> np.ndarray:
    """Row-wise softmax over all key blocks (no mask, no temperature)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def topp_select(s: np.ndarray, P: np.ndarray, p: float, k_min: int) -> dict:
    """Top-p selection with a Top-k floor for every row of s (rows x nb).

    Returns a dict with
      mask   uint8 [rows, nb]   M_ij
      counts int64 [rows]       m per row
      m_p    int64 [rows]       Top-p count before the floor
      order  int64 [rows, nb]   pi: block ids by decreasing score, ties -> lower id
      cum    fp64  [rows, nb]   c_r for r = 1..nb (sequential sums in pi order)
      kv_idx list of int64 arrays, the kept block ids of each row, ascending
    """
    s = np.asarray(s, dtype=np.float64)
    P = np.asarray(P, dtype=np.float64)
    rows, nb = s.shape
    p = float(p)
    if not (0.0 <= p <= 1.0):
        raise ValueError("p must lie in [0, 1]")
    if k_min < 0:
        raise ValueError("k_min must be non-negative")
    ids = np.broadcast_to(np.arange(nb), (rows, nb))
    order = np.lexsort((ids, -s), axis=-1)  # primary: score descending; secondary: id ascending
    cum = np.cumsum(np.take_along_axis(P, order, axis=-1), axis=-1)
    reached = cum >= p
    m_p = np.where(reached.any(axis=-1), reached.argmax(axis=-1) + 1, nb)
    if p <= 0.0:
        m_p[:] = 0  # c_0 = 0 already reaches p
    if p >= 1.0:
        # In exact arithmetic every P_ij > 0, so only the full set reaches 1;
        # a rounded running sum can touch 1.0 a few blocks early.
        m_p[:] = nb
    m = np.maximum(m_p, min(int(k_min), nb))
    mask = np.zeros((rows, nb), dtype=np.uint8)
    kv_idx = []
    for r in range(rows):
        kept = order[r, : m[r]]
        mask[r, kept] = 1
        kv_idx.append(np.sort(kept))
    return dict(mask=mask, counts=m.astype(np.int64), m_p=m_p.astype(np.int64), order=order, cum=cum, kv_idx=kv_idx)


def route_ref(Q: np.ndarray, K: np.ndarray, p: float, k_min: int, geo: TileGeometry) -> dict:
    """Route every head of Q, K (heads x N x d) -> per-head Top-p results.

    Returns a dict of arrays stacked over heads: mask [Hh, nb, nb],
    counts [Hh, nb], m_p, order, cum, scores, probs, and kv_idx
    (list over heads of lists over rows).
    """
    Q = np.asarray(Q)
    K = np.asarray(K)
    if Q.ndim != 3 or Q.shape != K.shape:
        raise ValueError("Q and K must both be (heads, N, d)")
    out = dict(mask=[], counts=[], m_p=[], order=[], cum=[], scores=[], probs=[], kv_idx=[])
    for h in range(Q.shape[0]):
        s = block_scores(pool_blocks(Q[h], geo), pool_blocks(K[h], geo))
        P = block_softmax(s)
        sel = topp_select(s, P, p, k_min)
        for key in ("mask", "counts", "m_p", "order", "cum", "kv_idx"):
            out[key].append(sel[key])
        out["scores"].append(s)
        out["probs"].append(P)
    for key in ("mask", "counts", "m_p", "order", "cum", "scores", "probs"):
        out[key] = np.stack(out[key])
    return out


def head_workload(counts: np.ndarray) -> np.ndarray:
    """L_h = mean_i sum_j M_{h,i,j} (Eq. 1); counts is [..., nb] per row."""
    return np.asarray(counts, dtype=np.float64).mean(axis=-1)
