"""Block-sparse attention over the retained blocks (oracle side).

For a query token n in query block i, the keys it sees are the real tokens of
every key block j with M_ij = 1 (§2.1: only selected query-key block pairs are
evaluated; §3.1: block-sparse attention runs after the mask is built):

    O_n = sum_{k in K(i)} softmax_k(tau * Q_n . K_k) V_k,   tau = 1/sqrt(d) by default.

A row whose mask is empty (possible only with k_min = 0 and p = 0) has
O_n = 0. Everything is fp64; padding tokens of partial blocks do not exist
here at all, because blocks hold real tokens only.
"""

import numpy as np

from .tiling import TileGeometry


def _scale(d: int, scale) -> float:
    if scale is None or scale <= 0:
        return 1.0 / np.sqrt(np.float64(d))
    return float(scale)


def attn_ref_rows(Q, K, V, mask, geo: TileGeometry, blocks, scale=None) -> dict:
    """Output of the query blocks listed in `blocks` for one head.

    Q, K, V: (N x d) arrays of one head; mask: (nb x nb) 0/1 for that head.
    Returns {i: (n_i x d) fp64} with the rows of block i in ascending token order.
    """
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    tau = _scale(Q.shape[1], scale)
    mask = np.asarray(mask)
    out = {}
    for i in blocks:
        qi = geo.block_tokens[i]
        kept = np.nonzero(mask[i])[0]
        if kept.size == 0:
            out[int(i)] = np.zeros((len(qi), Q.shape[1]))
            continue
        keys = np.concatenate([geo.block_tokens[j] for j in kept])
        S = tau * (Q[qi] @ K[keys].T)
        S -= S.max(axis=1, keepdims=True)
        E = np.exp(S)
        out[int(i)] = (E @ V[keys]) / E.sum(axis=1, keepdims=True)
    return out


def attn_ref_head(Q, K, V, mask, geo: TileGeometry, scale=None) -> np.ndarray:
    """Full (N x d) fp64 output of one head."""
    rows = attn_ref_rows(Q, K, V, mask, geo, range(geo.nb), scale)
    O = np.empty((geo.N, np.asarray(Q).shape[1]), dtype=np.float64)
    for i, o in rows.items():
        O[geo.block_tokens[i]] = o
    return O
