"""Pins of the oracle's block-sparse attention (§2.1 mask semantics, §3.1).

* p = 1 keeps every block, so the oracle must equal textbook dense softmax
  attention, written here independently;
* a token-level mask expanded from the block mask, applied to dense scores
  with -inf, must give the same output (partial tiles included);
* a per-token explicit loop on a tiny case (catches transposed operands);
* closed forms: constant V gives that constant; K = 0 gives the mean of the
  kept real V rows; an empty row gives 0.
"""

import numpy as np

from oracle import attn_ref_head, attn_ref_rows, route_ref, tile_geometry


def dense_attention(Q, K, V, scale):
    """softmax(scale * Q K^T) V, one head, fp64."""
    S = scale * (Q @ K.T)
    S = S - S.max(axis=1, keepdims=True)
    A = np.exp(S)
    A /= A.sum(axis=1, keepdims=True)
    return A @ V


def _rand_head(geo, d, seed):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((3, geo.N, d))


def test_p_one_equals_dense():
    geo = tile_geometry(3, 5, 7, 2, 2, 4)
    Q, K, V = _rand_head(geo, 16, 0)
    r = route_ref(Q[None], K[None], 1.0, 0, geo)
    assert np.all(r["mask"] == 1)
    O = attn_ref_head(Q, K, V, r["mask"][0], geo)
    np.testing.assert_allclose(O, dense_attention(Q, K, V, 1 / 4.0), rtol=0, atol=1e-12)


def test_token_mask_brute_force_partial_tiles():
    geo = tile_geometry(3, 5, 7, 2, 2, 4)
    Q, K, V = _rand_head(geo, 8, 1)
    rng = np.random.default_rng(2)
    mask = (rng.uniform(size=(geo.nb, geo.nb)) < 0.4).astype(np.uint8)
    mask[np.arange(geo.nb), rng.integers(0, geo.nb, geo.nb)] = 1  # no empty row
    scale = 0.3
    O = attn_ref_head(Q, K, V, mask, geo, scale)
    tok = mask[geo.block_of_token][:, geo.block_of_token].astype(bool)
    S = scale * (Q @ K.T)
    S[~tok] = -np.inf
    S -= S.max(axis=1, keepdims=True)
    A = np.exp(S)
    A /= A.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(O, A @ V, rtol=0, atol=1e-12)


def test_explicit_per_token_loop():
    geo = tile_geometry(2, 3, 4, 1, 2, 2)
    Q, K, V = _rand_head(geo, 4, 3)
    mask = np.zeros((geo.nb, geo.nb), np.uint8)
    mask[0, [0, 3]] = 1
    mask[1, [2]] = 1
    mask[2:, :] = 1
    O = attn_ref_head(Q, K, V, mask, geo, 0.5)
    for n in range(geo.N):
        i = geo.block_of_token[n]
        keys = [k for k in range(geo.N) if mask[i, geo.block_of_token[k]]]
        w = [np.exp(0.5 * sum(Q[n, c] * K[k, c] for c in range(4))) for k in keys]
        z = sum(w)
        for c in range(4):
            ref = sum(w[t] * V[keys[t], c] for t in range(len(keys))) / z
            assert abs(O[n, c] - ref) < 1e-12


def test_constant_v_and_zero_k():
    geo = tile_geometry(3, 5, 7, 2, 2, 4)
    Q, K, V = _rand_head(geo, 8, 4)
    rng = np.random.default_rng(5)
    mask = (rng.uniform(size=(geo.nb, geo.nb)) < 0.5).astype(np.uint8)
    mask[:, 0] = 1
    Vc = np.full_like(V, -1.75)
    np.testing.assert_allclose(attn_ref_head(Q, K, Vc, mask, geo), -1.75, atol=1e-13)
    out = attn_ref_rows(Q, np.zeros_like(K), V, mask, geo, range(geo.nb))
    for i, o in out.items():
        keys = np.concatenate([geo.block_tokens[j] for j in np.nonzero(mask[i])[0]])
        np.testing.assert_allclose(o, np.broadcast_to(V[keys].mean(axis=0), o.shape), atol=1e-13)


def test_empty_row_is_zero():
    geo = tile_geometry(2, 4, 4, 1, 2, 2)
    Q, K, V = _rand_head(geo, 4, 6)
    mask = np.ones((geo.nb, geo.nb), np.uint8)
    mask[3] = 0
    O = attn_ref_head(Q, K, V, mask, geo)
    assert np.all(O[geo.block_tokens[3]] == 0)
    assert np.all(np.isfinite(O))
