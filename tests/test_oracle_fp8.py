"""Pins of the oracle's E4M3 codec, V quantiser and P-rounding bound.

Checked against the format's definition rather than the codec's own code:
closed-form code values, strict monotonicity over all finite codes,
encode-of-decode identity, brute-force nearest search, ties to even at
every midpoint, the exponent rule by its defining inequality, the
quantisation error bound, the P-rounding factors against the codec itself
(normal range, subnormals, flush to zero), and the P-rounding bound against
direct perturbation of an explicit softmax and against codec-rounded rows.
"""

import numpy as np
import pytest

from oracle import tile_geometry
from oracle.fp8 import (
    E4M3_MAX,
    channel_exponents,
    dequantize_v,
    e4m3_decode,
    e4m3_encode,
    p_rounding_bound,
    p_rounding_factors,
    quantize_v,
)

ALL = np.arange(256, dtype=np.uint8)
FINITE = ALL[(ALL & 0x7F) != 0x7F]
POS = np.array([c for c in range(0x00, 0x7F)], dtype=np.uint8)  # +0 .. 448


def test_decode_closed_forms():
    v = e4m3_decode(ALL)
    assert v[0x00] == 0.0 and v[0x80] == 0.0 and np.signbit(v[0x80])
    assert v[0x01] == 2.0**-9 and v[0x07] == 7 * 2.0**-9
    assert v[0x08] == 2.0**-6 and v[0x0F] == 1.875 * 2.0**-6
    assert v[0x38] == 1.0 and v[0x39] == 1.125 and v[0x40] == 2.0
    assert v[0x7E] == 448.0 and v[0xFE] == -448.0
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF])
    assert np.sum(np.isnan(v)) == 2
    assert np.all(e4m3_decode(POS[1:]) > e4m3_decode(POS[:-1]))  # strictly increasing
    assert np.array_equal(e4m3_decode(FINITE | 0x80)[1:], -e4m3_decode(FINITE & 0x7F)[1:])


def test_encode_of_decode_is_identity():
    assert np.array_equal(e4m3_encode(e4m3_decode(FINITE)), FINITE)


def test_encode_is_nearest_by_brute_force():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.uniform(-448, 448, 4000), rng.normal(0, 1e-2, 4000), rng.normal(0, 3, 4000)])
    x = np.clip(x, -448, 448)
    table = e4m3_decode(FINITE)
    got = e4m3_decode(e4m3_encode(x))
    best = np.abs(x[:, None] - table[None, :]).min(axis=1)
    assert np.all(np.abs(got - x) == best)


def test_midpoints_round_to_even():
    lo, hi = e4m3_decode(POS[:-1]), e4m3_decode(POS[1:])
    mid = (lo + hi) / 2
    codes = e4m3_encode(mid)
    even = np.where(POS[:-1] % 2 == 0, POS[:-1], POS[1:])
    assert np.array_equal(codes, even)
    assert np.array_equal(e4m3_encode(-mid), even | 0x80)


def test_encode_rejects_out_of_range():
    with pytest.raises(ValueError):
        e4m3_encode([449.0])
    with pytest.raises(ValueError):
        e4m3_encode([np.nan])


def test_channel_exponent_rule():
    V = np.zeros((4, 6))
    V[:, 0] = [448.0, -1, 0, 2]  # amax 448 -> 0
    V[:, 1] = [0, 449.0, 0, 0]  # -> 1
    V[:, 2] = [-224.0, 0, 0, 0]  # 224 * 2 = 448 -> -1
    V[:, 3] = [1.0, 0.5, 0, 0]  # 1 * 2^8 = 256 <= 448 < 512 -> -8
    V[:, 4] = 0.0  # empty channel -> -127
    V[:, 5] = [3e-40, 0, 0, 0]  # tiny: clamped at -127
    e = channel_exponents(V)
    assert e.tolist() == [0, 1, -1, -8, -127, -127]
    rng = np.random.default_rng(5)
    W = rng.standard_normal((50, 64)) * np.exp2(rng.integers(-30, 30, 64))[None, :]
    e = channel_exponents(W)
    amax = np.abs(W).max(axis=0)
    assert np.all(np.ldexp(amax, -e) <= E4M3_MAX)
    assert np.all(np.ldexp(amax, -(e - 1)) > E4M3_MAX)


def test_quantisation_error_bound():
    rng = np.random.default_rng(8)
    V = rng.standard_normal((300, 16)) * np.exp2(rng.integers(-4, 4, 16))[None, :]
    codes, e = quantize_v(V)
    Vq = dequantize_v(codes, e)
    # relative 2^-4 in the normal range, half a subnormal quantum (2^(e-10)) below it
    bound = np.maximum(2.0**-4 * np.abs(V), np.ldexp(1.0, e - 10)[None, :])
    assert np.all(np.abs(Vq - V) <= bound)
    amax = np.abs(V).max(axis=0)
    assert np.all(np.abs(Vq).max(axis=0) <= np.ldexp(E4M3_MAX, e))
    assert np.all(np.abs(Vq).max(axis=0) >= amax * (1 - 2.0**-4))


def _softmax_parts(Q, K, V, rows_tok, d, tau=None):
    tau = 1.0 / np.sqrt(d) if tau is None else tau
    S = tau * (Q[rows_tok] @ K.T)
    X = np.exp(S - S.max(axis=1, keepdims=True))
    O = (X @ V) / X.sum(axis=1, keepdims=True)
    return X, O


def _codec_rounded(X, delta):
    """X rounded the way the kernel does it, through the oracle's own codec:
    E4M3(X * 2^(7 + delta)) * 2^-(7 + delta), delta >= 0 per key."""
    scale = np.exp2(7.0 + delta)
    return e4m3_decode(e4m3_encode(X * scale)) / scale


def test_p_rounding_factors_cover_the_codec():
    # |E4M3(x 2^(7+delta)) 2^-(7+delta) - x| <= c(x) x on a dense grid of x in
    # (2^-30, 1] and every delta in [0, 1] (the kernel's reference lies at most
    # one power of two below the row maximum when it rounds); flushed values
    # (rounded to 0) need c = 1, values in the subnormal range need more than u.
    x = np.exp2(-np.linspace(0.0, 30.0, 200001))
    for delta in (0.0, 0.25, 0.5, 0.999, 1.0, 3.0):
        xs = x[x * 2.0 ** (7 + delta) <= 256.0]  # the kernel rounds values <= 2^8
        r = _codec_rounded(xs, delta)
        c = p_rounding_factors(xs)
        assert np.all(np.abs(r - xs) <= c * xs * (1 + 1e-12)), delta
    r0 = _codec_rounded(x, 0.0)
    assert np.any((r0 == 0) & (x > 0))                      # flush to zero happens
    sub = (x < 2.0**-13) & (x > 2.0**-17)
    assert np.max(np.abs(r0 - x)[sub] / x[sub]) > 2.0**-4   # the normal-range u alone is not enough
    # the factor is tight: at each subnormal quantum midpoint the error reaches c(x) x
    mids = (np.arange(1, 8) + 0.5) * 2.0**-9 * 2.0**-7      # (k + 1/2) * subnormal quantum, in units of x
    err = np.abs(_codec_rounded(mids, 0.0) - mids)
    assert np.allclose(err, p_rounding_factors(mids) * mids, rtol=1e-12)
    assert p_rounding_factors(2.0**-13) == 2.0**-4 and p_rounding_factors(2.0**-17) == 1.0
    assert np.all(p_rounding_factors([1.0, 0.3, 2.0**-12]) == 2.0**-4)


def test_p_rounding_bound_holds_under_perturbation():
    # Explicit softmax of one row block, probabilities perturbed by the
    # largest errors the factors allow: random signs stay inside the bound,
    # and signs chosen against each deviation reach it up to (1-b)/(1+b).
    rng = np.random.default_rng(11)
    geo = tile_geometry(1, 8, 16, 1, 8, 8)  # 2 blocks of 64
    d = 8
    Q = rng.standard_normal((128, d)) * 2
    K = rng.standard_normal((128, d)) * 2
    V = rng.standard_normal((128, d))
    mask = np.ones((2, 2), np.uint8)
    res = p_rounding_bound(Q, K, V, mask, geo, [0])
    bound, rms = res[0]
    qi = geo.block_tokens[0]
    X, O = _softmax_parts(Q, K, V, qi, d)
    C = p_rounding_factors(X)
    assert np.any(C > 2.0**-4)  # this row has keys in the subnormal range
    beta = (C * X).sum(axis=1) / X.sum(axis=1)
    for trial in range(200):
        Xe = X * (1 + C * rng.uniform(-1, 1, X.shape))
        Oe = (Xe @ V) / Xe.sum(axis=1, keepdims=True)
        assert np.all(np.abs(Oe - O) <= bound * (1 + 1e-12))
    for c in range(d):
        dev = V[:, c][None, :] - O[:, c][:, None]
        Xe = X * (1 + C * np.sign(dev))
        Oe = (Xe @ V[:, c]) / Xe.sum(axis=1)
        assert np.all(np.abs(Oe - O[:, c]) <= bound[:, c] * (1 + 1e-12))
        assert np.all(np.abs(Oe - O[:, c]) >= bound[:, c] * (1 - beta) / (1 + beta) * (1 - 1e-12))
    assert np.all(rms <= bound)


def test_p_rounding_bound_holds_for_codec_rounding_wide_spread():
    # Rows with a wide logit spread (most keys in the subnormal or flush
    # range), P rounded through the oracle's own E4M3 codec at several
    # references below the row maximum: the output stays inside the bound;
    # the relative-u bound alone (no subnormal term) is broken by some of them.
    rng = np.random.default_rng(12)
    geo = tile_geometry(1, 8, 32, 1, 8, 8)  # 4 blocks of 64
    d = 16
    broke_u_only = False
    for spread in (2.0, 4.0, 8.0):
        Q = rng.standard_normal((256, d)) * spread
        K = rng.standard_normal((256, d)) * spread
        V = rng.standard_normal((256, d))
        mask = np.ones((4, 4), np.uint8)
        bnd = p_rounding_bound(Q, K, V, mask, geo, [1])
        bnd_u = p_rounding_bound(Q, K, V, mask, geo, [1], u=2.0**-4, prescale_log2=60)  # no subnormal term
        bound = bnd[1][0]
        qi = geo.block_tokens[1]
        X, O = _softmax_parts(Q, K, V, qi, d)
        for delta in (0.0, 0.5, 1.0, rng.uniform(0, 1, X.shape)):
            Xr = _codec_rounded(X, delta)
            Or = (Xr @ V) / Xr.sum(axis=1, keepdims=True)
            err = np.abs(Or - O)
            # 1e-14: the fp64 rounding of the two outputs themselves
            assert np.all(err <= bound * (1 + 1e-12) + 1e-14), (spread, delta)
            broke_u_only |= bool(np.any(err > bnd_u[1][0]))
    assert broke_u_only


def test_p_rounding_bound_is_reached_by_a_flushed_tail():
    # One key at the maximum with v = 0, a tail of 2^16 keys at x = 2^-18 with
    # v = 1: the codec flushes the whole tail, O' = 0.2 and the kernel's O = 0.
    # The bound (0.227) is within 15 % of that error.
    n = 1 << 16
    X = np.concatenate([[1.0], np.full(n, 2.0**-18)])
    v = np.concatenate([[0.0], np.ones(n)])
    Xr = _codec_rounded(X, 0.0)
    assert Xr[0] == 1.0 and not Xr[1:].any()
    O = (X @ v) / X.sum()
    Or = (Xr @ v) / Xr.sum()
    w = X / X.sum()
    C = p_rounding_factors(X)
    beta = (C * w).sum()
    bound = (C * w * np.abs(v - O)).sum() / (1 - beta)
    assert abs(O - 0.2) < 1e-12 and Or == 0.0
    assert 0.2 <= bound <= 0.2 / 0.85


def test_cauchy_bound_covers_the_exact_one_and_output_matches_attention():
    # The matrix-product form of the bound is never below the exact bound,
    # stays close to it on flat and on concentrated rows (heavy keys exact),
    # its rms equals the direct sum, and the output it returns is the
    # attention oracle's on the same V.
    from oracle import attn_ref_rows

    rng = np.random.default_rng(21)
    geo = tile_geometry(2, 8, 24, 1, 8, 8)  # 6 blocks of 64
    d = 32
    ratios = []
    for spread in (0.3, 1.0, 3.0, 6.0):
        Q = rng.standard_normal((geo.N, d)) * spread
        K = rng.standard_normal((geo.N, d)) * spread
        V = rng.standard_normal((geo.N, d)) * rng.uniform(0.5, 2, d)[None, :] + rng.uniform(-1, 1, d)[None, :]
        mask = (rng.random((geo.nb, geo.nb)) < 0.6).astype(np.uint8)
        mask[np.arange(geo.nb), np.arange(geo.nb)] = 1
        rows = list(range(geo.nb))
        ex = p_rounding_bound(Q, K, V, mask, geo, rows, with_output=True)
        cs = p_rounding_bound(Q, K, V, mask, geo, rows, method="cauchy", with_output=True)
        ref = attn_ref_rows(Q, K, V, mask, geo, rows)
        for i in rows:
            O_e, b_e, r_e = ex[i]
            O_c, b_c, r_c = cs[i]
            assert np.allclose(O_e, ref[i], rtol=0, atol=1e-12) and np.allclose(O_c, ref[i], rtol=0, atol=1e-12)
            assert np.all(b_c >= b_e * (1 - 1e-9) - 1e-7)
            assert np.allclose(r_c, r_e, rtol=1e-6, atol=1e-7)  # fp64 cancellation in the expanded squares
            ratios.append((b_c / np.maximum(b_e, 1e-300)).ravel())
    ratios = np.concatenate(ratios)
    assert np.median(ratios) < 1.5 and np.quantile(ratios, 0.99) < 4.0, (np.median(ratios), ratios.max())
