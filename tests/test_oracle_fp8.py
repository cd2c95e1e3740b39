"""Pins of the oracle's E4M3 codec, V quantiser and P-rounding bound.

Checked against the format's definition rather than the codec's own code:
closed-form code values, strict monotonicity over all finite codes,
encode-of-decode identity, brute-force nearest search, ties to even at
every midpoint, the exponent rule by its defining inequality, the
quantisation error bound, and the P-rounding bound against direct
perturbation of an explicit softmax.
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


def test_p_rounding_bound_holds_under_perturbation():
    # Explicit softmax of one row block, P perturbed by random relative
    # errors within u: the change of the normalised output stays inside the
    # bound, and the worst-case signs reach a good part of it.
    rng = np.random.default_rng(11)
    geo = tile_geometry(1, 8, 16, 1, 8, 8)  # 2 blocks of 64
    d = 8
    Q = rng.standard_normal((128, d)) * 2
    K = rng.standard_normal((128, d)) * 2
    V = rng.standard_normal((128, d))
    mask = np.ones((2, 2), np.uint8)
    u = 2.0**-4
    res = p_rounding_bound(Q, K, V, mask, geo, [0], u=u)
    bound, rms = res[0]
    qi = geo.block_tokens[0]
    S = (Q[qi] @ K.T) / np.sqrt(d)
    P = np.exp(S - S.max(axis=1, keepdims=True))
    O = (P @ V) / P.sum(axis=1, keepdims=True)
    worst = np.zeros_like(O)
    for trial in range(200):
        eps = rng.uniform(-u, u, P.shape)
        Pe = P * (1 + eps)
        Oe = (Pe @ V) / Pe.sum(axis=1, keepdims=True)
        worst = np.maximum(worst, np.abs(Oe - O))
        assert np.all(np.abs(Oe - O) <= bound * (1 + 1e-12))
    # signs chosen against each deviation reach the first-order bound closely
    for c in range(d):
        dev = V[:, c][None, :] - O[:, c][:, None]
        Pe = P * (1 + u * np.sign(dev))
        Oe = (Pe @ V[:, c]) / Pe.sum(axis=1)
        assert np.all(np.abs(Oe - O[:, c]) <= bound[:, c] * (1 + 1e-12))
        assert np.all(np.abs(Oe - O[:, c]) >= 0.9 * bound[:, c] * (1 - u))
    assert np.all(rms <= bound)
