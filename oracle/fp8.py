"""FP8 (E4M3) quantised-V attention (oracle side; test infrastructure).

The paper's runtime quantises V before attention on every step (§3.4,
overlap of the balance-plan search with GPU-side V quantisation); it does
not name the format. The reading taken here:

* format: OCP 8-bit floating point E4M3 (1 sign, 4 exponent bits with bias
  7, 3 mantissa bits; no infinities; S.1111.111 is NaN; largest finite
  value 448; subnormals m * 2^-9), values rounded to nearest, ties to even;
* V is scaled per (batch, head, channel) by a power of two, 2^e_d with
  e_d = max(-127, min{e : amax_d * 2^-e <= 448}) and amax_d the largest
  |V[., d]| over all tokens of the head, so the scaled values fit the format
  and the scaling itself is exact; the quantised V is 2^e_d * E4M3(V * 2^-e_d);
* attention then runs on the dequantised V with the same mask
  (attention.py); the probabilities P are also rounded to E4M3 inside the
  GPU kernel, which the oracle does not model (their effect is bounded in
  the tests instead).

Written from the format definition with numpy; nothing is shared with the
GPU library.
"""

import numpy as np

E4M3_MAX = 448.0
_MIN_NORMAL_EXP = -6  # smallest normal 2^-6
_SUB_QUANTUM = 2.0**-9  # subnormal spacing


def e4m3_decode(codes) -> np.ndarray:
    """Value of every E4M3 code (uint8 array) as fp64; NaN codes give NaN."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m * _SUB_QUANTUM, np.ldexp(1.0 + m / 8.0, e - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return sign * mag


def _round_half_even(x: np.ndarray) -> np.ndarray:
    return np.round(x)  # numpy rounds halves to the even integer


def e4m3_encode(x) -> np.ndarray:
    """E4M3 code of every value of x (|x| <= 448, finite), round to nearest even."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("values must be finite with |x| <= 448")
    sign = np.where(np.signbit(x), 0x80, 0)
    a = np.abs(x)
    sub = a < 2.0**_MIN_NORMAL_EXP
    # subnormal range: multiples of 2^-9 (a result of 8 is the smallest normal's code)
    q_sub = _round_half_even(a / _SUB_QUANTUM).astype(np.int64)
    # normal range: a = (1 + f) 2^E, mantissa rounded to 3 bits
    safe = np.where(sub, 1.0, a)
    E = np.floor(np.log2(safe)).astype(np.int64)
    # guard against log2 rounding at exact powers of two
    E = np.where(np.ldexp(1.0, E) > safe, E - 1, E)
    E = np.where(np.ldexp(1.0, E + 1) <= safe, E + 1, E)
    q = _round_half_even((safe / np.ldexp(1.0, E) - 1.0) * 8.0).astype(np.int64)
    E = np.where(q == 8, E + 1, E)
    q = np.where(q == 8, 0, q)
    code_norm = ((E + 7) << 3) | q
    code = np.where(sub, q_sub, code_norm)
    return (sign | code).astype(np.uint8)


def channel_exponents(V: np.ndarray) -> np.ndarray:
    """e_d for every channel of V (tokens x d): the smallest e with amax * 2^-e <= 448, at least -127."""
    amax = np.abs(np.asarray(V, dtype=np.float64)).max(axis=0)
    e = np.full(amax.shape, -127, dtype=np.int64)
    nz = amax > 0
    # start from the binary exponent and step to the smallest valid e
    est = np.where(nz, np.ceil(np.log2(np.where(nz, amax, 1.0) / E4M3_MAX)), -127).astype(np.int64)
    est = np.maximum(est, -127)
    for _ in range(2):
        too_small = nz & (np.ldexp(amax, -est) > E4M3_MAX)
        est = np.where(too_small, est + 1, est)
        can_lower = nz & (est > -127) & (np.ldexp(amax, -(est - 1)) <= E4M3_MAX)
        est = np.where(can_lower, est - 1, est)
    e = np.where(nz, est, e)
    return e


def quantize_v(V: np.ndarray):
    """(codes uint8 [tokens, d], exponents int64 [d]) of one head's V."""
    V = np.asarray(V, dtype=np.float64)
    e = channel_exponents(V)
    codes = e4m3_encode(np.ldexp(V, -e[None, :]))
    return codes, e


def dequantize_v(codes: np.ndarray, e: np.ndarray) -> np.ndarray:
    return np.ldexp(e4m3_decode(codes), np.asarray(e)[None, :])


def p_rounding_bound(Q, K, Vq, mask, geo, rows, scale=None, u=2.0**-4):
    """Per-element bounds on the effect of rounding P to E4M3 (relative error <= u).

    For each query block i in `rows` returns (bound, rms), both (n_i x d):
    with w_k the exact softmax weights of the row and O' the exact output on
    the dequantised V, a relative error eps_k (|eps_k| <= u) on every P_k
    changes the normalised output by sum_k w_k eps_k (v_k - O') / (1 + sum_k
    w_k eps_k), so
        bound = u / (1 - u) * sum_k w_k |v_k - O'|,
        rms   = u * sqrt(sum_k w_k^2 (v_k - O')^2)   (the size of the sum for
                independent errors of spread u).
    """
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    Vq = np.asarray(Vq, dtype=np.float64)
    d = Q.shape[1]
    tau = 1.0 / np.sqrt(np.float64(d)) if scale is None or scale <= 0 else float(scale)
    out = {}
    for i in rows:
        qi = geo.block_tokens[i]
        kept = np.nonzero(mask[i])[0]
        if kept.size == 0:
            z = np.zeros((len(qi), d))
            out[int(i)] = (z, z)
            continue
        keys = np.concatenate([geo.block_tokens[j] for j in kept])
        S = tau * (Q[qi] @ K[keys].T)
        S -= S.max(axis=1, keepdims=True)
        Wt = np.exp(S)
        Wt /= Wt.sum(axis=1, keepdims=True)
        O = Wt @ Vq[keys]
        bound = np.empty_like(O)
        rms = np.empty_like(O)
        for c in range(d):
            dev = Vq[keys, c][None, :] - O[:, c][:, None]
            bound[:, c] = (Wt * np.abs(dev)).sum(axis=1)
            rms[:, c] = np.sqrt((Wt * Wt * dev * dev).sum(axis=1))
        out[int(i)] = (bound * u / (1.0 - u), rms * u)
    return out
