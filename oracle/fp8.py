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
  GPU kernel, which the oracle does not model: p_rounding_bound bounds their
  effect, normal range, subnormals and flush to zero included.

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


# The GPU kernel rounds every probability as v = x * 2^(7 + delta) to E4M3,
# x = exp(s - s_max) being the probability relative to the row's maximum and
# delta >= 0 the distance (in powers of two) from the row's maximum down to the
# exponent reference the kernel held when it rounded that key (the reference
# never exceeds the running maximum). Hence, in units of x:
#   * x >= 2^-13 (v >= 2^-6, the smallest normal): |dx| <= u x (3-bit
#     mantissa, round to nearest: u = 2^-4);
#   * x < 2^-13 (v possibly subnormal, spacing 2^-9): |dv| <= min(v, 2^-10)
#     -- half a quantum, and values below half the smallest subnormal flush
#     to zero (|dv| = v) -- so |dx| <= min(x, 2^-17 * 2^-delta) <= min(x, 2^-17).
# Both cases together: |dx| <= c(x) x with c(x) = max(u, min(1, 2^-17 / x)),
# continuous in x (u at x = 2^-13, 1 at x = 2^-17), whatever delta >= 0 is, so
# the bound needs the row maximum only and not the kernel's reference.
P_PRESCALE_LOG2 = 7


def p_rounding_factors(x, u=2.0**-4, prescale_log2=P_PRESCALE_LOG2):
    """c(x): bound on |dx| / x for probabilities x <= 1 relative to the row maximum.

    x is rounded to E4M3 as x * 2^(prescale + delta) for any delta >= 0; the
    normal range starts at x = 2^(-6 - prescale), half a subnormal quantum is
    2^(-10 - prescale) in units of x.
    """
    x = np.asarray(x, dtype=np.float64)
    half_quantum = 2.0 ** (-10 - prescale_log2)
    with np.errstate(divide="ignore"):
        sub = np.where(x > 0, np.minimum(1.0, half_quantum / np.where(x > 0, x, 1.0)), 1.0)
    return np.maximum(u, sub)


def p_rounding_bound(Q, K, Vq, mask, geo, rows, scale=None, u=2.0**-4, prescale_log2=P_PRESCALE_LOG2,
                     method="exact", with_output=False, heavy_w=1e-3):
    """Per-element bounds on the effect of rounding P to E4M3.

    For each query block i in `rows` returns (bound, rms), both (n_i x d), or
    (O', bound, rms) with with_output. With x_k = exp(s_k - s_max) over the
    row's kept keys, Z = sum_k x_k, w_k = x_k / Z the exact softmax weights,
    O' = sum_k w_k v_k the exact output on the dequantised V, and the rounded
    x_k + e_k with |e_k| <= c_k x_k (c_k = p_rounding_factors(x_k)): the
    kernel's normalised output is sum_k (x_k + e_k) v_k / sum_k (x_k + e_k),
    and since sum_k x_k (v_k - O') = 0,
        O - O' = sum_k e_k (v_k - O') / (Z + sum_k e_k),
    so, with beta = sum_k c_k w_k < 1 and d_k = v_k - O',
        exact:   bound = sum_k c_k w_k |d_k| / (1 - beta)   (exact, not first order),
        cauchy:  the same sum taken exactly over the row's heavy keys
                 (w_k > heavy_w, at most 1 / heavy_w of them) and bounded by
                 Cauchy-Schwarz over the rest, sqrt(sum' c_k w_k) *
                 sqrt(sum' c_k w_k d_k^2), divided by (1 - beta): never below
                 the exact bound (up to fp64 cancellation in the expanded
                 squares, below 1e-7 absolute), and the light part is matrix
                 products only (for large row sets, where the exact sum costs
                 rows x keys x d),
        rms      = sqrt(sum_k (c_k w_k)^2 d_k^2)   (the size of the sum for
                 independent errors of that spread).
    A row with beta >= 1 gets an infinite bound (nothing is claimed for it).
    """
    if method not in ("exact", "cauchy"):
        raise ValueError("method is 'exact' or 'cauchy'")
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
            z = np.zeros((len(qi), Vq.shape[1]))
            out[int(i)] = (z, z, z) if with_output else (z, z)
            continue
        keys = np.concatenate([geo.block_tokens[j] for j in kept])
        S = tau * (Q[qi] @ K[keys].T)
        X = np.exp(S - S.max(axis=1, keepdims=True))
        Wt = X / X.sum(axis=1, keepdims=True)
        Vk = Vq[keys]
        O = Wt @ Vk
        CW = p_rounding_factors(X, u, prescale_log2) * Wt
        beta = CW.sum(axis=1)
        denom = np.where(beta < 1.0, 1.0 - beta, 0.0)
        if method == "exact":
            num = np.empty_like(O)
            ms = np.empty_like(O)
            for c in range(Vq.shape[1]):
                dev = Vk[:, c][None, :] - O[:, c][:, None]
                num[:, c] = (CW * np.abs(dev)).sum(axis=1)
                ms[:, c] = (CW * CW * dev * dev).sum(axis=1)
        else:
            # heavy keys exactly: one term per (query row, heavy key) pair
            heavy = Wt > heavy_w
            qh, kh = np.nonzero(heavy)  # row-major: pairs of one row are consecutive
            num = np.zeros_like(O)
            if qh.size:
                terms = CW[qh, kh][:, None] * np.abs(Vk[kh] - O[qh])
                starts = np.flatnonzero(np.r_[True, qh[1:] != qh[:-1]])
                num[qh[starts]] = np.add.reduceat(terms, starts, axis=0)
            # light keys by Cauchy-Schwarz, with
            # sum_k a_k (v_k - o)^2 = (a @ v^2) - 2 o (a @ v) + o^2 sum_k a_k
            V2 = Vk * Vk
            CL = np.where(heavy, 0.0, CW)
            bl = CL.sum(axis=1)
            var = CL @ V2 - 2.0 * O * (CL @ Vk) + O * O * bl[:, None]
            num += np.sqrt(bl[:, None] * np.maximum(var, 0.0))
            CW2 = CW * CW
            ms = CW2 @ V2 - 2.0 * O * (CW2 @ Vk) + O * O * CW2.sum(axis=1)[:, None]
        with np.errstate(divide="ignore", invalid="ignore"):
            bound = np.where(denom[:, None] > 0, num / np.where(denom > 0, denom, 1.0)[:, None], np.inf)
        rms = np.sqrt(np.maximum(ms, 0.0))
        out[int(i)] = (O, bound, rms) if with_output else (bound, rms)
    return out
