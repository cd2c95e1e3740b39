"""GPU parity of the FP8 (E4M3) quantised-V variant against the oracle.

* fva_quantize_v is exact integer/byte work: the exponents and every code of
  every tile must equal the oracle's quantiser (oracle/fp8.py) bit for bit,
  read through the layout include/fva.h documents.
* fva_attn_fp8v is compared with the fp64 oracle run on the dequantised V
  (the exact effect of the V rounding) with the same mask. The one rounding
  the oracle does not model is that of the probabilities to E4M3: relative
  2^-4 in the format's normal range, at most half a subnormal quantum
  (2^-17 of the row maximum) below it, the value itself where it flushes to
  zero; oracle.fp8.p_rounding_bound turns that into a bound on each output
  element (exact form on small cases, heavy keys exact plus a Cauchy-Schwarz
  tail on the full-size row sets). Bar, per element: |O - O'| <= that bound +
  1e-2, the error of the rest of the arithmetic (bf16 Q K^T products, fp32
  softmax and accumulation, bf16 output): the bf16 path, which does the same
  arithmetic with bf16 instead of E4M3 probabilities, stays within 9.6e-3 of
  the fp64 oracle on every case measured (largest of its parity cases: the
  stress workload on Hilbert-curve blocks). Over
  all compared elements: mean |O - O'| <= 1e-3 + mean of
  sqrt(sum_k (c_k w_k)^2 (v_k - O')^2) (the spread of the rounding sum for
  independent errors).
"""

import numpy as np
import pytest

import synth
from oracle import attn_ref_rows, curve_geometry, tile_geometry
from oracle.fp8 import dequantize_v, p_rounding_bound, quantize_v

from _gpu_util import (
    custom_config,
    describe_rows,
    f64,
    geometry_of,
    lib,
    log,
    map_blocks,
    rule_rows,
    tiling_of,
    to_dev,
    torch_mod,
    workload,
)

pytestmark = pytest.mark.gpu

ALLOW_OWN = 1e-2  # the rest of the arithmetic; the bf16 path's largest measured error is 9.6e-3
ALLOW_MEAN = 1e-3


def kap_of_pos():
    p = np.arange(128)
    g, hb, t, r = p >> 5, (p >> 4) & 1, (p >> 2) & 3, p & 3
    return 64 * hb + 32 * (t >> 1) + 8 * g + 4 * (t & 1) + r


def expected_tiles(codes, geo):
    """Oracle codes [N, 128] of one head -> tiles [nb, 128 d, 128 p] in the documented layout."""
    kap = kap_of_pos()
    out = np.zeros((geo.nb, 128, 128), np.uint8)
    for j, toks in enumerate(geo.block_tokens):
        real = kap < len(toks)
        out[j][:, real] = codes[toks[kap[real]]].T
    return out


def check_quantizer(name, Vb, tiling, geo, heads=None):
    fva, torch = lib(), torch_mod()
    v = to_dev(Vb)
    v8, vexp = fva.fva_quantize_v(v, tiling)
    torch.cuda.synchronize()
    v8, vexp = v8.cpu().numpy(), vexp.cpu().numpy()
    heads = range(Vb.shape[1]) if heads is None else heads
    for b in range(Vb.shape[0]):
        for h in heads:
            codes, e = quantize_v(f64(Vb[b, h]))
            assert np.array_equal(vexp[b, h], e), (name, b, h)
            assert np.array_equal(v8[b, h], expected_tiles(codes, geo)), (name, b, h)
    log(f"[fp8] quantizer {name}: {len(list(heads))} heads bit-exact")


@pytest.mark.parametrize("grid,tile", [((3, 16, 16), (1, 8, 8)), ((5, 13, 21), (2, 8, 8)), ((3, 9, 10), (1, 8, 8))])
def test_quantize_v_bit_exact(grid, tile):
    cfg = custom_config("q", 3, grid, tile, (0.3, 1.5, 5.0), seed=13)
    _, _, Vb = synth.gen_qkv(cfg)
    # channels of very different magnitude, an all-zero channel and a tiny one
    V = synth.bf16_bits_to_f32(Vb).astype(np.float64)
    V *= np.exp2(np.arange(128) % 40 - 20)[None, None, None, :]
    V[..., 7] = 0.0
    V[..., 9] *= 1e-30
    Vb = synth.f32_to_bf16_bits(V.astype(np.float32))
    check_quantizer(f"{grid}", Vb, tiling_of(cfg), geometry_of(cfg))


def test_quantize_v_curve_tiling():
    fva = lib()
    cfg = synth.get_config("tiny")
    _, _, Vb = workload("tiny")
    perm = fva.fva_curve_order(*cfg.grid, device="cuda:0").cpu().numpy().astype(np.int64)
    Vc = np.ascontiguousarray(Vb[:, :, perm])  # curve order on the host
    geo = curve_geometry(*cfg.grid, 64)
    # the GPU sees the permuted rows as one line: its block j is curve ranks [64j, 64j + 64)
    lin = tile_geometry(1, 1, cfg.N, 1, 1, 64)  # runs of 64 consecutive positions
    assert all(np.array_equal(perm[lin.block_tokens[j]], geo.block_tokens[j]) for j in range(geo.nb))
    check_quantizer("tiny-curve", Vc, fva.Tiling.curve(cfg.N, 64), lin)


def fp8_attn(Qb, Kb, Vb, tiling, mask_t, counts_t=None, kv_t=None, flags=0):
    fva, torch = lib(), torch_mod()
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    v8, vexp = fva.fva_quantize_v(v, tiling)
    out = fva.fva_attn_fp8v(q, k, v8, vexp, tiling, mask_t, counts_t, kv_t, flags=flags)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def compare_rows(name, Qb, Kb, Vb, mask, O, geo, rows_by_head):
    """Bar of the module docstring over the given (head -> query blocks)."""
    over, errs, rmss, errs_exact = [], [], [], []
    for h, rows in rows_by_head.items():
        Qh, Kh, Vh = f64(Qb[0, h]), f64(Kb[0, h]), f64(Vb[0, h])
        codes, e = quantize_v(Vh)
        Vq = dequantize_v(codes, e)
        ref_q = attn_ref_rows(Qh, Kh, Vq, mask[h], geo, rows)
        ref = attn_ref_rows(Qh, Kh, Vh, mask[h], geo, rows)
        bnd = p_rounding_bound(Qh, Kh, Vq, mask[h], geo, rows)
        for i in rows:
            toks = geo.block_tokens[i]
            err = np.abs(O[h][toks] - ref_q[i])
            bound, rms = bnd[i]
            over.append((err - bound).ravel())
            errs.append(err.ravel())
            rmss.append(rms.ravel())
            errs_exact.append(np.abs(O[h][toks] - ref[i]).ravel())
    over, errs, rmss, ex = (np.concatenate(x) for x in (over, errs, rmss, errs_exact))
    log(f"[fp8] {name}: vs dequantised-V oracle max {errs.max():.3e} mean {errs.mean():.3e} "
        f"(max excess over the P bound {over.max():.3e}, mean rms {rmss.mean():.3e}); "
        f"vs unquantised oracle max {ex.max():.3e} mean {ex.mean():.3e}")
    assert over.max() <= ALLOW_OWN, over.max()
    assert errs.mean() <= ALLOW_MEAN + rmss.mean(), (errs.mean(), rmss.mean())
    return errs, ex


def test_fp8_attn_tiny_both_schedulers_and_rebuilt_lists():
    fva, torch = lib(), torch_mod()
    cfg = synth.get_config("tiny")
    Qb, Kb, Vb = workload("tiny")
    geo = geometry_of(cfg)
    tiling = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(to_dev(Qb), to_dev(Kb), cfg.p, cfg.k_min, tiling)
    m = mask.cpu().numpy()[0]
    rows = {h: list(range(geo.nb)) for h in range(cfg.heads)}
    O_p = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv, flags=fva.FVA_SCHED_PERSISTENT)
    compare_rows("tiny persistent", Qb, Kb, Vb, m, O_p[0], geo, rows)
    O_n = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    O_m = fp8_attn(Qb, Kb, Vb, tiling, mask)
    assert np.array_equal(O_p, O_n) and np.array_equal(O_p, O_m)  # same item body, same order
    O_s = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv, flags=fva.FVA_SPLIT_BLOCKS(2))
    compare_rows("tiny split 2", Qb, Kb, Vb, m, O_s[0], geo, rows)


@pytest.mark.parametrize("kind", ["ones", "random50"])
@pytest.mark.parametrize("grid,tile", [((5, 13, 21), (2, 8, 8)), ((3, 9, 10), (1, 8, 8))])
def test_fp8_attn_host_masks_partial_blocks(kind, grid, tile):
    torch = torch_mod()
    cfg = custom_config("fp8mask", 3, grid, tile, (0.3, 1.5, 5.0), seed=17)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    geo = geometry_of(cfg)
    rng = np.random.default_rng(23)
    if kind == "ones":
        m = np.ones((1, 3, geo.nb, geo.nb), np.uint8)
    else:
        m = (rng.random((1, 3, geo.nb, geo.nb)) < 0.5).astype(np.uint8)
        m[0, :, np.arange(geo.nb), np.arange(geo.nb)] = 1
    O = fp8_attn(Qb, Kb, Vb, tiling_of(cfg), torch.from_numpy(m).to("cuda:0"))
    compare_rows(f"{grid} {kind}", Qb, Kb, Vb, m[0], O[0], geo, {h: list(range(geo.nb)) for h in range(3)})


@pytest.mark.parametrize("s", [1, 3])
def test_fp8_attn_empty_rows_and_forced_splits(s):
    # Partial blocks (21 = 2*10 + 1 frames, 13 = 8 + 5 rows) with every third
    # query block keeping nothing: those rows must be exactly zero, whole rows
    # and rows cut into chunks of s kept blocks (combined from partials) must
    # meet the same bar against the oracle.
    fva = lib()
    cfg = custom_config("fp8split", 3, (5, 13, 21), (2, 8, 8), (0.3, 1.5, 5.0), seed=29)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    geo = geometry_of(cfg)
    rng = np.random.default_rng(31)
    m = (rng.random((1, 3, geo.nb, geo.nb)) < 0.6).astype(np.uint8)
    empty = list(range(0, geo.nb, 3))
    m[0, :, empty, :] = 0
    mt = torch_mod().from_numpy(m).to("cuda:0")
    kept = {h: [i for i in range(geo.nb) if i not in empty] for h in range(3)}
    for flags, name in [(0, "whole rows"), (fva.FVA_SPLIT_BLOCKS(s), f"chunks of {s}")]:
        O = fp8_attn(Qb, Kb, Vb, tiling_of(cfg), mt, flags=flags)
        for h in range(3):
            for i in empty:
                assert np.all(O[0, h][geo.block_tokens[i]] == 0), (name, h, i)
        compare_rows(f"empty rows, {name}", Qb, Kb, Vb, m[0], O[0], geo, kept)


def compare_rule(name, Qb, Kb, Vb, mask, O, geo, rows):
    """The bar of the module docstring over {head: query blocks} at full size:
    the dequantised-V output and the bound (heavy keys exact, Cauchy-Schwarz
    tail) from one oracle pass per block, in the thread pool."""
    emax, esum, rsum, n, worst = 0.0, 0.0, 0.0, 0, -np.inf
    for h, blocks in rows.items():
        Qh, Kh = f64(Qb[0, h]), f64(Kb[0, h])
        codes, e = quantize_v(f64(Vb[0, h]))
        Vq = dequantize_v(codes, e)
        mh = mask[h]

        def part(chunk):
            res = p_rounding_bound(Qh, Kh, Vq, mh, geo, chunk, method="cauchy", with_output=True)
            out = {}
            for i, (o_ref, bound, rms) in res.items():
                err = np.abs(O[h][geo.block_tokens[i]] - o_ref)
                out[i] = (float(err.max()), float(err.sum()), float(rms.sum()), int(err.size),
                          float((err - bound).max()))
            return out

        for mx, sm, rs, cnt, ov in map_blocks(part, blocks).values():
            emax = max(emax, mx)
            esum += sm
            rsum += rs
            n += cnt
            worst = max(worst, ov)
    log(f"[fp8] {name}: {describe_rows(rows)}, {n} elements compared, vs dequantised-V oracle max {emax:.3e} "
        f"mean {esum / n:.3e} (max excess over the P bound {worst:.3e}, mean rms {rsum / n:.3e})")
    assert worst <= ALLOW_OWN, worst
    assert esum / n <= ALLOW_MEAN + rsum / n, (esum / n, rsum / n)


@pytest.mark.parametrize("name", ["480p", "720p", "720p_stress", "long"])
def test_fp8_attn_full_workloads_rule(name):
    # every query block of the lowest- and highest-density heads and of two
    # random heads, plus 64 random (head, block) rows
    fva = lib()
    cfg = synth.get_config(name)
    Qb, Kb, Vb = workload(name)
    geo = geometry_of(cfg)
    tiling = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(to_dev(Qb), to_dev(Kb), cfg.p, cfg.k_min, tiling)
    O = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv)
    m = mask.cpu().numpy()[0]
    c = counts.cpu().numpy()[0]
    compare_rule(name, Qb, Kb, Vb, m, O[0], geo, rule_rows(c, geo.nb, 29))


def test_fp8_attn_deterministic():
    fva = lib()
    cfg = synth.get_config("480p")
    Qb, Kb, Vb = workload("480p")
    tiling = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(to_dev(Qb), to_dev(Kb), cfg.p, cfg.k_min, tiling)
    O1 = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv)
    O2 = fp8_attn(Qb, Kb, Vb, tiling, mask, counts, kv)
    assert np.array_equal(O1, O2)


@pytest.mark.parametrize("name,B", [("tiny", 64), ("480p", 128)])
def test_fp8_attn_hilbert_blocks(name, B):
    # curve order + E4M3 V: the whole variant stack, against the oracle on
    # curve blocks and dequantised V (raster order), under the same bar
    fva, torch = lib(), torch_mod()
    cfg = synth.get_config(name)
    Qb, Kb, Vb = workload(name)
    geo = curve_geometry(*cfg.grid, B)
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    perm = fva.fva_curve_order(*cfg.grid, device="cuda:0")
    qc, kc, vc = (fva.fva_permute_tokens(t, perm, fva.FVA_TO_CURVE) for t in (q, k, v))
    tc = fva.Tiling.curve(cfg.N, B)
    mask, counts, kv = fva.fva_route(qc, kc, cfg.p, cfg.k_min, tc)
    v8, vexp = fva.fva_quantize_v(vc, tc)
    oc = fva.fva_attn_fp8v(qc, kc, v8, vexp, tc, mask, counts, kv)
    O = fva.fva_permute_tokens(oc, perm, fva.FVA_FROM_CURVE).float().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    m = mask.cpu().numpy()[0]
    # the quantiser saw the permuted rows, whose channel maxima are the same
    assert np.array_equal(vexp.cpu().numpy()[0], np.stack([quantize_v(f64(Vb[0, h]))[1] for h in range(cfg.heads)]))
    if geo.nb <= 16:
        compare_rows(f"{name} hilbert", Qb, Kb, Vb, m, O[0], geo, {h: list(range(geo.nb)) for h in range(cfg.heads)})
    else:
        compare_rule(f"{name} hilbert", Qb, Kb, Vb, m, O[0], geo, rule_rows(counts.cpu().numpy()[0], geo.nb, 37))


def test_fp8_attn_batch_two_odd_heads():
    fva, torch = lib(), torch_mod()
    cfg = synth.WorkloadConfig("fp8b2", 3, (5, 13, 21), (2, 8, 8), 0.9, 3, 19, "fixed", (0.7, 2.5, 4.0), batch=2)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    geo = geometry_of(cfg)
    t = tiling_of(cfg)
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, t)
    v8, vexp = fva.fva_quantize_v(v, t)
    O = fva.fva_attn_fp8v(q, k, v8, vexp, t, mask, counts, kv).float().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    for b in range(2):
        sel = lambda X: X[b:b + 1]
        compare_rows(f"batch {b}", sel(Qb), sel(Kb), sel(Vb), mask.cpu().numpy()[b], O[b], geo,
                     {h: list(range(geo.nb)) for h in range(3)})


def test_fp8_attn_max_blocks_sampled():
    # nb = 1024, the largest supported block count (16 x 128 x 64 tokens, 2x8x8 boxes)
    fva, torch = lib(), torch_mod()
    cfg = custom_config("fp8max", 1, (16, 128, 64), (2, 8, 8), (1.5,), seed=11)
    geo = geometry_of(cfg)
    assert geo.nb == 1024
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    t = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(to_dev(Qb), to_dev(Kb), cfg.p, cfg.k_min, t)
    O = fp8_attn(Qb, Kb, Vb, t, mask, counts, kv)
    rows = {0: [0, 511, 777, 1023]}
    compare_rule("max blocks", Qb, Kb, Vb, mask.cpu().numpy()[0], O[0], geo, rows)
