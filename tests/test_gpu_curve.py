"""GPU parity of the Hilbert-curve block organisation (§3.1, routing frontend).

* fva_curve_order equals the oracle's curve order bit for bit (integer work);
* fva_permute_tokens moves whole rows bit for bit, and a perm entry outside
  [0, tokens) zeroes a gathered row or drops a scattered one;
* fva_route and fva_attn on curve-ordered inputs with the one-dimensional
  tiling match the oracle run with curve blocks on the raster-ordered
  inputs: the mask by the routing rule (bit-exact except band and tie
  blocks, oracle/compare.py), the output (permuted back to raster order)
  within max 2e-2 / mean 1e-3.
"""

import numpy as np
import pytest

import synth
from oracle import attn_ref_head, attn_ref_rows, curve_geometry, curve_order, route_ref
from oracle.compare import ATTN_MAX_ABS, ATTN_MEAN_ABS, compare_mask_rows

from _gpu_util import attn_rule_errors, describe_rows, f64, lib, log, rule_rows, to_dev, torch_mod, workload

pytestmark = pytest.mark.gpu


def bits16(t):
    torch = torch_mod()
    return t.view(torch.int16).cpu().numpy()


@pytest.mark.parametrize(
    "grid",
    [(1, 1, 1), (2, 3, 5), (3, 16, 16), (21, 30, 52), (21, 45, 80), (31, 45, 80), (1, 256, 3), (256, 2, 1), (7, 1, 200)],
)
def test_curve_order_matches_oracle(grid):
    fva = lib()
    log(f"[curve] order {grid}")
    perm = fva.fva_curve_order(*grid, device="cuda:0")
    torch_mod().cuda.synchronize()
    assert np.array_equal(perm.cpu().numpy().astype(np.int64), curve_order(*grid))


def test_curve_order_twice_in_one_workspace():
    # The workspace is scratch: a second call over a smaller grid in the same
    # buffer must not see the first call's bitmap.
    fva, torch = lib(), torch_mod()
    ws = torch.empty(fva.fva_curve_workspace_size(21, 45, 80), dtype=torch.uint8, device="cuda:0")
    p1 = fva.fva_curve_order(21, 45, 80, device="cuda:0", workspace=ws)
    p2 = fva.fva_curve_order(5, 9, 11, device="cuda:0", workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(p1.cpu().numpy(), curve_order(21, 45, 80))
    assert np.array_equal(p2.cpu().numpy(), curve_order(5, 9, 11))


def test_permute_rows_strided_round_trip():
    fva, torch = lib(), torch_mod()
    N = 1000
    g = torch.Generator().manual_seed(4)
    big = torch.randn(2, 3, N, 192, generator=g).to(torch.bfloat16).to("cuda:0")
    x = big[..., :128]  # stride_n = 192
    perm = torch.randperm(N, generator=g).to(torch.int32)
    pd = perm.to("cuda:0")
    y = fva.fva_permute_tokens(x, pd, fva.FVA_TO_CURVE)
    z = fva.fva_permute_tokens(y, pd, fva.FVA_FROM_CURVE)
    torch.cuda.synchronize()
    xb = bits16(x)
    assert np.array_equal(bits16(y), xb[:, :, perm.numpy().astype(np.int64)])
    assert np.array_equal(bits16(z), xb)


def test_permute_rows_out_of_range_entries():
    fva, torch = lib(), torch_mod()
    N = 300
    x = torch.randn(1, 2, N, 128, generator=torch.Generator().manual_seed(9)).to(torch.bfloat16).to("cuda:0")
    perm = np.arange(N, dtype=np.int32)[::-1].copy()
    perm[5] = -1
    perm[7] = N
    pd = torch.from_numpy(perm).to("cuda:0")
    y = fva.fva_permute_tokens(x, pd, fva.FVA_TO_CURVE)
    sentinel = torch.full_like(x, 7.0)
    fva.fva_permute_tokens(x, pd, fva.FVA_FROM_CURVE, out=sentinel)
    torch.cuda.synchronize()
    xb, yb, sb = bits16(x), bits16(y), bits16(sentinel)
    ok = np.ones(N, bool)
    ok[[5, 7]] = False
    assert np.array_equal(yb[:, :, ok], xb[:, :, perm[ok]])
    assert not yb[:, :, ~ok].any()  # zero rows
    # scattered rows land at perm[r]; the targets of rows 5 and 7 (N-1-5, N-1-7) keep the sentinel
    assert np.array_equal(sb[:, :, perm[ok]], xb[:, :, ok])
    s7 = bits16(torch.full((1,), 7.0, dtype=torch.bfloat16))[0]
    assert np.all(sb[:, :, [N - 6, N - 8]] == s7)


def curve_run(Qb, Kb, Vb, grid, B, p, k_min):
    """Permute to curve order, route and attend on the GPU, permute O back."""
    fva, torch = lib(), torch_mod()
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    perm = fva.fva_curve_order(*grid, device="cuda:0")
    qc, kc, vc = (fva.fva_permute_tokens(t, perm, fva.FVA_TO_CURVE) for t in (q, k, v))
    tc = fva.Tiling.curve(q.shape[2], B)
    mask, counts, kv = fva.fva_route(qc, kc, p, k_min, tc)
    oc = fva.fva_attn(qc, kc, vc, tc, mask, counts, kv)
    o = fva.fva_permute_tokens(oc, perm, fva.FVA_FROM_CURVE)
    torch.cuda.synchronize()
    return mask.cpu().numpy(), counts.cpu().numpy(), kv.cpu().numpy(), o[0].float().cpu().numpy()


def check_mask(name, mask, counts, kv, Qb, Kb, geo, p, k_min):
    nb = geo.nb
    assert np.array_equal(mask.sum(axis=-1), counts)
    for h in range(mask.shape[1]):
        for i in range(nb):
            assert np.array_equal(kv[0, h, i, : counts[0, h, i]], np.nonzero(mask[0, h, i])[0])
    ref = route_ref(f64(Qb[0]), f64(Kb[0]), p, k_min, geo)
    cmp = compare_mask_rows(
        mask[0].reshape(-1, nb), ref["mask"].reshape(-1, nb), ref["order"].reshape(-1, nb),
        ref["cum"].reshape(-1, nb), ref["scores"].reshape(-1, nb), ref["counts"].reshape(-1), p, k_min,
    )
    log(f"[curve] {name}: nb={nb} mismatches={cmp['mismatch']} band={cmp['band']} tie={cmp['tie']} "
        f"density={counts.mean() / nb:.3f}")
    assert cmp["mismatch"] == 0, cmp


def test_curve_route_attn_tiny():
    cfg = synth.get_config("tiny")
    Qb, Kb, Vb = workload("tiny")
    geo = curve_geometry(*cfg.grid, 64)
    mask, counts, kv, O = curve_run(Qb, Kb, Vb, cfg.grid, 64, cfg.p, cfg.k_min)
    check_mask("tiny", mask, counts, kv, Qb, Kb, geo, cfg.p, cfg.k_min)
    errs = []
    for h in range(Qb.shape[1]):
        ref = attn_ref_head(f64(Qb[0, h]), f64(Kb[0, h]), f64(Vb[0, h]), mask[0, h], geo)
        errs.append(np.abs(O[h] - ref).ravel())
    e = np.concatenate(errs)
    log(f"[curve] tiny attn: max abs {e.max():.3e} mean abs {e.mean():.3e}")
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS


@pytest.mark.parametrize("name", ["480p", "720p", "720p_stress", "long"])
def test_curve_route_attn_full_workloads(name):
    # masks of every head against the oracle; attention on every query block
    # of the lowest- and highest-density heads and of two random heads (the
    # partial last block included), plus 64 random (head, block) rows
    cfg = synth.get_config(name)
    Qb, Kb, Vb = workload(name)
    geo = curve_geometry(*cfg.grid, 128)
    mask, counts, kv, O = curve_run(Qb, Kb, Vb, cfg.grid, 128, cfg.p, cfg.k_min)
    check_mask(name, mask, counts, kv, Qb, Kb, geo, cfg.p, cfg.k_min)
    rows = rule_rows(counts[0], geo.nb, 17)
    emax, emean, n = attn_rule_errors(Qb, Kb, Vb, mask[0], O, geo, rows)
    log(f"[curve] {name} attn: {describe_rows(rows)}, {n} elements compared, max abs {emax:.3e} mean abs {emean:.3e}")
    assert emax <= ATTN_MAX_ABS and emean <= ATTN_MEAN_ABS


def test_permute_rows_batch_two_bhnd_layout():
    # [batch, tokens, heads, 128] storage viewed as [batch, heads, tokens, 128]
    fva, torch = lib(), torch_mod()
    N, H = 500, 3
    g = torch.Generator().manual_seed(6)
    store = torch.randn(2, N, H, 128, generator=g).to(torch.bfloat16).to("cuda:0")
    x = store.permute(0, 2, 1, 3)
    perm = torch.randperm(N, generator=g).to(torch.int32)
    y = fva.fva_permute_tokens(x, perm.to("cuda:0"), fva.FVA_TO_CURVE)
    torch.cuda.synchronize()
    xb = bits16(x)
    assert y.stride() == x.stride()
    assert np.array_equal(bits16(y), xb[:, :, perm.numpy().astype(np.int64)])
