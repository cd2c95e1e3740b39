"""GPU parity of fva_attn against the fp64 oracle, on the same mask.

Bar: max |O_gpu - O_ref| <= 2e-2 and mean <= 1e-3 over compared real-token
elements. Small workloads compare every element; the full-size workloads
compare sampled query blocks (the lowest- and highest-density heads, two
more heads, plus random rows) in the launch configuration the benchmark
times (persistent scheduler, kept-block lists from fva_route).
"""

import zlib

import numpy as np
import pytest

import synth
from oracle import attn_ref_head, attn_ref_rows
from oracle.compare import ATTN_MAX_ABS, ATTN_MEAN_ABS, attn_errors

from _gpu_util import (
    attn_rule_errors,
    custom_config,
    describe_rows,
    f64,
    geometry_of,
    lib,
    log,
    rule_rows,
    tiling_of,
    to_dev,
    torch_mod,
    workload,
)

pytestmark = pytest.mark.gpu


def upload(Qb, Kb, Vb):
    return to_dev(Qb), to_dev(Kb), to_dev(Vb)


def run_attn(q, k, v, cfg, mask_t, counts_t=None, kv_t=None, flags=0, scale=0.0):
    fva = lib()
    out = fva.fva_attn(q, k, v, tiling_of(cfg), mask_t, counts_t, kv_t, flags=flags, scale=scale)
    torch_mod().cuda.synchronize()
    return out


def o64(out):
    return out.float().cpu().numpy().astype(np.float64)


def compare_full(name, Qb, Kb, Vb, cfg, mask, O, scale=None):
    geo = geometry_of(cfg)
    errs = []
    for b in range(Qb.shape[0]):
        for h in range(Qb.shape[1]):
            ref = attn_ref_head(f64(Qb[b, h]), f64(Kb[b, h]), f64(Vb[b, h]), mask[b, h], geo, scale)
            errs.append(np.abs(O[b, h] - ref))
    e = np.concatenate([x.ravel() for x in errs])
    log(f"[attn] {name}: max abs {e.max():.3e} mean abs {e.mean():.3e} over {e.size} elements")
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS
    return e.max(), e.mean()


def test_attn_tiny_routed_mask_both_schedulers():
    fva = lib()
    cfg = synth.get_config("tiny")
    Qb, Kb, Vb = workload("tiny")
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O_p = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_PERSISTENT)
    O_n = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    O_m = run_attn(q, k, v, cfg, mask)  # counts / kv_idx rebuilt from the mask
    assert torch_mod().equal(O_p, O_n) and torch_mod().equal(O_p, O_m)
    compare_full("tiny", Qb, Kb, Vb, cfg, mask.cpu().numpy(), o64(O_p))


MASK_KINDS = ["ones", "diagonal", "random30", "random70", "edge_only", "empty_rows"]


def make_mask(kind, B, H, nb, geo, rng):
    if kind == "ones":
        return np.ones((B, H, nb, nb), np.uint8)
    if kind == "diagonal":
        m = np.zeros((B, H, nb, nb), np.uint8)
        m[..., np.arange(nb), np.arange(nb)] = 1
        return m
    if kind.startswith("random"):
        dens = int(kind[6:]) / 100
        m = (rng.uniform(size=(B, H, nb, nb)) < dens).astype(np.uint8)
        m[..., np.arange(nb), rng.integers(0, nb, nb)] = 1
        return m
    if kind == "edge_only":
        small = geo.block_sizes < geo.block_sizes.max()
        m = np.zeros((B, H, nb, nb), np.uint8)
        m[..., :, small] = 1
        m[..., :, 0] = 1
        return m
    if kind == "empty_rows":
        m = (rng.uniform(size=(B, H, nb, nb)) < 0.5).astype(np.uint8)
        m[..., ::3, :] = 0
        return m
    raise ValueError(kind)


@pytest.mark.parametrize("kind", MASK_KINDS)
@pytest.mark.parametrize("grid,tile", [((5, 13, 21), (2, 8, 8)), ((3, 9, 10), (1, 8, 8)), ((3, 16, 16), (1, 8, 8))])
def test_attn_host_masks(kind, grid, tile):
    torch = torch_mod()
    fva = lib()
    cfg = custom_config("masks", 2, grid, tile, (0.5, 3.0), seed=21)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    mask = make_mask(kind, 1, 2, geo.nb, geo, np.random.default_rng(zlib.crc32(repr((kind, grid)).encode())))
    q, k, v = upload(Qb, Kb, Vb)
    mt = torch.from_numpy(mask).to("cuda:0")
    O = run_attn(q, k, v, cfg, mt)
    O_n = run_attn(q, k, v, cfg, mt, flags=fva.FVA_SCHED_NAIVE)
    assert torch.equal(O, O_n)
    Of = o64(O)
    compare_full(f"{kind} grid{grid}", Qb, Kb, Vb, cfg, mask, Of)
    if kind == "empty_rows":
        for i in range(0, geo.nb, 3):
            assert np.all(Of[:, :, geo.block_tokens[i]] == 0)


def test_attn_custom_scale_and_strided_layout():
    torch = torch_mod()
    cfg = custom_config("strided", 3, (3, 9, 10), (1, 8, 8), (0.5, 1.0, 3.0), seed=22)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    # [B, N, H, d] storage viewed as [B, H, N, d]
    def bnhd(bits):
        t = to_dev(np.ascontiguousarray(bits.transpose(0, 2, 1, 3)))
        return t.permute(0, 2, 1, 3)
    q, k, v = bnhd(Qb), bnhd(Kb), bnhd(Vb)
    assert q.stride(1) == 128 and q.stride(2) == 3 * 128
    mask = make_mask("random30", 1, 3, geo.nb, geo, np.random.default_rng(5))
    O = run_attn(q, k, v, cfg, torch.from_numpy(mask).to("cuda:0"), scale=0.05)
    compare_full("strided scale=0.05", Qb, Kb, Vb, cfg, mask, o64(O), scale=0.05)


def check_full(name, cfg, p, all_heads=False, seed=31):
    """Route and attend at full size in the benchmark's launch configuration
    (persistent scheduler, kept lists from fva_route), then compare the
    query blocks of rule_rows (all heads with all_heads) with the oracle."""
    fva = lib()
    geo = geometry_of(cfg)
    Qb, Kb, Vb = workload(cfg.name)
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, p, cfg.k_min, tiling_of(cfg))
    O = run_attn(q, k, v, cfg, mask, counts, kv)
    m = mask.cpu().numpy()[0]
    c = counts.cpu().numpy()[0]
    Of = O[0].float().cpu().numpy()
    del q, k, v, O
    rows = rule_rows(c, geo.nb, seed, all_heads=all_heads)
    emax, emean, n = attn_rule_errors(Qb, Kb, Vb, m, Of, geo, rows)
    log(f"[attn] {name} p={p}: {describe_rows(rows)}, {n} elements compared, max abs {emax:.3e} "
        f"mean abs {emean:.3e}, density {c.mean() / geo.nb:.3f}")
    assert emax <= ATTN_MAX_ABS and emean <= ATTN_MEAN_ABS


@pytest.mark.parametrize("name", ["720p", "720p_stress", "long"])
def test_attn_full_workloads_rule(name):
    # every query block of the lowest- and highest-density heads and of two
    # random heads, plus 64 random (head, block) rows
    cfg = synth.get_config(name)
    check_full(name, cfg, cfg.p)


def test_attn_480p_all_heads():
    cfg = synth.get_config("480p")
    check_full("480p", cfg, cfg.p, all_heads=True)


@pytest.mark.parametrize("p", [0.8, 0.95])
def test_attn_long_p_sweep_rule(p):
    cfg = synth.get_config("long")
    check_full("long", cfg, p, seed=int(p * 100))


def test_attn_deterministic_and_trace():
    torch = torch_mod()
    fva = lib()
    cfg = synth.get_config("720p")
    geo = geometry_of(cfg)
    Qb, Kb, Vb = workload("720p")
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O1 = run_attn(q, k, v, cfg, mask, counts, kv)
    desc = fva._desc_of(q)
    trace = torch.zeros(fva.fva_trace_words(desc, tiling_of(cfg)), dtype=torch.int64, device="cuda:0")
    O2 = fva.fva_attn(q, k, v, tiling_of(cfg), mask, counts, kv, flags=fva.FVA_TRACE, trace=trace)
    O3 = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    torch.cuda.synchronize()
    assert torch.equal(O1, O2) and torch.equal(O1, O3)
    tr = trace.view(-1, 4).cpu().numpy()
    rows = cfg.heads * geo.nb
    assert tr.shape[0] == rows + 2048  # rows, then chunk records (no row is split here)
    assert np.all(tr[:rows, 1] >= tr[:rows, 0]) and np.all(tr[:rows, 0] > 0)
    assert not tr[rows:].any()
    # engine clock of the run: shader cycles over the 100 MHz clock
    sclk = tr[:rows, 3].sum() * 100.0 / (tr[:rows, 1] - tr[:rows, 0]).sum()
    log(f"[attn] 720p trace: engine clock {sclk:.0f} MHz")
    assert np.all(tr[:rows, 3] > 0) and 500.0 < sclk < 3000.0


def test_attn_max_blocks_sampled():
    # nb = 1024, the largest supported block count; sampled query blocks.
    fva = lib()
    cfg = custom_config("max_blocks", 1, (16, 128, 64), (2, 8, 8), (1.5,), seed=11)
    geo = geometry_of(cfg)
    assert geo.nb == 1024
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O = run_attn(q, k, v, cfg, mask, counts, kv)
    m = mask.cpu().numpy()[0, 0]
    rows = [0, 7, 511, 512, 1000, 1023]
    ref = attn_ref_rows(f64(Qb[0, 0]), f64(Kb[0, 0]), f64(Vb[0, 0]), m, geo, rows)
    Of = O[0, 0].float().cpu().numpy()
    e = np.concatenate([np.abs(Of[geo.block_tokens[i]] - o).ravel() for i, o in ref.items()])
    log(f"[attn] max_blocks: rows {rows}, max abs {e.max():.3e} mean abs {e.mean():.3e}")
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS


def test_attn_batch_two_odd_heads():
    fva = lib()
    cfg = synth.WorkloadConfig("batch2", 3, (5, 13, 21), (2, 8, 8), 0.9, 3, 12, "fixed", (0.7, 2.5, 4.0), batch=2)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O_p = run_attn(q, k, v, cfg, mask, counts, kv)
    O_n = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    O_m = run_attn(q, k, v, cfg, mask)
    torch = torch_mod()
    assert torch.equal(O_p, O_n) and torch.equal(O_p, O_m)
    compare_full("batch2", Qb, Kb, Vb, cfg, mask.cpu().numpy(), o64(O_p))


def test_attn_more_heads_than_plan_lds():
    # 2 x 520 = 1040 (batch, head) pairs, more than the 1024 whose costs,
    # order and queue lengths the plan keeps in LDS: it takes them from the
    # workspace instead. The grid's one-frame last t-row forms query-block
    # pairs. The persistent launch must equal the unpaired one and the naive
    # grid bit for bit (no row is split: nb = 8), and a few heads the oracle.
    fva, torch = lib(), torch_mod()
    heads = 520
    alphas = tuple(float(a) for a in np.random.default_rng(71).uniform(0.3, 5.0, heads))
    cfg = synth.WorkloadConfig("manyheads", heads, (3, 16, 16), (2, 8, 8), 0.9, 2, 71, "fixed", alphas, batch=2)
    assert cfg.batch * cfg.heads > 1024 and geometry_of(cfg).nb == 8
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O_p = run_attn(q, k, v, cfg, mask, counts, kv)
    O_u = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_UNPAIRED)
    O_n = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    assert torch.equal(O_p, O_u) and torch.equal(O_p, O_n)
    sel = [0, 137, 519]
    m = mask.cpu().numpy()
    O = o64(O_p)
    compare_full("1040 heads, 2 x 3 of them", Qb[:, sel], Kb[:, sel], Vb[:, sel], cfg, m[:, sel], O[:, sel])


@pytest.mark.parametrize("s", [1, 2, 3, 5])
@pytest.mark.parametrize("grid,tile", [((3, 16, 16), (1, 8, 8)), ((5, 13, 21), (2, 8, 8))])
def test_attn_split_forced(s, grid, tile):
    # Every row keeping more than s blocks runs as ceil(count / s) chunk items
    # on different workgroups; combine_kernel merges their partial results in
    # chunk order, so the output is deterministic and within the bar.
    torch = torch_mod()
    fva = lib()
    cfg = custom_config("split", 2, grid, tile, (0.5, 3.0), seed=23)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    mask = make_mask("random70", 1, 2, geo.nb, geo, np.random.default_rng(s))
    mask[..., ::4, :] = 0  # some empty rows too
    q, k, v = upload(Qb, Kb, Vb)
    mt = torch.from_numpy(mask).to("cuda:0")
    O1 = run_attn(q, k, v, cfg, mt, flags=fva.FVA_SPLIT_BLOCKS(s))
    O2 = run_attn(q, k, v, cfg, mt, flags=fva.FVA_SPLIT_BLOCKS(s))
    assert torch.equal(O1, O2)
    O_whole = run_attn(q, k, v, cfg, mt)
    d = (O1.float() - O_whole.float()).abs().max().item()
    log(f"[attn] split s={s} grid{grid}: max |split - whole| {d:.3e}")
    compare_full(f"split s={s} grid{grid}", Qb, Kb, Vb, cfg, mask, o64(O1))


def test_attn_split_routed_tiny():
    fva = lib()
    cfg = synth.get_config("tiny")
    Qb, Kb, Vb = workload("tiny")
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    O = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SPLIT_BLOCKS(2))
    compare_full("tiny split s=2", Qb, Kb, Vb, cfg, mask.cpu().numpy(), o64(O))


def test_attn_split_automatic_one_head():
    # One flat head of the 480p shape: 308 query blocks for the 512 workgroup
    # slots, ~250 kept blocks a row. The automatic chunk size
    # max(32, ceil(total / 1024)) splits the long rows; the trace shows chunk
    # items, and sampled rows match the oracle.
    torch = torch_mod()
    fva = lib()
    cfg = custom_config("one_head", 1, (21, 30, 52), (2, 8, 8), (0.5,), seed=24)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = upload(Qb, Kb, Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    c = counts.cpu().numpy()[0, 0]
    total = int((c + 1).sum())
    S = max(32, -(-total // 1024))
    n_chunks = int(sum(-(-x // S) for x in c if x > S))
    assert n_chunks > 0
    desc = fva._desc_of(q)
    trace = torch.zeros(fva.fva_trace_words(desc, tiling_of(cfg)), dtype=torch.int64, device="cuda:0")
    O = fva.fva_attn(q, k, v, tiling_of(cfg), mask, counts, kv, flags=fva.FVA_TRACE, trace=trace)
    torch.cuda.synchronize()
    tr = trace.view(-1, 4).cpu().numpy()
    rows = geo.nb
    split_rows = c > S
    assert np.all(tr[:rows][~split_rows, 0] > 0) and not tr[:rows][split_rows].any()
    assert np.all(tr[rows:rows + n_chunks, 0] > 0) and not tr[rows + n_chunks:].any()
    O_naive = run_attn(q, k, v, cfg, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    log(f"[attn] one head: S={S}, {split_rows.sum()} rows split into {n_chunks} chunks, "
        f"max |split - whole| {(O.float() - O_naive.float()).abs().max().item():.3e}")
    m = mask.cpu().numpy()[0, 0]
    sample = sorted(set([int(i) for i in np.nonzero(split_rows)[0][:12]] + [0, rows - 1]))
    ref = attn_ref_rows(f64(Qb[0, 0]), f64(Kb[0, 0]), f64(Vb[0, 0]), m, geo, sample)
    Of = O[0, 0].float().cpu().numpy()
    e = np.concatenate([np.abs(Of[geo.block_tokens[i]] - o).ravel() for i, o in ref.items()])
    assert e.max() <= ATTN_MAX_ABS and e.mean() <= ATTN_MEAN_ABS
