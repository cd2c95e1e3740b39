"""Query-block pairs of the persistent scheduler.

Two neighbouring query blocks of at most 64 real tokens (x-neighbours, else
y-neighbours) run as one item over the union of their kept lists, each on
two of the four waves, each wave
skipping the key blocks its own block does not keep. Every row therefore
sees exactly its own key blocks in ascending order, as it does alone: the
paired launch must equal, bit for bit, the same launch under
FVA_SCHED_UNPAIRED and the naive grid, on every kind of workload that forms
pairs (one-frame last t-rows, the narrow last column of 480p, partial boxes
on every axis, 64-token boxes, 64-token curve runs, split rows next to
paired ones, E4M3 V). The oracle
parity of the same launches is covered by the other attention tests, which
run the default (paired) path.
"""

import numpy as np
import pytest

import synth

from _gpu_util import custom_config, geometry_of, lib, log, tiling_of, to_dev, torch_mod, workload

pytestmark = pytest.mark.gpu


def pairs_of(geo):
    """(first block, second block) of every pair of one head, by definition:
    x-neighbours (ix even, ix + 1) of one (t, y) line with at most 64 tokens
    each; then, among the blocks no x-pair holds, y-neighbours (iy even,
    iy + 1) of one (t, x) column with at most 64 tokens each."""
    n = geo.block_sizes.reshape(geo.nbt, geo.nby, geo.nbx)
    bid = lambda t, y, x: (t * geo.nby + y) * geo.nbx + x
    out, taken = [], set()
    for t in range(geo.nbt):
        for y in range(geo.nby):
            for x in range(0, geo.nbx - 1, 2):
                if n[t, y, x] <= 64 and n[t, y, x + 1] <= 64:
                    out.append((bid(t, y, x), bid(t, y, x + 1)))
                    taken |= {bid(t, y, x), bid(t, y, x + 1)}
    for t in range(geo.nbt):
        for x in range(geo.nbx):
            for y in range(0, geo.nby - 1, 2):
                a, b = bid(t, y, x), bid(t, y + 1, x)
                if a not in taken and b not in taken and n[t, y, x] <= 64 and n[t, y + 1, x] <= 64:
                    out.append((a, b))
    return sorted(out)


def split_rows(mask_np):
    """Rows the automatic chunk size splits: more kept blocks than
    max(32, ceil(sum over rows of (kept + 1) / 1024))."""
    c = mask_np.reshape(-1, mask_np.shape[-1]).sum(-1)
    S = max(32, -(-int((c + 1).sum()) // 1024))
    return c > S


def same_three_ways(q, k, v, tiling, mask, counts, kv, geo, extra=0):
    """Paired == FVA_SCHED_UNPAIRED everywhere; == the naive grid on the
    rows that are not split (a split row merges chunks in another order)."""
    fva, torch = lib(), torch_mod()
    O = fva.fva_attn(q, k, v, tiling, mask, counts, kv, flags=extra)
    O_u = fva.fva_attn(q, k, v, tiling, mask, counts, kv, flags=extra | fva.FVA_SCHED_UNPAIRED)
    torch.cuda.synchronize()
    assert torch.equal(O, O_u)
    if not extra:
        O_n = fva.fva_attn(q, k, v, tiling, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
        torch.cuda.synchronize()
        split = split_rows(mask.cpu().numpy())
        if not split.any():
            assert torch.equal(O, O_n)
        else:
            a = O.view(torch.int16).cpu().numpy().reshape(-1, O.shape[-2], O.shape[-1])
            b = O_n.view(torch.int16).cpu().numpy().reshape(a.shape)
            for r in np.nonzero(~split)[0]:
                tok = geo.block_tokens[r % geo.nb]
                assert np.array_equal(a[r // geo.nb, tok], b[r // geo.nb, tok]), r
    return O


@pytest.mark.parametrize("name,heads", [("tiny", None), ("720p", [0, 9, 21, 39]), ("480p", [3, 11, 25, 38])])
def test_pairs_equal_unpaired_on_routed_workloads(name, heads):
    fva = lib()
    cfg = synth.get_config(name)
    geo = geometry_of(cfg)
    Qb, Kb, Vb = workload(name)
    if heads is not None:
        Qb, Kb, Vb = Qb[:, heads], Kb[:, heads], Vb[:, heads]
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, tiling_of(cfg))
    pairs = pairs_of(geo)
    assert pairs  # every one of these workloads forms pairs
    c = counts.cpu().numpy().reshape(-1, geo.nb)
    m = mask.cpu().numpy().reshape(-1, geo.nb, geo.nb)
    both = sum(int((m[h, a] & m[h, b]).sum()) for h in range(m.shape[0]) for a, b in pairs)
    union = sum(int((m[h, a] | m[h, b]).sum()) for h in range(m.shape[0]) for a, b in pairs)
    log(f"[pairs] {name}: {len(pairs)} pairs per head, union/shared kept blocks {union}/{both}, "
        f"mean count {c.mean():.1f}")
    same_three_ways(q, k, v, tiling_of(cfg), mask, counts, kv, geo)
    same_three_ways(q, k, v, tiling_of(cfg), mask, None, None, geo)  # lists rebuilt from the mask


@pytest.mark.parametrize("s", [2, 5])
def test_pairs_next_to_split_rows(s):
    # Partial boxes on all three axes (5 = 2*2 + 1 frames, 13 = 8 + 5 rows,
    # 21 = 2*8 + 5 columns): the one-frame t-row forms the x-pairs (12, 13)
    # and (15, 16) and the y-pair (14, 17) of its narrow last column. Random
    # masks elsewhere; in every head row 13 keeps s + 2 blocks (split into
    # chunks, so its pair is not formed) and rows 15 and 16 keep at most s
    # blocks, one shared and one of their own each (paired).
    fva, torch = lib(), torch_mod()
    cfg = custom_config("pairsplit", 3, (5, 13, 21), (2, 8, 8), (0.3, 1.5, 5.0), seed=41)
    geo = geometry_of(cfg)
    assert pairs_of(geo) == [(12, 13), (14, 17), (15, 16)]
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    rng = np.random.default_rng(43 + s)
    m = (rng.random((1, 3, geo.nb, geo.nb)) < 0.25).astype(np.uint8)
    m[0, :, ::4, :] = 0
    m[0, :, 12:17, :] = 0
    m[0, :, 12, 0] = 1
    m[0, :, 13, :s + 2] = 1
    m[0, :, 15, [1, 3]] = 1
    m[0, :, 16, [3, 4]] = 1
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    mt = torch.from_numpy(m).to("cuda:0")
    same_three_ways(q, k, v, tiling_of(cfg), mt, None, None, geo, extra=fva.FVA_SPLIT_BLOCKS(s))
    O = same_three_ways(q, k, v, tiling_of(cfg), mt, None, None, geo)
    O_split = fva.fva_attn(q, k, v, tiling_of(cfg), mt, flags=fva.FVA_SPLIT_BLOCKS(s))
    torch.cuda.synchronize()
    # rows cut into chunks merge them in another rounding order; whole rows
    # (paired or not) are the same bit for bit
    a = O.view(torch.int16).cpu().numpy()
    b = O_split.view(torch.int16).cpu().numpy()
    counts = m.sum(-1)
    for h in range(3):
        for i in range(geo.nb):
            if counts[0, h, i] <= s:
                tok = geo.block_tokens[i]
                assert np.array_equal(a[0, h, tok], b[0, h, tok]), (h, i)


def test_pairs_64_token_curve_runs():
    # one-dimensional blocks of 64 consecutive tokens (the curve layout's
    # tiling): every block but a short last one pairs with its neighbour
    fva = lib()
    cfg = custom_config("run64", 2, (1, 1, 20000), (1, 1, 64), (0.5, 3.0), seed=47)
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    q, k, v = to_dev(Qb), to_dev(Kb), to_dev(Vb)
    t = fva.Tiling(1, 1, 20000, 1, 1, 64)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, t)
    same_three_ways(q, k, v, t, mask, counts, kv, geometry_of(cfg))


def test_pairs_fp8_v():
    fva, torch = lib(), torch_mod()
    cfg = synth.get_config("720p")
    heads = [2, 17, 30]
    Qb, Kb, Vb = workload("720p")
    q, k, v = to_dev(Qb[:, heads]), to_dev(Kb[:, heads]), to_dev(Vb[:, heads])
    t = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, t)
    v8, vexp = fva.fva_quantize_v(v, t)
    O = fva.fva_attn_fp8v(q, k, v8, vexp, t, mask, counts, kv)
    O_u = fva.fva_attn_fp8v(q, k, v8, vexp, t, mask, counts, kv, flags=fva.FVA_SCHED_UNPAIRED)
    O_n = fva.fva_attn_fp8v(q, k, v8, vexp, t, mask, counts, kv, flags=fva.FVA_SCHED_NAIVE)
    torch.cuda.synchronize()
    assert torch.equal(O, O_u) and torch.equal(O, O_n)


def test_pair_trace_records_split_the_item():
    fva, torch = lib(), torch_mod()
    cfg = synth.get_config("720p")
    geo = geometry_of(cfg)
    heads = [5, 12, 33, 38]
    Qb, Kb, Vb = workload("720p")
    q, k, v = to_dev(Qb[:, heads]), to_dev(Kb[:, heads]), to_dev(Vb[:, heads])
    t = tiling_of(cfg)
    mask, counts, kv = fva.fva_route(q, k, cfg.p, cfg.k_min, t)
    desc = fva._desc_of(q)
    trace = torch.zeros(fva.fva_trace_words(desc, t), dtype=torch.int64, device="cuda:0")
    fva.fva_attn(q, k, v, t, mask, counts, kv, flags=fva.FVA_TRACE, trace=trace)
    torch.cuda.synchronize()
    tr = trace.view(-1, 4).cpu().numpy()
    c = counts.cpu().numpy().reshape(-1)
    rows = c.size
    # the automatic chunk size; rows keeping more are split (no row record)
    S = max(32, -(-int((c + 1).sum()) // 1024))
    whole = c <= S
    assert np.all(tr[:rows][whole, 0] > 0) and np.all(tr[:rows][whole, 3] > 0)
    assert np.all(tr[:rows, 1] >= tr[:rows, 0]) and not tr[:rows][~whole].any()
    formed = 0
    for h in range(len(heads)):
        for a, b in pairs_of(geo):
            ra, rb = h * geo.nb + a, h * geo.nb + b
            if whole[ra] and whole[rb]:
                # one item: the same workgroup, the first record ends where the second starts
                assert tr[ra, 1] == tr[rb, 0] and tr[ra, 2] == tr[rb, 2], (h, a)
                formed += 1
    log(f"[pairs] 720p trace: S = {S}, {formed} pairs formed, {int((~whole).sum())} rows split")
    assert formed > 0
