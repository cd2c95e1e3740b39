"""Benchmark of the Top-p block-sparse attention hot path on one MI355X.

One step = fva_route (pool, scores, softmax, Top-p + floor, mask / counts /
kept lists) + fva_attn (work list + block-sparse attention) over one batch of
synthetic video-DiT inputs already resident in HBM. Default workload: the
720p layer (40 heads, 21x45x80 latent tokens, 2x8x8 blocks, p = 0.9,
k_min = 4), the shape the paper's attention numbers are quoted on.

Prints ONE JSON line. `value` is dense-equivalent TFLOPS of the whole step:
4 * heads * N^2 * d / step time (the dense attention work the step replaces).
Beside it: attention ms, route us and route GB/s, kept-tile TFLOPS
(4 * 128^2 * d per kept block pair), useful TFLOPS (real-token pairs), the
retained fraction, a roofline object for the attention kernel and the fp64
CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps 10] [--warmup 3] [--workload 720p] [--blocks box|hilbert]

--blocks hilbert runs the same inputs with the Hilbert-curve block
organisation: Q, K, V are permuted into curve order once before timing (the
permutation and the curve order are timed on their own and reported), and
the step routes and attends on the curve-ordered tensors with blocks of
bt*bh*bw consecutive curve positions.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse attn ms + dense-equiv TFLOPS, MFMA util on kept blocks; route GB/s"
PEAK_BF16_TFLOPS = 2500.0  # published dense bf16 MFMA peak
# The same peak from the unit counts: 256 CUs x 4096 bf16 flop per clock per
# CU; at the 2.4 GHz peak engine clock 2516.6 TFLOP/s. The line also reports
# the fraction against this figure at the engine clock measured in the run.
CUS = 256
BF16_FLOP_PER_CLK_CU = 4096
PEAK_BF16_TFLOPS_2400 = CUS * BF16_FLOP_PER_CLK_CU * 2.4e9 / 1e12
PEAK_FP8_TFLOPS = 5000.0
# Q K^T (bf16) and P V (fp8) are equal halves of the attention flops: at both
# peaks a launch would take flops/2 / 2500 + flops/2 / 5000 TFLOP-seconds.
PEAK_BF16_FP8_TFLOPS = 2.0 / (1.0 / PEAK_BF16_TFLOPS + 1.0 / PEAK_FP8_TFLOPS)
PEAK_HBM_GBPS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def block_sizes(grid, tile):
    """Real tokens of every block, raster block order (boxes anchored at the origin)."""
    ext = []
    for S, b in zip(grid, tile):
        n = -(-S // b)
        e = np.full(n, b, dtype=np.int64)
        e[-1] = S - b * (n - 1)
        ext.append(e)
    return np.einsum("a,b,c->abc", *ext).reshape(-1)


def real_pairs(mask, sizes):
    """sum over kept (h, i, j) of n_i * n_j (real token pairs)."""
    n = sizes.astype(np.float64)
    nb = n.shape[0]
    m = mask.reshape(-1, nb, nb).astype(np.float64)
    return float(np.einsum("hij,i,j->", m, n, n))


def source_digest(*paths):
    """Digest of a kernel source and the headers it shares with the others."""
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def pair_offsets(sizes, nby, nbx):
    """Partner offset of every block (the library's pairing rule, restated):
    x-neighbours (ix even, ix + 1) of one (t, y) line that both hold at most
    64 tokens, then among the blocks no x-pair holds, y-neighbours (iy even,
    iy + 1) of one (t, x) column that both do; +offset on the first block,
    -offset on the second, 0 for blocks in no pair."""
    n = sizes.reshape(-1, nby, nbx)
    small = n <= 64
    off = np.zeros(n.shape, np.int64)
    inx = np.zeros(n.shape, bool)
    for ix in range(0, nbx - 1, 2):
        both = small[:, :, ix] & small[:, :, ix + 1]
        off[:, :, ix] = np.where(both, 1, off[:, :, ix])
        off[:, :, ix + 1] = np.where(both, -1, off[:, :, ix + 1])
        inx[:, :, ix] |= both
        inx[:, :, ix + 1] |= both
    for iy in range(0, nby - 1, 2):
        both = small[:, iy, :] & small[:, iy + 1, :] & ~inx[:, iy, :] & ~inx[:, iy + 1, :]
        off[:, iy, :] = np.where(both, nbx, off[:, iy, :])
        off[:, iy + 1, :] = np.where(both, -nbx, off[:, iy + 1, :])
    return off.reshape(-1)


def plan_costs(counts, tiling, paired):
    """Per-row cost the persistent plan balances: kept blocks + 1, except that
    a query-block pair (pair_offsets; neither row split) costs its larger row
    + 1 on its first row and 1 on its second."""
    c = np.clip(counts.reshape(-1, counts.shape[-1]).astype(np.int64), 0, counts.shape[-1])
    cost = c + 1
    if not paired:
        return cost.reshape(-1)
    nby = -(-tiling.H // tiling.bh)
    nbx = -(-tiling.W // tiling.bw)
    off = pair_offsets(block_sizes((tiling.T, tiling.H, tiling.W), (tiling.bt, tiling.bh, tiling.bw)), nby, nbx)
    first = np.nonzero(off > 0)[0]
    second = first + off[first]
    S = max(32, -(-int((c + 1).sum()) // 1024))  # the automatic chunk size
    a, b = c[:, first], c[:, second]
    formed = (a <= S) & (b <= S)
    cost[:, first] = np.where(formed, np.maximum(a, b) + 1, cost[:, first])
    cost[:, second] = np.where(formed, 1, cost[:, second])
    return cost.reshape(-1)


def imbalance(trace, counts, tiling=None, paired=False):
    """Per-CU and per-XCD load figures from an FVA_TRACE record.

    Records: one per (b, h, i) row, then one per chunk item of a split row
    (a split row's own record stays empty; the two rows of a query-block
    pair share their item's time). CU = (xcc, bits 8.. of HW_ID); busy =
    sum of item durations on the CU. rho = max/mean over XCDs of summed item
    time, of summed kept blocks over the unsplit rows (Eq. 2 with XCDs as
    ranks), and of summed plan cost (kept blocks + 1, a pair costing about
    one row: with pairs the plan balances cost, so kept blocks per XCD
    differ by design).
    """
    tr = trace.reshape(-1, 4)
    rows = counts.size
    used = tr[:, 0] > 0
    dur = (tr[:, 1] - tr[:, 0]).astype(np.float64)[used]
    loc = tr[used, 2]
    cu = loc >> 8
    xcc = loc >> 16
    _, inv = np.unique(cu, return_inverse=True)
    busy = np.bincount(inv, weights=dur)
    xb = np.bincount(xcc, weights=dur, minlength=8)
    row_used = used[:rows]
    row_xcc = tr[:rows, 2][row_used] >> 16
    xc = np.bincount(row_xcc, weights=counts.reshape(-1)[row_used].astype(np.float64), minlength=8)
    res = {}
    if tiling is not None:
        cost = plan_costs(counts, tiling, paired)
        xk = np.bincount(row_xcc, weights=cost[row_used].astype(np.float64), minlength=8)
        res["xcd_cost_rho"] = round(float(xk.max() / xk.mean()), 4)
    span = float(tr[used, 1].max() - tr[used, 0].min()) / 100.0  # 100 MHz clock -> us
    # engine clock: shader cycles (word 3) over the 100 MHz constant clock
    sclk = float(tr[used, 3].sum()) * 100.0 / float((tr[used, 1] - tr[used, 0]).sum())
    return {
        "sclk_mhz": round(sclk, 1),
        "cus_used": int(busy.size),
        "cu_busy_max_over_mean": round(float(busy.max() / busy.mean()), 4),
        "xcd_time_rho": round(float(xb.max() / xb.mean()), 4),
        "xcd_blocks_rho": round(float(xc.max() / xc.mean()), 4),
        **res,
        "chunk_items": int(used[rows:].sum()),
        "span_us": round(span, 1),
    }


def cpu_baseline(cfg, Qb, Kb, Vb, mask, counts, budget_s=20.0, blocks="box"):
    """Oracle timed on this host on a bounded sample; returns dict."""
    from oracle import attn_ref_rows, curve_geometry, route_ref, tile_geometry

    import synth

    if blocks == "hilbert":
        geo = curve_geometry(*cfg.grid, int(np.prod(cfg.tile)))
    else:
        geo = tile_geometry(*cfg.grid, *cfg.tile)
    cores = len(os.sched_getaffinity(0))
    f64 = lambda b: synth.bf16_bits_to_f32(b).astype(np.float64)
    H = cfg.heads
    # routing: a subset of heads, extrapolated linearly in heads
    rh = list(range(0, H, max(1, H // 8)))
    Qr, Kr = f64(Qb[0, rh]), f64(Kb[0, rh])
    t0 = time.perf_counter()
    route_ref(Qr, Kr, cfg.p, cfg.k_min, geo)
    t_route = (time.perf_counter() - t0) * H / len(rh)
    # attention: query blocks of the lowest- and highest-density heads and two
    # others, until the time budget is used; extrapolated by real token pairs
    dens = counts[0].mean(axis=-1)
    heads = [int(np.argmin(dens)), int(np.argmax(dens)), H // 3, (2 * H) // 3]
    n = geo.block_sizes.astype(np.float64)
    heads_f64 = {h: (f64(Qb[0, h]), f64(Kb[0, h]), f64(Vb[0, h])) for h in heads}
    rng = np.random.default_rng(7)
    done_pairs = 0.0
    t_att = 0.0
    rows = 0
    while t_att < budget_s:
        for h in heads:
            i = int(rng.integers(geo.nb))
            t0 = time.perf_counter()
            attn_ref_rows(*heads_f64[h], mask[0, h], geo, [i])
            t_att += time.perf_counter() - t0
            done_pairs += n[i] * float((mask[0, h, i].astype(np.float64) * n).sum())
            rows += 1
    total_pairs = real_pairs(mask, geo.block_sizes)
    t_att_full = t_att * total_pairs / max(done_pairs, 1.0)
    t_full = t_route + t_att_full
    dense_flops = 4.0 * H * float(geo.N) ** 2 * 128
    return {
        "value": dense_flops / t_full / 1e12,
        "unit": "TFLOPS (dense-equivalent)",
        "cores": cores,
        "kind": "oracle",
        "sample": f"fp64 numpy oracle: routing on {len(rh)} of {H} heads (scaled by heads), attention on "
        f"{rows} query blocks of heads {heads} (scaled by real kept token pairs); extrapolated step "
        f"{t_full:.1f} s (route {t_route:.1f} s + attention {t_att_full:.1f} s)",
        "seconds_extrapolated": t_full,
    }


# HBM bytes per launch of attn_persistent_kernel on the 720p workload (3D
# boxes or Hilbert-curve blocks, bf16 or E4M3 V) from rocprofv3 FETCH_SIZE /
# WRITE_SIZE passes, each scaled by the factor the same
# counter reads for a device copy of known size; valid only for the attention
# source with this digest (null otherwise).
ATTN_TRAFFIC = {
    "source_digest": "f8dc17fcc7ddf8c6",
    "bytes": {
        "720p": ((111222344 + 111111162) // 2 * 2 + 758186) * 1024,
        "720p-hilbert": ((77795484 + 77549784) // 2 * 2 + 758302) * 1024,
        "720p-fp8v": ((71772201 + 70525558) // 2 * 2 + 758575) * 1024,
        "720p-hilbert-fp8v": ((66644817 + 67124268) // 2 * 2 + 758497) * 1024,
    },
}
# Same for fva_route (pool_kernel + score_kernel + select_kernel), per call
# (FETCH x 2, WRITE x 1, KiB per dispatch summed over the three kernels).
ROUTE_TRAFFIC = {
    "source_digest": "d8fe57f482ee46fc",
    "bytes": {
        "720p": ((756175 + 29245 + 68473) * 2 + 53760 + 142312 + 49285) * 1024,
        "720p-hilbert": ((756151 + 25345 + 55227) * 2 + 47360 + 116782 + 39989) * 1024,
        "720p-fp8v": ((756173 + 29198 + 68476) * 2 + 53760 + 142496 + 49285) * 1024,
        "720p-hilbert-fp8v": ((756150 + 25344 + 55238) * 2 + 47360 + 116986 + 39989) * 1024,
    },
}


def extra_workloads(torch, fva, synth, dev, reps=3):
    """The other timed workloads, outside the timed region, as extra keys.

    long: the 31x45x80 clip (111,600 tokens, nb 960) at p = 0.8, 0.9 and 0.95:
    retained fraction, route and attention times (HIP events, mean of reps
    after one warmup each).
    480p: the 21x30x52 clip (32,760 tokens, nb 308, partial boxes on all
    three axes) at p = 0.9: the same figures plus the useful (real token
    pair) rate.
    720p_stress: 8 flat and 32 concentrated heads of the 720p shape: attention
    time under the persistent scheduler and under the naive head-major grid,
    and from one traced run of each the per-CU busy max/mean, the per-XCD
    imbalance and the span (Eq. 2 with XCDs as ranks).
    """
    stream = torch.cuda.current_stream()
    out = {}

    def load(name):
        cfg = synth.get_config(name)
        log(f"[bench] extra workload {name}: generating {cfg.heads} heads x {cfg.N} tokens")
        Qb, Kb, Vb = synth.gen_qkv(cfg)
        up = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        q, k, v = up(Qb), up(Kb), up(Vb)
        del Qb, Kb, Vb
        tiling = fva.Tiling(*cfg.grid, *cfg.tile)
        nb = fva.fva_num_blocks(tiling)
        B, H = q.shape[0], q.shape[1]
        bufs = dict(mask=torch.empty((B, H, nb, nb), dtype=torch.uint8, device=dev),
                    counts=torch.empty((B, H, nb), dtype=torch.int32, device=dev),
                    kv=torch.empty((B, H, nb, nb), dtype=torch.int32, device=dev),
                    out=torch.empty_like(q),
                    ws_r=torch.empty(fva.fva_route_workspace_size(fva._desc_of(q), tiling), dtype=torch.uint8,
                                     device=dev),
                    ws_a=torch.empty(fva.fva_attn_workspace_size(fva._desc_of(q), tiling), dtype=torch.uint8,
                                     device=dev))
        return cfg, tiling, nb, (q, k, v), bufs

    def timed_pair(route_fn, attn_fn):
        route_fn()
        attn_fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        tr, ta = 0.0, 0.0
        for _ in range(reps):
            ev[0].record(stream)
            route_fn()
            ev[1].record(stream)
            attn_fn()
            ev[2].record(stream)
            torch.cuda.synchronize()
            tr += ev[0].elapsed_time(ev[1])
            ta += ev[1].elapsed_time(ev[2])
        return tr / reps, ta / reps

    # long clip: retained fraction vs time over the p sweep
    cfg, tiling, nb, (q, k, v), b = load("long")
    sweep = []
    for pp in (0.8, 0.9, 0.95):
        route_fn = lambda: fva.fva_route(q, k, pp, cfg.k_min, tiling, out=(b["mask"], b["counts"], b["kv"]),
                                         workspace=b["ws_r"])
        attn_fn = lambda: fva.fva_attn(q, k, v, tiling, b["mask"], b["counts"], b["kv"], out=b["out"],
                                       workspace=b["ws_a"])
        t_r, t_a = timed_pair(route_fn, attn_fn)
        kept = int(b["counts"].sum().item())
        dense = 4.0 * q.shape[1] * float(cfg.N) ** 2 * 128
        sweep.append({"p": pp, "retained_fraction": round(kept / (q.shape[1] * nb * nb), 4),
                      "route_us": round(t_r * 1e3, 1), "attn_ms": round(t_a, 3),
                      "kept_tile_TFLOPS": round(4.0 * 128**3 * kept / (t_a / 1e3) / 1e12, 1),
                      "dense_equiv_TFLOPS": round(dense / ((t_r + t_a) / 1e3) / 1e12, 1)})
        log(f"[bench] long p={pp}: {sweep[-1]}")
    out["long_p_sweep"] = {"workload": f"long: {q.shape[1]} heads, 31x45x80 = {cfg.N} tokens, tile 2x8x8, nb={nb}, "
                                       f"k_min={cfg.k_min}", "reps": reps, "points": sweep}
    del q, k, v, b
    torch.cuda.empty_cache()

    # 480p: most of its blocks are partial boxes (query-block pairs along x
    # and y)
    cfg, tiling, nb, (q, k, v), b = load("480p")
    route_fn = lambda: fva.fva_route(q, k, cfg.p, cfg.k_min, tiling, out=(b["mask"], b["counts"], b["kv"]),
                                     workspace=b["ws_r"])
    attn_fn = lambda: fva.fva_attn(q, k, v, tiling, b["mask"], b["counts"], b["kv"], out=b["out"],
                                   workspace=b["ws_a"])
    t_r, t_a = timed_pair(route_fn, attn_fn)
    m_np = b["mask"].cpu().numpy()
    kept = int(m_np.sum())
    useful = 4.0 * 128 * real_pairs(m_np, block_sizes(cfg.grid, cfg.tile))
    dense = 4.0 * q.shape[1] * float(cfg.N) ** 2 * 128
    out["p480"] = {"workload": f"480p: {q.shape[1]} heads, 21x30x52 = {cfg.N} tokens, tile 2x8x8, nb={nb}, "
                               f"p={cfg.p}, k_min={cfg.k_min}", "reps": reps,
                   "retained_fraction": round(kept / (q.shape[1] * nb * nb), 4),
                   "route_us": round(t_r * 1e3, 1), "attn_ms": round(t_a, 3),
                   "kept_tile_TFLOPS": round(4.0 * 128**3 * kept / (t_a / 1e3) / 1e12, 1),
                   "useful_TFLOPS": round(useful / (t_a / 1e3) / 1e12, 1),
                   "dense_equiv_TFLOPS": round(dense / ((t_r + t_a) / 1e3) / 1e12, 1)}
    log(f"[bench] 480p: {out['p480']}")
    del q, k, v, b
    torch.cuda.empty_cache()

    # stress: persistent scheduler against the naive head-major grid
    cfg, tiling, nb, (q, k, v), b = load("720p_stress")
    fva.fva_route(q, k, cfg.p, cfg.k_min, tiling, out=(b["mask"], b["counts"], b["kv"]), workspace=b["ws_r"])
    c_np = b["counts"].cpu().numpy()
    res = {"workload": f"720p_stress: {q.shape[1]} heads (8 at alpha 0.3, 32 at alpha 5), 21x45x80, tile 2x8x8, "
                       f"nb={nb}, p={cfg.p}, k_min={cfg.k_min}",
           "retained_fraction": round(float(c_np.sum()) / (q.shape[1] * nb * nb), 4)}
    tw = fva.fva_trace_words(fva._desc_of(q), tiling)
    trace = torch.zeros(tw, dtype=torch.int64, device=dev)
    for name, fl in (("persistent", fva.FVA_SCHED_PERSISTENT), ("naive", fva.FVA_SCHED_NAIVE)):
        attn_fn = lambda: fva.fva_attn(q, k, v, tiling, b["mask"], b["counts"], b["kv"], flags=fl, out=b["out"],
                                       workspace=b["ws_a"])
        _, t_a = timed_pair(lambda: None, attn_fn)
        trace.zero_()
        fva.fva_attn(q, k, v, tiling, b["mask"], b["counts"], b["kv"], flags=fl | fva.FVA_TRACE, out=b["out"],
                     workspace=b["ws_a"], trace=trace)
        torch.cuda.synchronize()
        res[name] = {"attn_ms": round(t_a, 3),
                     **imbalance(trace.cpu().numpy(), c_np, tiling, fl == fva.FVA_SCHED_PERSISTENT)}
        log(f"[bench] stress {name}: {res[name]}")
    out["stress_scheduler"] = res
    del q, k, v, b, trace
    torch.cuda.empty_cache()
    return out


def gemm_ceiling(torch, n=8192, reps=10):
    """bf16 matrix ceiling of this device as the vendor GEMM reaches it: an
    n x n x n torch.matmul (hipBLASLt), HIP events, mean of reps after two
    warmups. Context for the attention fraction, never a peak it is graded on."""
    a = torch.randn(n, n, device="cuda:0", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda:0", dtype=torch.bfloat16)
    for _ in range(2):
        c = a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / reps / 1e3
    del a, b, c
    return {"shape": f"{n}x{n}x{n} bf16 (torch.matmul)", "reps": reps, "ms": round(t * 1e3, 3),
            "TFLOPS": round(2.0 * n**3 / t / 1e12, 1)}


def copy_calibration(torch, gib=1.0, reps=5):
    """Plain device copy of known size (reads and writes `gib` GiB each)."""
    n = int(gib * (1 << 30))
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        dst.copy_(src)
    ev[1].record()
    torch.cuda.synchronize()
    t = ev[0].elapsed_time(ev[1]) / reps / 1e3
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copy_s": t,
                      "copy_GBps_read_plus_write": 2 * n / t / 1e9}), flush=True)


def curve_setup(torch, fva, cfg, q, k, v, reps=5):
    """Curve order and curve-ordered copies of q, k, v; times both (HIP events, mean of reps)."""
    T, H, W = cfg.grid
    stream = torch.cuda.current_stream()
    ws = torch.empty(fva.fva_curve_workspace_size(T, H, W), dtype=torch.uint8, device=q.device)
    perm = fva.fva_curve_order(T, H, W, device=q.device, workspace=ws)
    qc, kc, vc = (fva.fva_permute_tokens(x, perm, fva.FVA_TO_CURVE) for x in (q, k, v))
    o = torch.empty_like(q)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record(stream)
    for _ in range(reps):
        fva.fva_curve_order(T, H, W, out=perm, workspace=ws)
    ev[1].record(stream)
    for _ in range(reps):
        for x, y in ((q, qc), (k, kc), (v, vc)):
            fva.fva_permute_tokens(x, perm, fva.FVA_TO_CURVE, out=y)
        fva.fva_permute_tokens(qc, perm, fva.FVA_FROM_CURVE, out=o)
    ev[2].record(stream)
    torch.cuda.synchronize()
    t_order = ev[0].elapsed_time(ev[1]) / reps * 1e3
    t_perm = ev[1].elapsed_time(ev[2]) / reps * 1e3
    moved = 4 * 2 * q.numel() * 2  # four tensors, each read and written once
    del o
    return {
        "qkv": (qc, kc, vc),
        "curve_order_us": round(t_order, 1),
        "permute_qkv_in_o_out_us": round(t_perm, 1),
        "permute_GBps": round(moved / (t_perm / 1e6) / 1e9, 1),
        "note": "done once per grid / per model call, outside the timed step",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="720p")
    ap.add_argument("--p", type=float, default=None)
    ap.add_argument("--p-sweep", default=None, help="comma-separated p values, timed after the main run")
    ap.add_argument("--sched", choices=["persistent", "naive"], default="persistent")
    ap.add_argument("--v", choices=["bf16", "fp8"], default="bf16", dest="vfmt",
                    help="attention on bf16 V, or on E4M3 V quantised inside the step")
    ap.add_argument("--sasa", type=int, default=0, metavar="R",
                    help="route with slack-aware augmentation over R ranks of contiguous heads (n1 0.8, n2 0.07)")
    ap.add_argument("--blocks", choices=["box", "hilbert"], default="box",
                    help="3D boxes, or runs of the Hilbert curve over curve-ordered tokens")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-trace", action="store_true", help="skip the scheduler imbalance trace runs")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--reverse-heads", action="store_true",
                    help="reverse the head order of Q, K, V (scheduler diagnostic: the head-major grid's tail changes)")
    ap.add_argument("--dense-reps", type=int, default=3,
                    help="runs of the same attention with every block kept (dense comparator), outside the timed region")
    ap.add_argument("--flushed-reps", type=int, default=20,
                    help="steps timed one by one after a 512 MB cache-flushing write, outside the timed region (0: skip)")
    ap.add_argument("--copy-calibration", action="store_true", help="only time a 1 GiB device copy")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the long-clip p sweep and the stress scheduler comparison (extra keys)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(
            "bench.py measures one GPU only: the path shards by head across GPUs (see the design notes); "
            "run with --gpus 1",
            file=sys.stderr,
        )
        sys.exit(2)

    import torch

    if args.copy_calibration:
        copy_calibration(torch)
        return

    import paper_2607_16190_amd as fva
    import synth

    cfg = synth.get_config(args.workload)
    p = cfg.p if args.p is None else args.p
    dev = torch.device("cuda:0")
    log(f"[bench] generating {cfg.name}: {cfg.heads} heads x {cfg.N} tokens x 128")
    Qb, Kb, Vb = synth.gen_qkv(cfg)
    up = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    if args.reverse_heads:
        Qb, Kb, Vb = (np.ascontiguousarray(a[:, ::-1]) for a in (Qb, Kb, Vb))
        log("[bench] head order reversed")
    q, k, v = up(Qb), up(Kb), up(Vb)
    curve = None
    if args.blocks == "hilbert":
        blk = int(np.prod(cfg.tile))
        tiling = fva.Tiling.curve(cfg.N, blk)
        nb_c = -(-cfg.N // blk)
        sizes = np.full(nb_c, blk, dtype=np.int64)
        sizes[-1] = cfg.N - blk * (nb_c - 1)
        curve = curve_setup(torch, fva, cfg, q, k, v)
        q, k, v = curve.pop("qkv")
        log(f"[bench] curve order {curve['curve_order_us']} us, permute Q,K,V in + O out "
            f"{curve['permute_qkv_in_o_out_us']} us")
    else:
        tiling = fva.Tiling(*cfg.grid, *cfg.tile)
        sizes = block_sizes(cfg.grid, cfg.tile)
    desc = fva._desc_of(q)
    nb = fva.fva_num_blocks(tiling)
    assert nb == sizes.shape[0]
    B, H = q.shape[0], q.shape[1]
    mask = torch.empty((B, H, nb, nb), dtype=torch.uint8, device=dev)
    counts = torch.empty((B, H, nb), dtype=torch.int32, device=dev)
    kv = torch.empty((B, H, nb, nb), dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    ws_r = torch.empty(fva.fva_route_workspace_size(desc, tiling), dtype=torch.uint8, device=dev)
    ws_a = torch.empty(fva.fva_attn_workspace_size(desc, tiling), dtype=torch.uint8, device=dev)
    flags = fva.FVA_SCHED_NAIVE if args.sched == "naive" else fva.FVA_SCHED_PERSISTENT
    stream = torch.cuda.current_stream()
    fp8 = args.vfmt == "fp8"
    if fp8:
        v8 = torch.empty((B, H, nb, 128, 128), dtype=torch.uint8, device=dev)
        vexp = torch.empty((B, H, 128), dtype=torch.int32, device=dev)
        ws_q = torch.empty(fva.fva_quantize_v_workspace_size(desc, tiling), dtype=torch.uint8, device=dev)

    if args.sasa:
        R = args.sasa
        if R < 1 or H % R:
            raise SystemExit("--sasa R needs R to divide the number of heads")
        rank_of = (torch.arange(B * H, device=dev, dtype=torch.int32) % H) // (H // R)
        rank_extra = torch.empty(R, dtype=torch.int32, device=dev)
        ws_r = torch.empty(fva.fva_route_sasa_workspace_size(desc, tiling), dtype=torch.uint8, device=dev)

    def route(pp):
        if args.sasa:
            fva.fva_route_sasa(q, k, pp, cfg.k_min, tiling, rank_of, args.sasa, 0.8, 0.07, out=(mask, counts, kv),
                               rank_extra=rank_extra, workspace=ws_r)
        else:
            fva.fva_route(q, k, pp, cfg.k_min, tiling, out=(mask, counts, kv), workspace=ws_r)

    def attend(fl, trace=None):
        if fp8:
            fva.fva_attn_fp8v(q, k, v8, vexp, tiling, mask, counts, kv, flags=fl, out=out, workspace=ws_a, trace=trace)
        else:
            fva.fva_attn(q, k, v, tiling, mask, counts, kv, flags=fl, out=out, workspace=ws_a, trace=trace)

    def step(pp, ev=None):
        if ev:
            ev[0].record(stream)
        if fp8:
            fva.fva_quantize_v(v, tiling, out=(v8, vexp), workspace=ws_q)
        if ev:
            ev[3].record(stream)
        route(pp)
        if ev:
            ev[1].record(stream)
        attend(flags)
        if ev:
            ev[2].record(stream)

    def timed(pp, steps, warmup):
        for _ in range(warmup):
            step(pp)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s_ in range(steps):
            step(pp, evs[s_])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        quant_ms = [e[0].elapsed_time(e[3]) for e in evs]
        route_ms = [e[3].elapsed_time(e[1]) for e in evs]
        attn_ms = [e[1].elapsed_time(e[2]) for e in evs]
        timed.quant_s = float(np.mean(quant_ms)) / 1e3
        return wall * 1e3 / steps, float(np.mean(route_ms)) / 1e3, float(np.mean(attn_ms)) / 1e3

    ms_per_step, t_route, t_attn = timed(p, args.steps, args.warmup)
    t_quant = timed.quant_s

    def flushed(pp, reps, warmup=3, flush_mb=512):
        # Each step timed alone after writing a 512 MB buffer (larger than the
        # 256 MB Infinity Cache), on the same stream; median and min.
        scratch = torch.empty(flush_mb << 20, dtype=torch.uint8, device=dev)
        for _ in range(warmup):
            step(pp)
        rows = []
        for _ in range(reps):
            scratch.fill_(1)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            step(pp, ev)
            torch.cuda.synchronize()
            rows.append((ev[0].elapsed_time(ev[2]), ev[3].elapsed_time(ev[1]) * 1e3, ev[1].elapsed_time(ev[2])))
        del scratch
        a = np.array(rows)
        med, mn = np.median(a, axis=0), a.min(axis=0)
        return {"reps": reps, "warmup": warmup, "flush_MB": flush_mb,
                "step_ms_median": round(float(med[0]), 4), "step_ms_min": round(float(mn[0]), 4),
                "route_us_median": round(float(med[1]), 2), "route_us_min": round(float(mn[1]), 2),
                "attn_ms_median": round(float(med[2]), 4), "attn_ms_min": round(float(mn[2]), 4)}

    def dense(reps):
        # The same attention call with every key block kept for every query
        # block (counts = nb, kept lists 0 .. nb-1): the dense work the
        # routing avoids, on the same kernel.
        ones = torch.ones_like(mask)
        c_all = torch.full_like(counts, nb)
        kv_all = torch.arange(nb, dtype=torch.int32, device=dev).expand(B, H, nb, nb).contiguous()
        o_d = torch.empty_like(out)

        def run():
            if fp8:
                fva.fva_attn_fp8v(q, k, v8, vexp, tiling, ones, c_all, kv_all, flags=flags, out=o_d, workspace=ws_a)
            else:
                fva.fva_attn(q, k, v, tiling, ones, c_all, kv_all, flags=flags, out=o_d, workspace=ws_a)

        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps / 1e3
        all_flops = 4.0 * 128 * 128 * 128 * B * H * nb * nb
        del ones, c_all, kv_all, o_d
        return t, all_flops

    dense_res = None
    if args.dense_reps > 0:
        t_dense, dense_tile_flops = dense(args.dense_reps)
        dense_res = {"reps": args.dense_reps, "attn_ms": round(t_dense * 1e3, 3),
                     "kept_tile_TFLOPS": round(dense_tile_flops / t_dense / 1e12, 1),
                     "useful_TFLOPS": round(4.0 * B * H * float(cfg.N) ** 2 * 128 / t_dense / 1e12, 1)}
        log(f"[bench] dense comparator (every block kept): {t_dense * 1e3:.2f} ms")

    flushed_res = flushed(p, args.flushed_reps) if args.flushed_reps > 0 else None
    if flushed_res:
        log(f"[bench] {args.flushed_reps} steps after a cache flush each: median {flushed_res['step_ms_median']:.3f} ms, "
            f"min {flushed_res['step_ms_min']:.3f} ms")
    log(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step (route {t_route*1e6:.1f} us, "
        f"attn {t_attn*1e3:.3f} ms" + (f", V quantisation {t_quant*1e6:.1f} us)" if fp8 else ")"))

    m_np = mask.cpu().numpy()
    c_np = counts.cpu().numpy()
    kept = int(c_np.sum())
    d = 128
    N = cfg.N
    kept_tile_flops = 4.0 * 128 * 128 * d * kept
    useful_flops = 4.0 * d * real_pairs(m_np, sizes)
    dense_flops = 4.0 * B * H * float(N) ** 2 * d
    route_bytes = 2.0 * B * H * N * d * 2 + B * H * nb * nb + 4.0 * B * H * nb + 4.0 * kept
    here = os.path.dirname(os.path.abspath(__file__))
    csrc = os.path.join(here, "paper_2607_16190_amd", "csrc")
    shared = [os.path.join(csrc, f) for f in ("fva_common.h", "fva_geometry.h")]
    digest = source_digest(os.path.join(csrc, "attn_kernels.hip"), *shared)
    traffic = None
    bench_workload = ((cfg.name if curve is None else cfg.name + "-hilbert") + ("-fp8v" if fp8 else "")
                      + (f"-sasa{args.sasa}" if args.sasa else ""))
    if ATTN_TRAFFIC["source_digest"] == digest and args.sched == "persistent":
        traffic = ATTN_TRAFFIC["bytes"].get(bench_workload)
    route_digest = source_digest(os.path.join(csrc, "route_kernels.hip"), *shared)
    route_traffic = None
    if ROUTE_TRAFFIC["source_digest"] == route_digest:
        route_traffic = ROUTE_TRAFFIC["bytes"].get(bench_workload)
    peak = PEAK_BF16_FP8_TFLOPS if fp8 else PEAK_BF16_TFLOPS
    res = {
        "metric": METRIC,
        "value": round(dense_flops / (ms_per_step / 1e3) / 1e12, 2),
        "unit": "TFLOPS (dense-equivalent, route + attention step)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 Q/K, e4m3 V and P (fp32 accumulation)" if fp8 else "bf16",
        "data": "synthetic (seeded video-shaped Q/K/V, sinusoidal (t,y,x) embedding, per-head alpha)",
        "config": {
            "workload": f"{cfg.name}: {H} heads, d=128, latent grid {'x'.join(map(str, cfg.grid))} = {N} tokens, "
            + (f"tile {'x'.join(map(str, cfg.tile))}" if curve is None
               else f"Hilbert-curve blocks of {int(np.prod(cfg.tile))} tokens")
            + f", nb={nb}, p={p}, k_min={cfg.k_min}" + (", E4M3 V (quantised each step)" if fp8 else "")
            + (f", slack-aware augmentation over {args.sasa} ranks of {H // args.sasa} heads" if args.sasa else ""),
            "blocks": args.blocks,
            "v": args.vfmt,
            "batch": B,
            "heads": H,
            "tokens": N,
            "p": p,
            "k_min": cfg.k_min,
            "scheduler": args.sched,
            **({"head_order": "reversed"} if args.reverse_heads else {}),
            "parallelism": "single GPU",
        },
        "attn_ms": round(t_attn * 1e3, 4),
        **({"v_quantise_us": round(t_quant * 1e6, 1)} if fp8 else {}),
        "route_us": round(t_route * 1e6, 2),
        "route_GBps": round(route_bytes / t_route / 1e9, 1),
        "route_frac_hbm": round(route_bytes / t_route / 1e9 / PEAK_HBM_GBPS, 4),
        "route_roofline": {
            "bound": "hbm",
            "achieved": round(route_bytes / t_route / 1e9, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(route_bytes / t_route / 1e9 / PEAK_HBM_GBPS, 4),
            "traffic": route_traffic,
            "algorithmic_bytes_per_call": route_bytes,
        },
        "kept_tile_TFLOPS": round(kept_tile_flops / t_attn / 1e12, 2),
        "kept_tile_frac_bf16_peak": round(kept_tile_flops / t_attn / 1e12 / PEAK_BF16_TFLOPS, 4),
        "kept_tile_frac_bf16_2516": round(kept_tile_flops / t_attn / 1e12 / PEAK_BF16_TFLOPS_2400, 4),
        "useful_frac_bf16_2516": round(useful_flops / t_attn / 1e12 / PEAK_BF16_TFLOPS_2400, 4),
        "kept_tile_frac_peak": round(kept_tile_flops / t_attn / 1e12 / peak, 4),
        "useful_TFLOPS": round(useful_flops / t_attn / 1e12, 2),
        "dense_equiv_attn_TFLOPS": round(dense_flops / t_attn / 1e12, 2),
        "retained_fraction": round(kept / (B * H * nb * nb), 4),
        "roofline": {
            "bound": "mfma",
            "achieved": round(useful_flops / t_attn / 1e12, 2),
            "peak": round(peak, 1),
            "unit": "TFLOP/s",
            "frac": round(useful_flops / t_attn / 1e12 / peak, 4),
            "traffic": traffic,
            "kernel": "attn_persistent_kernel (fva_attn; timed with its plan_kernel)" if not fp8 else
            "attn_persistent_kernel<true> (fva_attn_fp8v; timed with its plan_kernel); peak = bf16 Q K^T and "
            "fp8 P V at their own peaks",
            "algorithmic_flops_per_launch": useful_flops,
            "attn_source_digest": digest,
        },
    }
    if dense_res:
        dense_res["speedup_attn"] = round(dense_res["attn_ms"] / (t_attn * 1e3), 3)
        dense_res["speedup_step"] = round(dense_res["attn_ms"] / ms_per_step, 3)
        res["dense_comparator"] = dense_res
    if flushed_res:
        res["flushed_steps"] = flushed_res
    if curve is not None:
        res["curve_layout"] = curve
    if args.sasa:
        # loads before the augmentation, from a plain routing pass outside the timed region
        c_aug = c_np.reshape(B * H, nb).astype(np.int64)
        m0 = torch.empty_like(mask)
        c0 = torch.empty_like(counts)
        ws0 = torch.empty(fva.fva_route_workspace_size(desc, tiling), dtype=torch.uint8, device=dev)
        kv0 = torch.empty_like(kv)
        fva.fva_route(q, k, p, cfg.k_min, tiling, out=(m0, c0, kv0), workspace=ws0)
        torch.cuda.synchronize()

        def rank_times(mm, cc, kk, reps=3):
            """Attention time of each rank's heads alone (what that rank's GPU would run)."""
            hp = H // args.sasa
            out_t = []
            for r in range(args.sasa):
                sl = slice(r * hp, (r + 1) * hp)
                qs, ks_, vs = q[:, sl], k[:, sl], v[:, sl]
                ms, cs, kvs = mm[:, sl], cc[:, sl], kk[:, sl]
                o_s = torch.empty_strided(qs.shape, qs.stride(), dtype=torch.bfloat16, device=dev)
                if fp8:
                    v8s, vexps = v8[:, sl], vexp[:, sl]
                    fn = lambda: fva.fva_attn_fp8v(qs, ks_, v8s.contiguous(), vexps.contiguous(), tiling, ms, cs, kvs,
                                                   out=o_s, workspace=ws_a)
                else:
                    fn = lambda: fva.fva_attn(qs, ks_, vs, tiling, ms, cs, kvs, out=o_s, workspace=ws_a)
                fn()
                torch.cuda.synchronize()
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                ev[0].record(stream)
                for _ in range(reps):
                    fn()
                ev[1].record(stream)
                torch.cuda.synchronize()
                out_t.append(ev[0].elapsed_time(ev[1]) / reps)
            return out_t
        c_plain = c0.cpu().numpy().reshape(B * H, nb).astype(np.int64)
        ro = rank_of.cpu().numpy()
        S0 = np.bincount(ro, weights=c_plain.sum(axis=1), minlength=args.sasa) / nb
        S1 = np.bincount(ro, weights=c_aug.sum(axis=1), minlength=args.sasa) / nb
        res["sasa"] = {
            "ranks": args.sasa, "n1": 0.8, "n2": 0.07,
            "extra_blocks_per_row": rank_extra.cpu().numpy().tolist(),
            "rank_load_rows_before": np.round(S0, 2).tolist(),
            "rank_load_rows_after": np.round(S1, 2).tolist(),
            "rho_before": round(float(S0.max() / S0.mean()), 4),
            "rho_after": round(float(S1.max() / S1.mean()), 4),
            "retained_before": round(float(c_plain.sum()) / (B * H * nb * nb), 4),
            "retained_after": round(float(c_aug.sum()) / (B * H * nb * nb), 4),
        }
        if B == 1:
            t0 = rank_times(m0, c0, kv0)
            t1 = rank_times(mask, counts, kv)
            res["sasa"]["rank_attn_ms_before"] = [round(x, 3) for x in t0]
            res["sasa"]["rank_attn_ms_after"] = [round(x, 3) for x in t1]
            res["sasa"]["critical_attn_ms_before_after"] = [round(max(t0), 3), round(max(t1), 3)]
        log(f"[bench] sasa: {res['sasa']}")
    if not args.no_trace:
        tw = fva.fva_trace_words(desc, tiling)
        trace = torch.zeros(tw, dtype=torch.int64, device=dev)
        imb = {}
        for name, fl in (("persistent", fva.FVA_SCHED_PERSISTENT), ("naive", fva.FVA_SCHED_NAIVE)):
            trace.zero_()
            attend(fl | fva.FVA_TRACE, trace)
            torch.cuda.synchronize()
            imb[name] = imbalance(trace.cpu().numpy(), c_np, tiling, fl == fva.FVA_SCHED_PERSISTENT)
        res["scheduler_trace"] = imb
        log(f"[bench] trace: {imb}")
        # engine clock of the traced persistent run, and the attention's
        # fraction of the peak at that clock
        sclk = imb["persistent"]["sclk_mhz"]
        res["sclk_mhz"] = sclk
        peak_clk = CUS * BF16_FLOP_PER_CLK_CU * sclk * 1e6 / 1e12
        if not fp8:
            res["roofline"]["peak_at_sclk"] = round(peak_clk, 1)
            res["roofline"]["frac_at_sclk"] = round(useful_flops / t_attn / 1e12 / peak_clk, 4)
            res["kept_tile_frac_at_sclk"] = round(kept_tile_flops / t_attn / 1e12 / peak_clk, 4)
    if not args.no_extra and args.workload == "720p" and not args.sasa:
        res.update(extra_workloads(torch, fva, synth, dev))
        res["gemm_ceiling"] = gemm_ceiling(torch)
        log(f"[bench] vendor bf16 GEMM: {res['gemm_ceiling']}")
        res["roofline"]["frac_of_gemm_ceiling"] = round(useful_flops / t_attn / 1e12 / res["gemm_ceiling"]["TFLOPS"], 4)
    if args.p_sweep:
        sweep = []
        for pp in [float(x) for x in args.p_sweep.split(",")]:
            msp, tr_, ta_ = timed(pp, max(2, args.steps // 2), 1)
            cc = counts.cpu().numpy()
            sweep.append({"p": pp, "retained_fraction": round(float(cc.sum()) / (B * H * nb * nb), 4),
                          "ms_per_step": round(msp, 3), "route_us": round(tr_ * 1e6, 1),
                          "attn_ms": round(ta_ * 1e3, 3)})
            log(f"[bench] p={pp}: {sweep[-1]}")
        res["p_sweep"] = sweep
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline(cfg, Qb, Kb, Vb, m_np, c_np, args.cpu_budget, args.blocks)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
