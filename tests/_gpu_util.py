"""Helpers shared by the GPU parity tests: input upload, oracle conversions."""

import functools
import os

import numpy as np

import synth
from oracle import tile_geometry


def torch_mod():
    import torch

    return torch


def lib():
    import paper_2607_16190_amd as fva

    return fva


def to_dev(bits: np.ndarray):
    """uint16 bf16 bit patterns -> bf16 tensor on cuda:0."""
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def f64(bits: np.ndarray) -> np.ndarray:
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def tiling_of(cfg):
    return lib().Tiling(*cfg.grid, *cfg.tile)


def geometry_of(cfg):
    return tile_geometry(*cfg.grid, *cfg.tile)


@functools.lru_cache(maxsize=2)
def workload(name: str):
    """Host bits of a named workload (cached: full-size generation takes seconds)."""
    return synth.gen_qkv(synth.get_config(name))


def custom_config(name, heads, grid, tile, alphas, seed, p=0.9, k_min=4):
    return synth.WorkloadConfig(name, heads, grid, tile, p, k_min, seed, "fixed", tuple(alphas))


def log(msg: str):
    print(msg, flush=True)


def pool_threads() -> int:
    """Worker threads for oracle evaluation: the CPU share, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def map_blocks(fn, blocks, threads=None):
    """fn(list of query blocks) -> dict, evaluated over chunks of `blocks` in a
    thread pool (numpy releases the GIL in its gathers, ufuncs and BLAS calls;
    BLAS runs one thread per worker), merged into one dict."""
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    blocks = list(blocks)
    n = min(threads or pool_threads(), max(1, len(blocks)))
    chunks = [blocks[k::n] for k in range(n)]
    out = {}
    with threadpool_limits(limits=1, user_api="blas"):
        with ThreadPoolExecutor(max_workers=n) as ex:
            for part in ex.map(fn, chunks):
                out.update(part)
    return out


def rule_rows(counts, nb, seed, n_random=64, all_heads=False):
    """Query blocks compared at full size: every block of the lowest- and
    highest-density heads and of two random other heads, plus n_random random
    (head, block) rows elsewhere; every block of every head with all_heads.
    counts: [heads, nb] kept blocks per row. Returns {head: sorted blocks}."""
    H = counts.shape[0]
    rng = np.random.default_rng(seed)
    if all_heads:
        return {h: list(range(nb)) for h in range(H)}
    dens = counts.mean(axis=-1)
    heads = [int(np.argmin(dens)), int(np.argmax(dens))]
    others = [h for h in range(H) if h not in heads]
    heads += [int(h) for h in rng.choice(others, min(2, len(others)), replace=False)]
    rows = {h: set(range(nb)) for h in heads}
    rest = [h for h in range(H) if h not in heads]
    added = 0
    while rest and added < n_random:
        h = int(rng.choice(rest))
        i = int(rng.integers(nb))
        if i not in rows.setdefault(h, set()):
            rows[h].add(i)
            added += 1
    return {h: sorted(v) for h, v in rows.items()}


def describe_rows(rows):
    n = sum(len(v) for v in rows.values())
    return f"{n} query blocks over {len(rows)} heads"


def attn_rule_errors(Qb, Kb, Vb, mask, O, geo, rows, scale=None, batch=0):
    """Element errors of the GPU output O [heads, N, d] (float) against the
    fp64 oracle on the given {head: query blocks}, the oracle rows computed in
    the thread pool. Returns (max abs, mean abs, elements compared)."""
    from oracle import attn_ref_rows

    emax, esum, n = 0.0, 0.0, 0
    for h, blocks in rows.items():
        Qh, Kh, Vh = f64(Qb[batch, h]), f64(Kb[batch, h]), f64(Vb[batch, h])
        mh = mask[h]

        def part(chunk):
            ref = attn_ref_rows(Qh, Kh, Vh, mh, geo, chunk, scale)
            res = {}
            for i, o in ref.items():
                e = np.abs(O[h][geo.block_tokens[i]] - o)
                res[i] = (float(e.max()) if e.size else 0.0, float(e.sum()), int(e.size))
            return res

        for mx, sm, cnt in map_blocks(part, blocks).values():
            emax = max(emax, mx)
            esum += sm
            n += cnt
    return emax, (esum / n if n else 0.0), n
