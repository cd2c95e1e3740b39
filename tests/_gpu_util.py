"""Helpers shared by the GPU parity tests: input upload, oracle conversions."""

import functools

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
