"""Calibration of the synthetic generator's embedding gain (run by hand).

Prints the retained block density that the oracle's routing gives, on the
720p shape (p = 0.9, k_min = 4), for a range of per-head alphas and candidate
gains. The chosen gain (synth.video.GAMMA2) is the one for which density
spreads from ~80 % at alpha = 0.5 to a few % at alpha = 4, and reaches ~90 %
at alpha = 0.3 and < 5 % at alpha = 5.

    python tests/calibrate_inputs.py
"""

import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import synth  # noqa: E402
from oracle import block_scores, block_softmax, pool_blocks, tile_geometry, topp_select  # noqa: E402


def main():
    cfg = synth.get_config("720p")
    geo = tile_geometry(*cfg.grid, *cfg.tile)
    q0 = pool_blocks(np.random.default_rng([cfg.seed, 0, 0]).standard_normal((cfg.N, 128), dtype=np.float32), geo)
    k0 = pool_blocks(np.random.default_rng([cfg.seed, 0, 1]).standard_normal((cfg.N, 128), dtype=np.float32), geo)
    eb = pool_blocks(synth.positional_embedding(cfg.grid, cfg.tile), geo)
    alphas = [0.3, 0.5, 1, 2, 3, 4, 5]
    print("gamma2 " + " ".join("a=%-5g" % a for a in alphas))
    for g2 in (0.2, 0.3, 0.4, 0.5):
        row = []
        for a in alphas:
            g = np.sqrt(g2 * a)
            s = block_scores(q0 + g * eb, k0 + g * eb)
            row.append(topp_select(s, block_softmax(s), cfg.p, cfg.k_min)["counts"].mean() / geo.nb)
        print("%-6g " % g2 + " ".join("%-7.3f" % x for x in row))


if __name__ == "__main__":
    main()
