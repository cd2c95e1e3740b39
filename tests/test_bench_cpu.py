"""bench.py's host-side contract, without a GPU.

* More than one GPU (the flag, or a launcher's WORLD_SIZE) is refused with
  exit status 2 and a message, before anything touches a device: the path
  is measured on one GPU and shards by head across GPUs.
* Every option parses (--help lists them).
* Every global name the script's functions read is defined at module level
  or is a builtin (a function deleted while still called fails here, not in
  the timed run on the GPU).
"""

import builtins
import os
import subprocess
import symtable
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def run(args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, timeout=300, env=e)


def test_more_than_one_gpu_is_refused():
    r = run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    r = run([], env={"WORLD_SIZE": "4"})
    assert r.returncode == 2


def test_help_lists_the_options():
    r = run(["--help"])
    assert r.returncode == 0
    for opt in ("--gpus", "--steps", "--warmup", "--workload", "--v", "--blocks", "--sasa", "--p-sweep",
                "--dense-reps", "--flushed-reps", "--reverse-heads", "--no-cpu-baseline"):
        assert opt in r.stdout, opt


def test_every_global_name_resolves():
    with open(BENCH) as f:
        top = symtable.symtable(f.read(), BENCH, "exec")
    defined = {s.get_name() for s in top.get_symbols() if s.is_assigned() or s.is_imported() or s.is_namespace()}
    defined |= {"__file__", "__name__", "__doc__", "__spec__"}
    missing = set()

    def walk(table):
        for child in table.get_children():
            for sym in child.get_symbols():
                name = sym.get_name()
                if sym.is_global() and sym.is_referenced() and name not in defined and not hasattr(builtins, name):
                    missing.add(f"{child.get_name()}: {name}")
            walk(child)

    walk(top)
    assert not missing, sorted(missing)


def _bench_module():
    import importlib.util

    spec = importlib.util.spec_from_file_location("bench_under_test", BENCH)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_plan_costs_follow_the_pairing_rule():
    import numpy as np

    import paper_2607_16190_amd as fva

    bench = _bench_module()
    # 3 x 16 x 64 tokens in 1 x 8 x 8 boxes: 3 t-rows x 2 lines x 8 blocks,
    # every block 64 tokens, so blocks (0,1), (2,3), ... pair; the automatic
    # chunk size is 32 here, so row 5 (40 kept blocks) is split and its pair
    # is not formed
    t = fva.Tiling(3, 16, 64, 1, 8, 8)
    c = np.full((1, 48), 3)
    c[0, 0] = 7
    c[0, 5] = 40
    want = [4, 1] * 24
    want[0] = 8
    want[4], want[5] = 4, 41
    assert [int(x) for x in bench.plan_costs(c, t, paired=True)] == want
    assert [int(x) for x in bench.plan_costs(c, t, paired=False)] == list(c[0] + 1)
    # 480p boxes (21 x 30 x 52 in 2 x 8 x 8, 11 x 4 x 7 blocks): the
    # one-frame last t-row x-pairs (3 per line), and the last, 4-token-wide
    # column pairs along y in every t-row (2 per column): 12 + 22 pairs
    t480 = fva.Tiling(21, 30, 52, 2, 8, 8)
    off = bench.pair_offsets(bench.block_sizes((21, 30, 52), (2, 8, 8)), 4, 7)
    assert (off == 1).sum() == 12 and (off == 7).sum() == 22 and (off > 0).sum() == 34
    assert off[6] == 7 and off[13] == -7 and off[20] == 7 and off[27] == -7  # column ix = 6, t-row 0
    assert off[280] == 1 and off[281] == -1 and off[286] == 7  # last t-row: x-pairs, then its column
    c480 = np.full((1, 308), 10)
    cost = bench.plan_costs(c480, t480, paired=True)
    assert (cost == 1).sum() == 34 and cost[6] == 11 and cost[13] == 1
    # 720p boxes: only the 60 blocks of the one-frame last t-row pair (5 per line)
    t720 = fva.Tiling(21, 45, 80, 2, 8, 8)
    c720 = np.full((1, 660), 10)
    cost = bench.plan_costs(c720, t720, paired=True)
    assert (cost == 1).sum() == 30 and (cost == 11).sum() == 630
    assert list(np.nonzero(cost == 1)[0][:3]) == [601, 603, 605]
