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
