"""bench.py's host-side contract, without a GPU.

* More than one GPU (the flag, or a launcher's WORLD_SIZE) is refused with
  exit status 2 and a message, before anything touches a device: the path
  is measured on one GPU and shards by head across GPUs.
* Every option parses (--help lists them).
"""

import os
import subprocess
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
