"""CPU: bench.py's command-line contract that needs no GPU."""
from __future__ import annotations

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120, env=env)


def test_more_than_one_gpu_exits_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_world_size_above_one_exits_with_a_message():
    env = dict(os.environ, WORLD_SIZE="2")
    r = _run(env=env)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_help_lists_the_workloads_and_modes():
    r = _run("--help")
    assert r.returncode == 0
    for flag in ("--workload", "--knn", "--no-graph", "--steps", "--warmup", "--gpus"):
        assert flag in r.stdout
