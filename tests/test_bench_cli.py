"""bench.py's argument checks that run before any GPU work."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_staleness_bound_is_refused_for_the_key_value_mix():
    r = _run("--config", "kv-uniform", "--staleness-bound", "0")
    assert r.returncode == 2
    assert "staleness-bound" in r.stderr
