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


def test_unknown_dedup_mode_is_refused():
    r = _run("--dedup", "bucket")
    assert r.returncode == 2
    assert "--dedup" in r.stderr


def test_radix_dedup_moves_the_reduce_bytes_to_its_reduce_kernel():
    sys.path.insert(0, ROOT)
    import bench
    for n, U, M, D in ((212_992, 60_864, 0, 64), (4096, 1700, 1700, 16)):
        h = bench.kernel_bytes(n, U, M, D)
        r = bench.kernel_bytes(n, U, M, D, "radix")
        assert sum(h.values()) == sum(r.values())
        assert r["rsort_reduce"] == h["put_reduce"] and r["put_reduce"] == 0
        assert r["rsort_count"] == r["rsort_scatter"] == 0
    kv_h = bench.kernel_bytes_kv(1 << 19, 400_000, 1 << 19, 400_000, 4)
    kv_r = bench.kernel_bytes_kv(1 << 19, 400_000, 1 << 19, 400_000, 4, "radix")
    assert sum(kv_h.values()) == sum(kv_r.values()) and kv_r["rsort_reduce"] == kv_h["put_reduce"]


def test_pipelined_steps_are_refused_at_bound_zero_and_for_the_key_value_mix():
    for extra in (("--staleness-bound", "0"), ("--config", "kv-zipf")):
        r = _run("--pipelined", *extra)
        assert r.returncode == 2
        assert "--pipelined" in r.stderr
