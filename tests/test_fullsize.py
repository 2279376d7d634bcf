"""GPU against the oracle at the workloads' full sizes, in the same calls the
benchmark times (a table opened with the default load factor, get(keys, out)
then put_grad(keys, grads) on one stream).

Compared every step: the whole get output (bit-exact for rows never updated,
1e-5 row-scaled otherwise), key -> row of every key of the batch (bit-exact),
every row the step updated and its accumulator (1e-5), and a seeded sample of
other rows (bit-exact, initial values); table size after every call.
"""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, dev, dev_keys, log, record

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

STEPS = {"dlrm": 3, "kg": 2, "gnn": 2, "large": 2}


def check_step(pr, keys, rng, n_sample=20000):
    # key -> row of the batch
    want_rows = pr.ora.lookup_rows(keys)
    got_rows = pr.gpu.lookup_rows(dev_keys(keys)).cpu().numpy()
    assert np.array_equal(got_rows, want_rows), "key -> row differs"
    # rows updated by the step, and a sample of the rest
    touched = np.unique(want_rows)
    size = pr.ora.size
    assert pr.gpu.size == size
    other = rng.integers(0, size, size=n_sample).astype(np.int64)
    pr.compare_rows(touched)
    pr.compare_rows(np.unique(other))


@pytest.mark.parametrize("name", ["dlrm", "kg", "gnn", "large"])
def test_full_size_config(name):
    wl = W.make(name, scale=1.0)
    steps = STEPS[name]
    log(f"[full] {name}: cap={wl.capacity} dim={wl.dim} n={wl.n} steps={steps}")
    pr = Pair(wl.dim, wl.capacity)
    pre = wl.prefill_keys()
    if pre.size:
        pr.prefill(pre)
    log(f"[full] {name}: prefilled {pre.size} keys, size={pr.gpu.size}")
    del pre
    rng = np.random.default_rng(99)
    for s in range(steps):
        keys = wl.keys(s)
        pr.get(keys)
        log(f"[full] {name} step {s}: get ok, size={pr.ora.size}")
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        check_step(pr, keys, rng)
        log(f"[full] {name} step {s}: put ok, stats={pr.stats}")
    record(f"full-{name}-{steps}steps", pr.stats)
    pr.close()


def test_full_size_dlrm_all_100_steps():
    """The DLRM-shaped workload for its stated 100 steps: every get and put
    on both sides; the get output compared in full, key -> row of the batch,
    the rows each step updated and a sample of the others every 10th step
    (fp32 drift over a real run stays within the bound)."""
    wl = W.make("dlrm", scale=1.0)
    pr = Pair(wl.dim, wl.capacity)
    pr.prefill(wl.prefill_keys())
    rng = np.random.default_rng(100)
    for s in range(100):
        keys = wl.keys(s)
        check = s % 10 == 9
        pr.get(keys, check=check)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        if check:
            check_step(pr, keys, rng, n_sample=5000)
            log(f"[full] dlrm step {s}: ok, stats={pr.stats}")
    record("full-dlrm-100steps", pr.stats)
    pr.close()


@pytest.mark.parametrize("name,bound", [("dlrm", None), ("dlrm", 1), ("kg", None), ("gnn", None)])
def test_full_size_pipelined(name, bound):
    """A workload in the calls `bench.py --pipelined` times: the get of batch
    s and the put_grad of batch s - 1 in one mlkv_get_put_grad call (the
    oracle takes the get, then the put), unbounded and (DLRM) at staleness
    bound 1; every output and the rows each put updated compared."""
    wl = W.make(name, scale=1.0)
    pr = Pair(wl.dim, wl.capacity, staleness_bound=bound)
    pr.prefill(wl.prefill_keys())
    rng = np.random.default_rng(101)
    prev = wl.keys(0)
    if bound is None:
        pr.get(prev)
    else:
        assert not pr.get_bounded(prev).any()
    for s in range(1, STEPS[name] + 1):
        keys = wl.keys(s)
        bl = pr.get_put_grad(keys, prev, wl.grads(s - 1), wl.lr, wl.eps)
        assert bl is None or not bl.any()
        check_step(pr, prev, rng, n_sample=5000)
        log(f"[full] {name} pipelined bound {bound} step {s}: ok, stats={pr.stats}")
        prev = keys
    if bound is not None:
        pr.compare_staleness()
    record(f"full-{name}-pipelined-bound{bound}", pr.stats)
    pr.close()


def test_full_size_ragged_batch_and_repeat():
    """DLRM-sized table, a batch whose length is not a multiple of any tile,
    then the same keys again (all present)."""
    wl = W.make("dlrm", scale=1.0)
    pr = Pair(wl.dim, wl.capacity)
    pr.prefill(wl.prefill_keys())
    rng = np.random.default_rng(7)
    keys = wl.keys(0)[: 212992 - 333]
    for _ in range(2):
        pr.get(keys)
        pr.put(keys, rng.normal(0, 0.01, size=(keys.size, wl.dim)).astype(np.float32), wl.lr, wl.eps)
        check_step(pr, keys, rng, n_sample=5000)
    log(f"[full] ragged ok, stats={pr.stats}")
    pr.close()


def test_full_size_max_batch_of_one_hot_key():
    """The largest batch the benchmark issues, every position one key: the
    longest possible segment (212,992 gradient rows into one row)."""
    dim, n = 64, 212992
    pr = Pair(dim, 1000)
    keys = np.full(n, 12345, dtype=np.uint64)
    rng = np.random.default_rng(8)
    pr.get(keys)
    pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
    pr.compare_rows()
    log(f"[full] one-hot ok, stats={pr.stats}")
    pr.close()


def test_full_size_dlrm_bounded_staleness_pipeline():
    """DLRM-sized table with staleness bound 0, each step's get issued before
    the previous step's put: the keys shared with the pending step are blocked
    (flags compared at every position), fetched again after the put, and the
    counts end at 0 for every key."""
    wl = W.make("dlrm", scale=1.0)
    pr = Pair(wl.dim, wl.capacity, staleness_bound=0)
    pr.prefill(wl.prefill_keys())
    rng = np.random.default_rng(12)
    prev = wl.keys(0)
    bl = pr.get_bounded(prev)
    assert not bl.any()
    for s in range(1, 3):
        keys = wl.keys(s)
        bl = pr.get_bounded(keys)
        assert bl.any()
        pr.put(prev, wl.grads(s - 1), wl.lr, wl.eps)
        again = pr.get_bounded(keys[bl == 1])
        assert not again.any()
        log(f"[full] bounded step {s}: {int(bl.sum())} blocked positions, stats={pr.stats}")
        prev = keys
    pr.put(prev, wl.grads(2), wl.lr, wl.eps)
    rows = np.unique(pr.ora.lookup_rows(np.concatenate([wl.keys(s) for s in range(3)])))
    got = pr.gpu.read_staleness(torch.from_numpy(rows).cuda()).cpu().numpy()
    assert np.all(got == 0) and np.all(pr.ora.staleness(rows) == 0)
    pr.compare_rows(rows)
    pr.close()
