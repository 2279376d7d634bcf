"""Tiered tables (rows at home in pinned host memory, an HBM cache of a fifth
of them, filled by Lookahead) against the oracle, which has no tiers: the
cache must never change a result.

* DLRM-shaped tables with the cache forced to 20 % of the rows: a lookahead
  warms the cache, then steps of lookahead(keys), get(keys), put_grad(keys);
  the cache evicts rows every step and writes back the ones puts changed.
* A cache smaller than one batch (rows beyond it stay at home), puts on rows
  that are later evicted and read back from home, gets and puts without any
  lookahead (every row at home), and ordinary Put / SGD updates.
"""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, dev, dev_keys, log, record

pytestmark = pytest.mark.gpu


def dlrm_run(scale, steps, cache_frac=0.2):
    wl = W.make("dlrm", scale=scale, steps=steps)
    cache = max(1, int(wl.capacity * cache_frac))
    pr = Pair(wl.dim, wl.capacity, cache_rows=cache)
    pre = wl.prefill_keys()
    pr.prefill(pre)
    # warm the cache with a slice of the table
    rng = np.random.default_rng(31)
    warm = rng.choice(pre, size=min(cache, pre.size), replace=False)
    pr.lookahead(warm)
    st0 = pr.gpu.cache_stats()
    assert st0["loaded"] == warm.size and st0["filled"] == warm.size
    for s in range(steps):
        keys = wl.keys(s)
        pr.lookahead(keys)
        pr.get(keys)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        log(f"[tiered] dlrm@{scale} step {s}: {pr.gpu.cache_stats()} stats={pr.stats}")
    st = pr.gpu.cache_stats()
    assert st["evicted"] > 0 and st["written_back"] > 0, st
    assert st["filled"] == cache
    touched = np.unique(pr.ora.lookup_rows(np.concatenate([wl.keys(s) for s in range(steps)])))
    pr.compare_rows(touched)
    sample = np.unique(rng.integers(0, pr.ora.size, size=20000))
    pr.compare_rows(sample)
    record(f"tiered dlrm@{scale}x{steps} cache={cache_frac}", {**pr.stats, **st})
    pr.close()
    return st


def test_tiered_dlrm_scaled_with_a_fifth_cached():
    dlrm_run(0.02, 6)


@pytest.mark.slow
def test_tiered_dlrm_full_size_with_a_fifth_cached():
    st = dlrm_run(1.0, 4)
    log(f"[tiered] full-size counters: {st}")


def test_cache_smaller_than_a_batch_and_evicted_rows_read_back_from_home():
    rng = np.random.default_rng(32)
    dim, cap, cache = 16, 5000, 300
    pr = Pair(dim, cap, cache_rows=cache)
    a = rng.choice(np.arange(1, 10**6, dtype=np.uint64), size=1000, replace=False)
    b = rng.choice(np.arange(10**6, 2 * 10**6, dtype=np.uint64), size=1000, replace=False)
    pr.lookahead(a)                      # 1000 rows asked, 300 slots: the rest stay at home
    st = pr.gpu.cache_stats()
    assert st["loaded"] == cache and st["filled"] == cache
    pr.get(a)
    pr.put(a, rng.normal(0, 0.01, size=(a.size, dim)).astype(np.float32), 0.05, 1e-8)  # cached and home rows
    pr.lookahead(b)                      # evicts a's cached rows, writing the changed ones back
    st = pr.gpu.cache_stats()
    assert st["evicted"] == cache and st["written_back"] == cache, st
    pr.get(a)                            # from home
    pr.get(b)
    pr.put(np.concatenate([a, b]), rng.normal(0, 0.01, size=(2000, dim)).astype(np.float32), 0.05, 1e-8)
    pr.lookahead(a[:200])
    pr.get(a)
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_tiered_table_without_lookahead_and_other_updates():
    rng = np.random.default_rng(33)
    dim, cap = 8, 4000
    pr = Pair(dim, cap, cache_rows=100)
    keys = rng.integers(0, 3000, size=2500).astype(np.uint64)
    pr.get(keys)                         # every row at home
    pr.put(keys, rng.normal(0, 0.01, size=(keys.size, dim)).astype(np.float32), 0.01, 1e-8)
    pr.lookahead(keys[:150])
    pr.put_sgd(keys, rng.normal(0, 0.01, size=(keys.size, dim)).astype(np.float32), 0.1)
    pr.upsert(keys[::3].copy(), rng.normal(0, 1, size=(keys[::3].size, dim)).astype(np.float32))
    pr.lookahead(keys[1000:1100])
    pr.get(keys)
    pr.compare_rows()
    st = pr.gpu.cache_stats()
    assert st["loaded"] > 0 and st["filled"] == 100
    pr.close()


def test_tiered_open_rejects_bad_cache_sizes():
    with pytest.raises(mlkv.MlkvError):
        mlkv.Table(4, 100, cache_rows=0)
    with pytest.raises(mlkv.MlkvError):
        mlkv.Table(4, 100, cache_rows=101)
    t = mlkv.Table(4, 100)
    with pytest.raises(mlkv.MlkvError):
        t.cache_stats()
    t.close()
