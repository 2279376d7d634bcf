"""Puts with radix dedup (mlkv_set_dedup(MLKV_DEDUP_RADIX): a stable LSD
radix sort of the batch's items by row, then run-length encoding) against
the oracle, which has one dedup only: results must not depend on the mode.

* the scaled workloads, inserts in gets and in puts, all three put ops;
* a hot key over many tiles, every position one key, ragged and tiny batches;
* a capacity overflow inside a put (the whole call rolls back);
* the same calls on a hash-dedup table give bit-identical tables (both sum a
  key's items in fp64 in position order, split between lane groups at
  different places; the rounded results agree on these inputs);
* the full-size DLRM table for three steps, as the bench runs it;
* staleness counts on a bounded table and a tiered table's cache;
* the per-call limit (2^20 keys) and unknown modes are refused.
"""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, dev, dev_keys, log, record

pytestmark = pytest.mark.gpu


def run_config(name, scale, steps):
    wl = W.make(name, scale=scale, steps=steps)
    log(f"[radix] {name} scale={scale} n={wl.n} dim={wl.dim} cap={wl.capacity}")
    pr = Pair(wl.dim, wl.capacity, dedup="radix")
    pre = wl.prefill_keys()
    if pre.size:
        pr.prefill(pre)
    for s in range(steps):
        keys = wl.keys(s)
        pr.get(keys)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        pr.compare_rows()
        log(f"[radix] {name} step {s} ok size={pr.ora.size} stats={pr.stats}")
    pr.check_index()
    record(f"radix dedup {name}@{scale}x{steps}", pr.stats)
    pr.close()


def test_tiny_with_inserts_every_step():
    run_config("tiny", 1.0, 6)


@pytest.mark.parametrize("name,scale", [("dlrm", 0.01), ("kg", 0.002), ("gnn", 0.005), ("large", 0.005)])
def test_scaled_configs(name, scale):
    run_config(name, scale, 3)


def test_puts_that_insert_and_every_op():
    rng = np.random.default_rng(41)
    dim = 12
    pr = Pair(dim, 20000, dedup="radix")
    for n in (1, 63, 1000, 4097, 9000):
        keys = rng.integers(0, 6000, size=n).astype(np.uint64) * np.uint64(0x9E3779B1)
        g = rng.normal(0, 0.01, size=(n, dim)).astype(np.float32)
        pr.put(keys, g, 0.02, 1e-8)          # unseen keys are inserted by the put itself
        pr.put_sgd(keys, g, 0.1)
        vals = rng.normal(0, 1, size=(n, dim)).astype(np.float32)
        pr.upsert(keys, vals)                # last position wins
        pr.get(keys)
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_hot_keys_across_many_tiles():
    rng = np.random.default_rng(42)
    dim = 64
    pr = Pair(dim, 100000, dedup="radix")
    n = 200000
    keys = rng.integers(0, 50000, size=n).astype(np.uint64)
    keys[::3] = 7                            # one key in every put tile, a third of the batch
    keys[1::97] = 11
    pr.get(keys)
    for s in range(2):
        pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
    one = np.full(n, 5, dtype=np.uint64)     # every position the same key
    pr.put(one, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
    pr.compare_rows()
    pr.check_index()
    record("radix dedup hot keys", pr.stats)
    pr.close()


def test_overflow_in_a_put_rolls_the_call_back():
    rng = np.random.default_rng(43)
    pr = Pair(8, 3000, dedup="radix")
    first = rng.choice(np.arange(1, 10**6, dtype=np.uint64), size=2500, replace=False)
    pr.put(first, rng.normal(0, 0.01, size=(2500, 8)).astype(np.float32), 0.01, 1e-8)
    over = rng.choice(np.arange(10**6, 2 * 10**6, dtype=np.uint64), size=800, replace=False)
    both = np.concatenate([first[:300], over])
    pr.gpu.put_grad(dev_keys(both), dev(np.ones((both.size, 8), np.float32)), 0.01, 1e-8)
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    assert pr.gpu.size == 2500
    pr.compare_rows()                        # nothing changed, not even the 300 present keys
    pr.check_index()
    pr.close()


def test_same_tables_as_hash_dedup():
    wl = W.make("dlrm", scale=0.02, steps=3)
    tabs = {m: mlkv.Table(wl.dim, wl.capacity, dedup=m) for m in ("hash", "radix")}
    pre = dev_keys(wl.prefill_keys())
    for t in tabs.values():
        t.get(pre, None)
    for s in range(3):
        k = dev_keys(wl.keys(s))
        g = dev(wl.grads(s))
        for t in tabs.values():
            t.get(k, None)
            t.put_grad(k, g, wl.lr, wl.eps)
    out = {}
    for m, t in tabs.items():
        assert t.sync() == mlkv.MLKV_OK
        rows = torch.arange(t.size, dtype=torch.int64, device="cuda")
        w, st = t.read_rows(rows)
        out[m] = (w.cpu().numpy(), st.cpu().numpy())
        t.close()
    assert np.array_equal(out["hash"][0].view(np.uint32), out["radix"][0].view(np.uint32))
    assert np.array_equal(out["hash"][1].view(np.uint32), out["radix"][1].view(np.uint32))


@pytest.mark.slow
def test_full_size_dlrm():
    wl = W.make("dlrm", scale=1.0, steps=3)
    pr = Pair(wl.dim, wl.capacity, lazy_oracle=True, dedup="radix")
    pr.prefill(wl.prefill_keys())
    touched = []
    for s in range(3):
        keys = wl.keys(s)
        pr.get(keys, check=(s == 0))
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        touched.append(keys)
        log(f"[radix] full dlrm step {s}")
    pr.compare_rows(np.unique(pr.ora.lookup_rows(np.concatenate(touched))))
    record("radix dedup full-dlrm-3steps", pr.stats)
    pr.close()


def test_limits():
    t = mlkv.Table(4, 1000)
    with pytest.raises(mlkv.MlkvError):
        mlkv._check(mlkv.mlkv_set_dedup(t.h, 7))
    t.set_dedup("radix")
    n = (1 << 20) + 1
    k = torch.zeros(n, dtype=torch.int64, device="cuda")
    g = torch.zeros((n, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(mlkv.MlkvError):
        t.put_grad(k, g, 0.01, 1e-8)
    t.set_dedup("hash")
    t.close()


def test_bounded_staleness_counts_with_radix():
    # gets two steps ahead of the puts (bound 1: some keys block); every put
    # op lowers the counts of its distinct keys once, as with hash dedup
    rng = np.random.default_rng(44)
    dim = 16
    pr = Pair(dim, 30_000, staleness_bound=1, dedup="radix")
    batches, nblocked = [], 0
    for s in range(9):
        k = rng.integers(0, 7000, size=int(rng.integers(1000, 5000))).astype(np.uint64) * np.uint64(0x9E3779B1)
        batches.append(k)
        bl = pr.get_bounded(k)
        nblocked += int(bl.sum())
        if len(batches) > 2:
            done = batches.pop(0)
            g = rng.normal(0, 0.01, size=(done.size, dim)).astype(np.float32)
            if s % 3 == 0:
                pr.put(done, g, 0.01, 1e-8)
            elif s % 3 == 1:
                pr.put_sgd(done, g, 0.05)
            else:
                pr.upsert(done, g)
            if bl.any():
                pr.get_bounded(batches[-1][bl == 1])
        pr.compare_staleness()
    assert nblocked > 0
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_tiered_table_with_radix():
    wl = W.make("dlrm", scale=0.02, steps=4)
    cache = int(wl.capacity * 0.2)
    pr = Pair(wl.dim, wl.capacity, cache_rows=cache, dedup="radix")
    pr.prefill(wl.prefill_keys())
    for s in range(4):
        keys = wl.keys(s)
        pr.lookahead(keys)
        pr.get(keys)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
    st = pr.gpu.cache_stats()
    assert st["loaded"] > 0 and st["loaded"] == st["filled"] + st["evicted"] and st["filled"] <= cache
    pr.compare_rows()
    record("radix dedup tiered dlrm@0.02x4 cache=0.2", {**pr.stats, **st})
    pr.close()


def test_reserved_key_in_a_put_fails_the_whole_call():
    rng = np.random.default_rng(45)
    pr = Pair(8, 5000, dedup="radix")
    keys = rng.choice(np.arange(1, 10**6, dtype=np.uint64), size=1500, replace=False)
    pr.put(keys[:1000], rng.normal(0, 0.01, size=(1000, 8)).astype(np.float32), 0.01, 1e-8)
    bad = keys.copy()
    bad[700] = np.uint64(mlkv.MLKV_RESERVED_KEY)  # and 500 keys never seen
    pr.gpu.put_grad(dev_keys(bad), dev(np.ones((bad.size, 8), np.float32)), 0.01, 1e-8)
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    assert pr.gpu.size == 1000
    pr.compare_rows()  # no row changed, nothing inserted
    pr.check_index()
    pr.close()
