"""GPU Put (batch upsert) and the SGD Rmw against the CPU oracle.

Bar: rows written by Put equal the oracle's bit for bit (a copy); SGD rows
within 1e-5 row-scaled; key -> row bit-exact; the index invariants hold.
"""
import numpy as np
import pytest

from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dim", [1, 4, 7, 64, 400])
def test_put_upsert_and_sgd_interleaved_with_adagrad(dim):
    rng = np.random.default_rng(dim + 50)
    pr = Pair(dim, 6000)
    for n in (1, 255, 1025, 3001):
        keys = rng.integers(0, 4000, size=n).astype(np.uint64) * np.uint64(11400714819323198485)
        keys[keys == np.uint64(mlkv.MLKV_RESERVED_KEY)] = np.uint64(1)
        pr.upsert(keys, rng.normal(0, 1, size=(n, dim)).astype(np.float32))
        pr.put_sgd(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.05)
        pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
        pr.get(keys)
    pr.compare_rows()
    pr.check_index()
    log(f"[put-ops] dim {dim} stats={pr.stats}")
    pr.close()


def test_put_of_new_keys_only_and_repeated_keys():
    rng = np.random.default_rng(5)
    dim = 16
    pr = Pair(dim, 3000)
    keys = np.repeat(np.arange(1, 500, dtype=np.uint64), 4)
    rng.shuffle(keys)
    pr.upsert(keys, rng.normal(size=(keys.size, dim)).astype(np.float32))   # inserts; last position wins
    pr.upsert(keys[::-1].copy(), rng.normal(size=(keys.size, dim)).astype(np.float32))
    pr.compare_rows()
    pr.check_index()
    pr.close()


@pytest.mark.parametrize("op", ["adagrad", "sgd", "put"])
def test_one_key_in_more_tiles_than_a_partition_holds_uses_the_spill_path(op):
    # every position holds one of two keys, so each tile contributes one item
    # per key: about 3900 items of the same key in one partition, more than a
    # block groups in LDS
    rng = np.random.default_rng(21)
    dim, n = 4, 4_000_000
    pr = Pair(dim, 10)
    keys = np.full(n, 77, dtype=np.uint64)
    keys[::1000] = 78
    rows = rng.normal(0, 0.01, size=(n, dim)).astype(np.float32)
    if op == "adagrad":
        pr.put(keys, rows, 0.01, 1e-8)
    elif op == "sgd":
        pr.put_sgd(keys, rows, 0.1)
    else:
        pr.upsert(keys, rows)
    pr.compare_rows()
    log(f"[spill] {op} stats={pr.stats}")
    pr.close()


def test_full_size_dlrm_sgd_and_put():
    wl = W.make("dlrm", scale=1.0)
    pr = Pair(wl.dim, wl.capacity)
    pr.prefill(wl.prefill_keys())
    rng = np.random.default_rng(3)
    keys = wl.keys(0)
    pr.put_sgd(keys, wl.grads(0), 0.05)
    rows = np.unique(pr.ora.lookup_rows(keys))
    pr.compare_rows(rows)
    keys = wl.keys(1)
    pr.upsert(keys, rng.normal(0, 0.01, size=(keys.size, wl.dim)).astype(np.float32))
    pr.get(keys)
    log(f"[full] dlrm sgd+put stats={pr.stats}")
    pr.close()


@pytest.mark.parametrize("dim,bound", [(4, None), (64, None), (130, None), (16, 1)])
def test_upsert_of_present_keys_takes_the_last_position_across_tiles(dim, bound):
    # a put whose partitions hold no key new in the call writes each row from
    # its key's last position without grouping; a call with a few new keys
    # mixes such partitions with grouped ones. Zipf repeats put one key in
    # many tiles, so the last position is found across tiles.
    rng = np.random.default_rng(dim + 7)
    nkeys, n = 40_000, 300_000
    pr = Pair(dim, 60_000, staleness_bound=bound)
    universe = np.arange(1, nkeys + 1, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    pr.prefill(np.sort(universe))
    ranks = np.minimum(rng.zipf(1.1, size=n), nkeys) - 1
    keys = universe[ranks]
    if bound is not None:
        pr.get_bounded(keys)
        assert pr.compare_staleness().any()
    pr.upsert(keys, rng.normal(0, 1, size=(n, dim)).astype(np.float32))
    if bound is not None:
        assert not pr.compare_staleness().any()  # the put lowered the counts the get raised
    keys = keys.copy()
    keys[rng.choice(n, size=64, replace=False)] = np.arange(10**6, 10**6 + 64, dtype=np.uint64)
    pr.upsert(keys, rng.normal(0, 1, size=(n, dim)).astype(np.float32))
    pr.compare_rows()
    pr.check_index()
    log(f"[upsert] dim {dim} bound {bound} size {pr.ora.size}")
    pr.close()
