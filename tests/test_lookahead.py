"""Lookahead with the table in HBM (insert ahead of the gets, no output, no
staleness count) on the GPU against the CPU oracle.

Bar: key -> row and size bit-exact after every call; rows of keys inserted
ahead equal their initial values bit for bit when read by a later get;
staleness counts unchanged by a lookahead; failures leave the table as it was.
"""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv
from _harness import Pair, dev_keys, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("bound", [None, 0])
@pytest.mark.parametrize("m,dim", [(1, 16), (700, 1), (700, 1024), (20_000, 16), (300_000, 16), (300_000, 7)])
def test_lookahead_then_steps(bound, m, dim):
    # m keys looked ahead (few, one block's worth, key ranges), then gets and
    # puts that find them present
    rng = np.random.default_rng(m + dim + (0 if bound is None else 1))
    pr = Pair(dim, 2 * m + 10_000, staleness_bound=bound)
    keys = rng.choice(np.uint64(1) << np.uint64(50), size=m, replace=False).astype(np.uint64)
    batch = np.concatenate([keys, keys[: m // 3]])
    rng.shuffle(batch)
    pr.lookahead(batch)
    if bound is not None:
        assert not pr.compare_staleness().any()
    pr.lookahead(batch[: m // 2 + 1])   # all present: nothing changes
    for s in range(2):
        k = batch[rng.integers(0, batch.size, size=min(batch.size, 5000))]
        if bound is None:
            pr.get(k)
        else:
            assert not pr.get_bounded(k).any()
        pr.put(k, rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32), 0.01, 1e-8)
    pr.compare_rows()
    pr.check_index()
    if bound is not None:
        pr.compare_staleness()
    log(f"[lookahead] m {m} bound {bound}: size {pr.ora.size} stats={pr.stats}")
    pr.close()


@pytest.mark.parametrize("kind", ["plain", "bounded", "tiered"])
def test_get_after_lookahead_takes_recorded_rows(kind):
    # a get right after a lookahead takes, at each position holding the key
    # the lookahead found present there, the row it recorded, and probes the
    # others: same keys at the same positions, other present keys, new keys,
    # keys moved to other positions, a batch longer than the lookahead's
    dim, m = 16, 40_000
    rng = np.random.default_rng({"plain": 1, "bounded": 2, "tiered": 3}[kind])
    pr = Pair(dim, 4 * m, staleness_bound=0 if kind == "bounded" else None,
              cache_rows=m // 2 if kind == "tiered" else None)
    keys = rng.choice(np.uint64(1) << np.uint64(40), size=2 * m, replace=False).astype(np.uint64)
    present = keys[:m]

    def get(k):
        if kind == "bounded":
            pr.get_bounded(k)
        else:
            pr.get(k)
        grads = rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32)
        pr.put(k, grads, 0.01, 1e-8)   # completes the get (bounded) and updates the rows

    get(present)                                   # all new
    a = present[rng.integers(0, m, size=30_000)]
    pr.lookahead(a)                                # every key present: rows recorded by position
    b = a.copy()
    b[5_000:10_000] = present[rng.integers(0, m, size=5_000)]      # other present keys
    b[10_000:12_000] = keys[m:m + 2_000]                            # new keys
    rng.shuffle(b[20_000:25_000])                                   # same keys, other positions
    get(b)
    pr.lookahead(b[:7_000])
    get(np.concatenate([b[:7_000], keys[m + 2_000:m + 3_000]]))     # longer batch than the lookahead
    pr.compare_rows()
    pr.check_index()
    if kind == "bounded":
        pr.compare_staleness()
    log(f"[lookahead] get after lookahead ({kind}): size {pr.ora.size} stats={pr.stats}")
    pr.close()


def test_failed_lookahead_leaves_the_table_unchanged():
    pr = Pair(4, 100, staleness_bound=1)
    pr.get_bounded(np.arange(1, 51, dtype=np.uint64))
    before = pr.compare_staleness()
    k = dev_keys(np.arange(1000, 1100, dtype=np.uint64))       # 100 new keys, 50 fit
    assert mlkv.mlkv_lookahead(pr.gpu.h, k, 100) == mlkv.MLKV_OK
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    bad = np.array([3, 7, mlkv.MLKV_RESERVED_KEY], np.uint64)
    assert mlkv.mlkv_lookahead(pr.gpu.h, dev_keys(bad), 3) == mlkv.MLKV_OK
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    assert pr.gpu.size == 50
    assert np.array_equal(pr.compare_staleness(), before)
    pr.check_index()
    pr.close()
