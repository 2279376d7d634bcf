"""Row assignment of many new keys by key range, against the CPU oracle.

A get that inserts many keys ranks them by key range: either by ranges a
sample of its own new keys gives, or, when the previous such call left cut
points for as many ranges, by the range lists the probe kernel filled as it
inserted (every new key filed in its range's list). The sequences below
take each way, and the ways out of the lists: another number of ranges, a
range whose list overflows, a call that fails. Bar: key -> row and every
row bit-exact (no put changes a row here), size after every call.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2504_01506_amd import mlkv
from _harness import Pair, dev_keys, log

pytestmark = pytest.mark.gpu

MULT = np.uint64(0x9E3779B97F4A7C15)


def _spread(ids):
    return np.asarray(ids, dtype=np.uint64) * MULT + np.uint64(11)


def _check(pr, keys):
    assert pr.gpu.size == pr.ora.size
    rows = pr.ora.lookup_rows(keys)
    got = pr.gpu.lookup_rows(dev_keys(keys)).cpu().numpy()
    assert np.array_equal(got, rows), "key -> row differs"


@pytest.mark.parametrize("dim", [4, 64])
def test_range_lists_and_their_fallbacks(dim):
    rng = np.random.default_rng(61 + dim)
    cap = 3_000_000
    pr = Pair(dim, cap)
    n = 200_000  # 782 get tiles: 256 ranges
    used = 0

    def fresh(count):
        nonlocal used
        ids = np.arange(used, used + count)
        used += count
        return ids

    # 1: sampled ranges (no cut points yet); 2-3: the same number of ranges,
    # so the lists are filed; keys half new, half present, with repeats
    for step in range(3):
        new_ids = fresh(n // 2)
        old_ids = rng.integers(0, max(used - n // 2, 1), size=n - n // 2)
        keys = _spread(rng.permutation(np.concatenate([new_ids, old_ids])))
        pr.get(keys)
        _check(pr, keys)
    # another batch size: fewer ranges than the cut points are for
    keys = _spread(rng.permutation(fresh(30_000)))
    pr.get(keys)
    _check(pr, keys)
    # back to 256 ranges, twice (the first leaves cut points again)
    for _ in range(2):
        keys = _spread(rng.permutation(fresh(n)))
        pr.get(keys)
        _check(pr, keys)
    # new keys all inside one range of the last cut points: its list overflows
    lo = int(_spread([used])[0])
    crowd = np.uint64(lo) + np.arange(1, 150_001, dtype=np.uint64) * np.uint64(3)
    crowd = crowd[np.isin(crowd, _spread(np.arange(used)), invert=True)]
    pr.get(rng.permutation(crowd))
    _check(pr, crowd)
    # a call over capacity fails and leaves the table alone; the next one lists again
    size = pr.ora.size
    over = _spread(np.arange(10**9, 10**9 + (cap - size) + 5))
    assert pr.ora.get(over)[0] == O.EFULL
    assert mlkv.mlkv_get(pr.gpu.h, dev_keys(over), over.size, None) == mlkv.MLKV_OK
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    assert pr.gpu.size == size
    keys = _spread(rng.permutation(fresh(n)))
    pr.get(keys)
    _check(pr, keys)
    # a lookahead inserts through the same kernels
    keys = _spread(rng.permutation(fresh(n)))
    pr.lookahead(keys)
    pr.compare_rows()
    pr.check_index()
    log(f"[ranges] dim {dim}: size {pr.ora.size}")
    pr.close()
