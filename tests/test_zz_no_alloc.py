"""mlkv_get_noalloc (the get that allocates nothing, its scratch in a fixed
device array) against mlkv_get on a twin table: two calls in a row, the
second smaller, then again after a put_grad on both tables; bit-exact
output rows, key -> row and size; the same on tiered twin tables, with rows
cached, at home and evicted. Larger batches are refused."""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv
from _harness import dev, dev_keys, log

pytestmark = pytest.mark.gpu


def get_both(a, b, keys, dim):
    k = dev_keys(keys)
    out_a = torch.full((keys.size, dim), -1.0, device="cuda")
    out_b = torch.full((keys.size, dim), -2.0, device="cuda")
    assert mlkv.mlkv_get(a.h, k, keys.size, out_a) == mlkv.MLKV_OK
    assert mlkv.mlkv_get_noalloc(b.h, k, keys.size, out_b) == mlkv.MLKV_OK
    assert a.sync() == mlkv.MLKV_OK and b.sync() == mlkv.MLKV_OK
    assert torch.equal(out_a.view(torch.int32), out_b.view(torch.int32)), "rows differ"
    assert a.size == b.size
    assert torch.equal(a.lookup_rows(k), b.lookup_rows(k)), "key -> row differs"


@pytest.mark.parametrize("dim", [16, 64])
def test_noalloc_get_matches_get_on_consecutive_calls(dim):
    rng = np.random.default_rng(dim)
    a = mlkv.Table(dim, 200_000)
    b = mlkv.Table(dim, 200_000)
    first = rng.integers(0, 120_000, size=mlkv.MLKV_NOALLOC_MAX_KEYS).astype(np.uint64) * np.uint64(7919)
    second = np.concatenate([first[:2000], rng.integers(10**9, 10**9 + 5000, size=1500).astype(np.uint64)])
    get_both(a, b, first, dim)          # the largest batch: every key new
    get_both(a, b, second, dim)         # smaller, old and new keys mixed
    g = torch.from_numpy(rng.normal(0, 0.01, size=(second.size, dim)).astype(np.float32)).cuda()
    for t in (a, b):
        t.put_grad(dev_keys(second), g, 0.01, 1e-8)
        assert t.sync() == mlkv.MLKV_OK
    get_both(a, b, second[::-1].copy(), dim)  # updated rows read back through both
    log(f"[noalloc] dim {dim}: size {a.size}")
    a.close()
    b.close()


def test_noalloc_get_on_tiered_tables():
    """Rows cached in HBM, at home in host memory, and evicted by a later
    lookahead are read alike through both gets."""
    dim, cap, cache = 32, 60_000, 3_000
    rng = np.random.default_rng(11)
    a = mlkv.Table(dim, cap, cache_rows=cache)
    b = mlkv.Table(dim, cap, cache_rows=cache)
    keys = rng.integers(0, 40_000, size=20_000).astype(np.uint64) * np.uint64(104729)
    get_both(a, b, keys, dim)                      # inserts; rows at home
    for t in (a, b):
        t.lookahead(dev_keys(keys[:5_000]))        # part of the batch cached
        assert t.sync() == mlkv.MLKV_OK
    g = torch.from_numpy(rng.normal(0, 0.01, size=(keys.size, dim)).astype(np.float32)).cuda()
    for t in (a, b):
        t.put_grad(dev_keys(keys), g, 0.01, 1e-8)  # cached and home rows updated
        assert t.sync() == mlkv.MLKV_OK
    get_both(a, b, keys[::-1].copy(), dim)
    for t in (a, b):
        t.lookahead(dev_keys(keys[10_000:16_000]))  # evicts the first cached rows, writing them back
        assert t.sync() == mlkv.MLKV_OK
    get_both(a, b, keys[:12_000].copy(), dim)
    # which rows stay at home when a lookahead asks for more than the free
    # slots depends on the order the misses are listed in: the counters of the
    # twins may differ, each table's must add up
    for t in (a, b):
        st = t.cache_stats()
        log(f"[noalloc] tiered: {st}")
        assert st["evicted"] > 0 and st["written_back"] > 0, "the second lookahead evicts dirty rows"
        assert st["loaded"] == st["filled"] + st["evicted"] and st["filled"] == cache
    a.close()
    b.close()


def test_noalloc_get_refuses_larger_batches_and_bounded_tables():
    t = mlkv.Table(8, 100_000)
    k = torch.zeros(mlkv.MLKV_NOALLOC_MAX_KEYS + 1, dtype=torch.int64, device="cuda")
    assert mlkv.mlkv_get_noalloc(t.h, k, k.numel(), None) == mlkv.MLKV_EINVAL
    assert "65536" in mlkv.last_error()
    assert t.sync() == mlkv.MLKV_OK and t.size == 0
    t.close()
    tb = mlkv.Table(8, 100, staleness_bound=0)
    assert mlkv.mlkv_get_noalloc(tb.h, k, 4, None) == mlkv.MLKV_EINVAL
    tb.close()
