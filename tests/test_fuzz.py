"""Random call sequences on the GPU and the CPU oracle side by side.

Each sequence draws a row width, a capacity, optionally a staleness bound
or (tiered tables) an HBM cache of 2-20 % of the rows, the dedup of its puts
(hash partition, or radix sort), and 30 calls, each one of: get (with or without an output), lookahead, put_grad,
put_grad_sgd, put (upsert), a get whose new keys overflow the capacity, or a
call holding the reserved key; some sequences also draw mlkv_get_put_grad
calls (a get with a put_grad of keys already in the table). Batch lengths cover the tile boundaries
(1, 63..65, 255..257, 1023..1025) and random lengths; keys mix present keys,
duplicates and new keys. After every call: the return codes agree (failures
leave both tables unchanged), sizes agree, key -> row of the call's keys is
bit-exact, and the call's rows agree (bit-exact until updated, then within
1e-5 row-scaled); at the end every row, accumulator, staleness count and the
index invariants.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2504_01506_amd import mlkv
from _harness import Pair, dev, dev_keys, log

pytestmark = pytest.mark.gpu

LENGTHS = [1, 63, 64, 65, 255, 256, 257, 1023, 1024, 1025]
MULT = np.uint64(0x9E3779B97F4A7C15)


def _to_keys(ids):
    k = np.asarray(ids, dtype=np.uint64) * MULT
    k[k == np.uint64(mlkv.MLKV_RESERVED_KEY)] = np.uint64(5)
    return k


def _raw_get(pr, keys, out=None):
    k = dev_keys(keys)
    if pr.gpu.staleness_bound is None:
        return mlkv.mlkv_get(pr.gpu.h, k, keys.size, out)
    blocked = torch.empty(keys.size, dtype=torch.uint8, device="cuda")
    return mlkv.mlkv_get_bounded(pr.gpu.h, k, keys.size, out, blocked)


def _ora_get(pr, keys):
    if pr.ora.staleness_bound is None:
        return pr.ora.get(keys)[0]
    return pr.ora.get_bounded(keys)[0]


def _sequence(seed, tiered, dedup="hash", pipe=False):
    rng = np.random.default_rng(5000 + seed + (1000 if tiered else 0) + (2000 if dedup != "hash" else 0)
                                + (3000 if pipe else 0))
    dim = int(rng.choice([1, 2, 4, 5, 8, 16, 31, 64, 128]))
    cap = int(rng.integers(3000, 40000))
    bound = int(rng.integers(0, 3)) if seed % 3 == 2 and not tiered else None
    cache = max(1, int(cap * rng.uniform(0.02, 0.2))) if tiered else None
    pr = Pair(dim, cap, staleness_bound=bound, cache_rows=cache, dedup=dedup)
    space = int(rng.choice([cap // 8, cap // 2, 4 * cap]))  # many repeats .. mostly new keys
    counts = {}
    for step in range(30):
        op = str(rng.choice(["get", "get", "get_null", "lookahead", "put_grad", "put_grad", "put_sgd", "put",
                             "over", "bad"] + (["pipe", "pipe", "pipe"] if pipe else [])))
        n = int(rng.choice(LENGTHS)) if rng.random() < 0.6 else int(rng.integers(1, 20000))
        if tiered and op == "lookahead":  # large enough to fill the cache and evict
            n = int(rng.integers(max(1, cache // 2), min(20000, 3 * cache) + 1))
        size = pr.ora.size
        if op == "over":
            # more new keys than the table has room for (ids beyond the space)
            room = cap - size
            ids = np.arange(space + 10 * step * cap, space + 10 * step * cap + room + 1 + int(rng.integers(0, 50)))
            keys = _to_keys(ids)
            rc_o = _ora_get(pr, keys)
            assert rc_o == O.EFULL
            assert _raw_get(pr, keys) == mlkv.MLKV_OK
            assert pr.gpu.sync() == mlkv.MLKV_EFULL
            assert pr.gpu.size == size
            counts[op] = counts.get(op, 0) + 1
            continue
        ids = rng.integers(0, space, size=n)
        keys = _to_keys(ids)
        if op == "bad":
            keys[int(rng.integers(0, n))] = np.uint64(mlkv.MLKV_RESERVED_KEY)
            assert _ora_get(pr, keys) == O.EINVAL
            assert _raw_get(pr, keys) == mlkv.MLKV_OK
            assert pr.gpu.sync() == mlkv.MLKV_EINVAL
            g = torch.zeros((n, dim), device="cuda")
            assert mlkv.mlkv_put_grad(pr.gpu.h, dev_keys(keys), g, n, 0.1, 0.0) == mlkv.MLKV_OK
            assert pr.gpu.sync() == mlkv.MLKV_EINVAL
            assert pr.gpu.size == size
            counts[op] = counts.get(op, 0) + 1
            continue
        new = np.setdiff1d(np.unique(keys), pr.ora.row_keys(np.arange(size, dtype=np.int64)) if size else [])
        if size + new.size > cap:
            continue  # drawn batch would not fit: the "over" case covers that
        if op == "get":
            if bound is None:
                pr.get(keys)
            else:
                pr.get_bounded(keys)
        elif op == "lookahead":
            pr.lookahead(keys)
        elif op == "get_null":
            assert _raw_get(pr, keys) == mlkv.MLKV_OK
            assert _ora_get(pr, keys) == O.OK
            assert pr.gpu.sync() == mlkv.MLKV_OK
        elif op == "put_grad":
            pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
        elif op == "pipe":
            if size == 0:
                continue
            m = int(rng.choice(LENGTHS)) if rng.random() < 0.5 else int(rng.integers(1, 20000))
            put_keys = pr.ora.row_keys(rng.integers(0, size, size=m).astype(np.int64))
            pr.get_put_grad(keys, put_keys, rng.normal(0, 0.01, size=(m, dim)).astype(np.float32), 0.01, 1e-8)
            pr.compare_rows(np.unique(pr.ora.lookup_rows(put_keys)))
        elif op == "put_sgd":
            pr.put_sgd(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.05)
        else:
            pr.upsert(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32))
        counts[op] = counts.get(op, 0) + 1
        assert pr.gpu.size == pr.ora.size
        pr.compare_rows(np.unique(pr.ora.lookup_rows(keys)))
    pr.compare_rows()
    pr.check_index()
    if bound is not None:
        pr.compare_staleness()
    cs = pr.gpu.cache_stats() if tiered else None
    if tiered:
        assert cs["loaded"] == cs["filled"] + cs["evicted"] and cs["filled"] <= cache
        assert cs["loaded"] > 0 or counts.get("lookahead", 0) == 0, "lookaheads bring rows into the cache"
    log(f"[fuzz] seed {seed}: dim {dim} cap {cap} bound {bound} cache {cache} dedup {dedup} space {space} size {pr.ora.size} "
        f"calls {counts} stats={pr.stats} cache_stats={cs}")
    pr.close()


@pytest.mark.parametrize("seed", range(24))
def test_random_call_sequences(seed):
    _sequence(seed, tiered=False)


@pytest.mark.parametrize("seed", range(8))
def test_random_call_sequences_on_tiered_tables(seed):
    _sequence(seed, tiered=True)


@pytest.mark.parametrize("seed", range(6))
def test_random_call_sequences_with_radix_dedup(seed):
    _sequence(seed, tiered=seed % 2 == 1, dedup="radix")


@pytest.mark.parametrize("seed", range(9))
def test_random_call_sequences_with_pipelined_calls(seed):
    _sequence(seed, tiered=seed % 3 == 1, pipe=True)
