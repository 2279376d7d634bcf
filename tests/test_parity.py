"""GPU get / put_grad against the CPU oracle, element by element.

Bar: key -> row and rows never updated are bit-exact; updated rows and the
Adagrad accumulators are within 1e-5 relative (row-scaled for row elements).
"""
import numpy as np
import pytest
import torch

from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, dev, dev_keys, log, record

pytestmark = pytest.mark.gpu


def run_config(name, scale, steps, full_check_every=1):
    wl = W.make(name, scale=scale, steps=steps)
    log(f"[parity] {name} scale={scale} n={wl.n} dim={wl.dim} cap={wl.capacity}")
    pr = Pair(wl.dim, wl.capacity)
    pre = wl.prefill_keys()
    if pre.size:
        pr.prefill(pre)
    for s in range(steps):
        keys = wl.keys(s)
        pr.get(keys)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
        if (s + 1) % full_check_every == 0 or s == steps - 1:
            pr.compare_rows()
        log(f"[parity] {name} step {s} ok size={pr.ora.size} stats={pr.stats}")
    pr.check_index()
    record(f"{name}@{scale}x{steps}", pr.stats)
    pr.close()
    return pr.stats


def test_tiny_full_config():
    st = run_config("tiny", 1.0, 10)
    assert st["max_err"] <= 1e-5


@pytest.mark.parametrize("name", ["dlrm", "kg", "gnn", "large"])
def test_scaled_configs(name):
    run_config(name, 0.01, 3)


@pytest.mark.parametrize("dim", [1, 3, 4, 7, 16, 33, 64, 100, 128, 400, 1024])
def test_dims_and_ragged_batches(dim):
    rng = np.random.default_rng(dim)
    pr = Pair(dim, 5000)
    for n in (1, 255, 257, 1023, 1025, 3001):
        keys = rng.integers(0, 3000, size=n).astype(np.uint64) * np.uint64(2654435761)
        pr.get(keys)
        g = rng.normal(0, 0.01, size=(n, dim)).astype(np.float32)
        pr.put(keys, g, 0.01, 1e-8)
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_misaligned_output_and_grads_use_the_scalar_path():
    rng = np.random.default_rng(11)
    dim, n = 16, 700
    pr = Pair(dim, 2000)
    keys = rng.integers(0, 500, size=n).astype(np.uint64)
    k = dev_keys(keys)
    buf = torch.empty(n * dim + 1, dtype=torch.float32, device="cuda")
    out = buf[1:].view(n, dim)                     # 4-byte aligned, not 16
    pr.gpu.get(k, out)
    rc, want = pr.ora.get(keys)
    assert pr.gpu.sync() == 0
    assert np.array_equal(out.cpu().numpy().view(np.uint32), want.view(np.uint32))
    g = rng.normal(0, 0.01, size=(n, dim)).astype(np.float32)
    gbuf = torch.empty(n * dim + 1, dtype=torch.float32, device="cuda")
    gbuf[1:] = dev(g.reshape(-1))
    pr.gpu.put_grad(k, gbuf[1:], 0.01, 1e-8)
    pr.ora.put_grad(keys, g, 0.01, 1e-8)
    assert pr.gpu.sync() == 0
    pr.updated[pr.ora.lookup_rows(keys)] = True
    pr.compare_rows()
    pr.close()


def test_one_hot_key_spills_beyond_lds():
    # every position holds the same key: one segment far longer than a block's
    # LDS share, split over the block and sorted in the global spill area
    rng = np.random.default_rng(12)
    dim = 64
    pr = Pair(dim, 100)
    for n in (5000, 40000):
        keys = np.full(n, 77, dtype=np.uint64)
        keys[::997] = 78
        pr.get(keys)
        pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, 1e-8)
    pr.compare_rows()
    pr.close()


def test_put_inserts_unseen_keys_then_updates_them():
    rng = np.random.default_rng(13)
    dim = 32
    pr = Pair(dim, 1000)
    keys = rng.integers(0, 400, size=900).astype(np.uint64)
    pr.put(keys, rng.normal(0, 0.01, size=(900, dim)).astype(np.float32), 0.05, 1e-8)
    pr.compare_rows()
    pr.check_index()
    pr.get(keys)
    pr.close()


# direct ranking up to 768 new keys x chunks of 256 get tiles: 768 for a
# batch of up to 65,536 keys, 192 for 213k keys (832 tiles)
@pytest.mark.parametrize("n_new,n", [(1, 213_000), (192, 213_000), (193, 213_000), (768, 768), (769, 769),
                                     (1000, 1000), (4096, 213_000), (8193, 8193), (20_000, 300_000)])
def test_new_keys_just_past_the_direct_ranking(n_new, n):
    """Calls on either side of the limit of the direct ranking,
    few blocks or many blocks each with a small key range (one local
    sub-range, or none: fewer new keys than samples), hits mixed in."""
    rng = np.random.default_rng(n_new + n)
    dim = 3
    pr = Pair(dim, n + n_new + 10)
    old = rng.choice(np.uint64(1) << np.uint64(62), size=max(1, n - n_new), replace=False).astype(np.uint64)
    if n > n_new:
        pr.get(np.sort(old))
    new = rng.choice(np.uint64(1) << np.uint64(62), size=n_new, replace=False).astype(np.uint64) | (np.uint64(1) << np.uint64(62))
    keys = np.concatenate([new, old[: n - n_new]]) if n > n_new else new
    keys = keys[rng.permutation(keys.size)]
    pr.get(keys)
    pr.compare_rows()
    pr.check_index()
    pr.close()


@pytest.mark.parametrize("case", ["random", "descending", "second_half_new", "clustered", "one_feature"])
def test_many_new_keys_get_rows_in_key_order(case):
    """A call inserting many more new keys than one block ranks against all
    others (key ranges split among the blocks): rows follow the ascending
    order of the call's new keys, whatever their batch order or spread."""
    rng = np.random.default_rng(21)
    dim, n = 5, 120_000
    pr = Pair(dim, 400_000)
    keys = rng.choice(np.uint64(1) << np.uint64(62), size=n, replace=False).astype(np.uint64)
    if case == "descending":
        keys = np.sort(keys)[::-1].copy()
    elif case == "second_half_new":  # the first half of the batch are hits
        pr.get(np.sort(keys[: n // 2]))
    elif case == "clustered":  # a dense run of small keys and a few huge ones
        keys = np.concatenate([np.arange(1, n - 100, dtype=np.uint64) * np.uint64(3),
                               (np.uint64(1) << np.uint64(63)) + np.arange(100, dtype=np.uint64)])
        keys = keys[rng.permutation(keys.size)]
    elif case == "one_feature":  # feature << 40 | id, ids dense and small, repeated positions
        ids = rng.integers(0, 90_000, size=n).astype(np.uint64)
        keys = (np.uint64(7) << np.uint64(40)) | ids
    pr.get(keys)
    log(f"[parity] many new keys ({case}): size={pr.gpu.size}")
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_millions_of_new_keys_in_one_get():
    """Key ranges holding more keys than LDS: gathered in global scratch."""
    rng = np.random.default_rng(22)
    n = 2_600_000
    pr = Pair(2, n + 10)
    keys = rng.choice(np.uint64(1) << np.uint64(40), size=n, replace=False).astype(np.uint64)
    k = dev_keys(keys)
    pr.gpu.get(k, None)
    rc, _ = pr.ora.get(keys)
    assert rc == 0 and pr.gpu.sync() == mlkv.MLKV_OK
    got = pr.gpu.lookup_rows(k).cpu().numpy()
    assert np.array_equal(got, np.argsort(np.argsort(keys)))
    pr.compare_rows(np.arange(0, n, 997, dtype=np.int64))
    pr.close()


def test_many_new_keys_over_capacity_roll_back():
    dim = 3
    pr = Pair(dim, 30_000)
    pr.get(np.arange(1000, dtype=np.uint64))
    k = dev_keys(np.arange(10_000, 50_000, dtype=np.uint64))
    pr.gpu.get(k, None)
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    assert pr.gpu.size == 1000
    pr.check_index()
    pr.get(np.arange(10_000, 35_000, dtype=np.uint64))  # 25,000 new keys fit
    assert pr.gpu.size == 26_000
    pr.compare_rows()
    pr.check_index()
    pr.close()


@pytest.mark.parametrize("name", ["kv-uniform", "kv-zipf"])
def test_key_value_mix(name):
    """The 50/50 get/put mix: gets of half a batch, then puts of values for
    the other half, over prefilled records."""
    wl = W.make(name, scale=0.01)
    pr = Pair(wl.dim, wl.capacity)
    pr.prefill(wl.prefill_keys())
    h = wl.n // 2
    for s in range(3):
        k = wl.keys(s)
        pr.get(k[:h])
        pr.upsert(k[h:], wl.values(s))
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_hot_keys_across_many_tiles():
    """Keys present in hundreds of put tiles (more than 256 tiles, up to the
    1024 a tile bitmask covers), whose items are put in tile order through
    the mask, and some beyond that."""
    rng = np.random.default_rng(41)
    dim = 8
    for n in (600_000, 1_300_000):
        pr = Pair(dim, 200_000)
        hot = rng.integers(1, 2**62, size=40, dtype=np.uint64)
        cold = rng.integers(1, 2**62, size=100_000, dtype=np.uint64)
        keys = np.where(rng.random(n) < 0.3, hot[rng.integers(0, hot.size, n)], cold[rng.integers(0, cold.size, n)])
        g = rng.normal(0, 0.01, size=(n, dim)).astype(np.float32)
        pr.put(keys, g, 0.05, 1e-8)
        for ks in (hot, cold[:2000]):
            r = pr.ora.lookup_rows(ks)
            pr.compare_rows(np.unique(r[r >= 0]))
        pr.close()


def test_empty_call_is_a_no_op():
    pr = Pair(8, 10)
    k = torch.empty(0, dtype=torch.int64, device="cuda")
    pr.gpu.get(k, None)
    pr.gpu.put_grad(k, torch.empty(0, device="cuda"), 0.1, 0.0)
    assert pr.gpu.sync() == 0 and pr.gpu.size == 0
    pr.close()


def test_capacity_overflow_fails_the_whole_call():
    rng = np.random.default_rng(14)
    dim = 8
    pr = Pair(dim, 100)
    first = np.arange(90, dtype=np.uint64) * np.uint64(3)
    pr.get(first)
    _, _, sk0, sr0 = pr.gpu.export(0)
    w0, st0, _, _ = pr.gpu.export()
    over = np.arange(1000, 1020, dtype=np.uint64)       # 20 new keys, only 10 fit
    out = torch.empty((20, dim), device="cuda")
    pr.gpu.get(dev_keys(over), out)
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    assert pr.gpu.sync() == mlkv.MLKV_OK                 # cleared once reported
    g = torch.zeros((20, dim), device="cuda")
    pr.gpu.put_grad(dev_keys(over), g, 0.1, 0.0)
    assert pr.gpu.sync() == mlkv.MLKV_EFULL
    assert pr.gpu.size == 90
    _, _, sk1, sr1 = pr.gpu.export(0)
    w1, st1, _, _ = pr.gpu.export()
    assert torch.equal(sk0, sk1) and torch.equal(sr0, sr1)
    assert torch.equal(w0, w1) and torch.equal(st0, st1)
    # exactly filling the table is fine
    pr.get(np.arange(2000, 2010, dtype=np.uint64))
    assert pr.gpu.size == 100
    pr.check_index()
    pr.close()


def test_reserved_key_fails_the_whole_call():
    dim = 4
    pr = Pair(dim, 50)
    pr.get(np.arange(10, dtype=np.uint64))
    bad = np.array([3, 20, mlkv.MLKV_RESERVED_KEY, 21], dtype=np.uint64)
    out = torch.empty((4, dim), device="cuda")
    pr.gpu.get(dev_keys(bad), out)
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    pr.gpu.put_grad(dev_keys(bad), torch.ones((4, dim), device="cuda"), 0.1, 0.0)
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    assert pr.gpu.size == 10
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_host_rejects_bad_arguments():
    t = mlkv.Table(8, 10)
    k = torch.zeros(4, dtype=torch.int64, device="cuda")
    g = torch.zeros((4, 8), device="cuda")
    assert mlkv.mlkv_put_grad(t.h, k, g, 4, float("nan"), 0.0) == mlkv.MLKV_EINVAL
    assert mlkv.mlkv_put_grad(t.h, k, g, 4, 0.1, -1.0) == mlkv.MLKV_EINVAL
    assert mlkv.mlkv_get(t.h, k, -1, None) == mlkv.MLKV_EINVAL
    assert mlkv.mlkv_get(t.h, None, 4, None) == mlkv.MLKV_EINVAL
    assert t.sync() == 0 and t.size == 0
    t.close()


def test_deterministic_across_runs():
    wl = W.make("dlrm", scale=0.005, steps=2)
    res = []
    for _ in range(2):
        t = mlkv.Table(wl.dim, wl.capacity)
        pre = wl.prefill_keys()
        t.get(dev_keys(pre), None)
        outs = []
        for s in range(2):
            k = dev_keys(wl.keys(s))
            out = torch.empty((k.numel(), wl.dim), device="cuda")
            t.get(k, out)
            t.put_grad(k, dev(wl.grads(s)), wl.lr, wl.eps)
            outs.append(out.clone())
        assert t.sync() == 0
        res.append((outs, t.export()))
        t.close()
    (o1, e1), (o2, e2) = res
    for a, b in zip(o1, o2):
        assert torch.equal(a, b)
    assert torch.equal(e1[0], e2[0]) and torch.equal(e1[1], e2[1])   # rows, accumulators
    # which slot of a bucket a key lands in may depend on CAS races; the
    # key -> row map may not
    def pairs(sk, sr):
        used = sk != -1
        k, r = sk[used].cpu().numpy(), sr[used].cpu().numpy()
        o = np.argsort(k)
        return k[o], r[o]
    k1, r1 = pairs(e1[2], e1[3])
    k2, r2 = pairs(e2[2], e2[3])
    assert np.array_equal(k1, k2) and np.array_equal(r1, r2)


def test_get_output_equals_exported_rows():
    wl = W.make("kg", scale=0.002, steps=2)
    t = mlkv.Table(wl.dim, wl.capacity)
    t.get(dev_keys(wl.prefill_keys()), None)
    k = dev_keys(wl.keys(0))
    t.put_grad(k, dev(wl.grads(0)), wl.lr, wl.eps)
    out = torch.empty((k.numel(), wl.dim), device="cuda")
    t.get(k, out)
    rows = t.lookup_rows(k)
    w, _, _, _ = t.export()
    assert t.sync() == 0
    assert torch.equal(out, w[rows])
    t.close()


def test_put_after_get_with_shuffled_and_replaced_positions():
    """A put reuses the rows its preceding get found, position by position,
    only where the key is the same: positions holding another present key, a
    new key, or a key the get inserted must be probed."""
    rng = np.random.default_rng(31)
    dim = 8
    pr = Pair(dim, 50_000)
    pr.get(np.arange(1, 20_001, dtype=np.uint64) * np.uint64(7919))
    keys = rng.integers(1, 20_001, size=30_000).astype(np.uint64) * np.uint64(7919)
    keys[::7] = np.arange(100_000, 100_000 + keys[::7].size, dtype=np.uint64)  # new in the get
    pr.get(keys)
    later = keys.copy()
    later[1::3] = rng.integers(1, 20_001, size=later[1::3].size).astype(np.uint64) * np.uint64(7919)
    later[2::11] = np.arange(500_000, 500_000 + later[2::11].size, dtype=np.uint64)  # new in the put
    pr.put(later, rng.normal(0, 0.01, size=(later.size, dim)).astype(np.float32), 0.01, 1e-8)
    pr.put(later[::-1].copy(), rng.normal(0, 0.01, size=(later.size, dim)).astype(np.float32), 0.01, 1e-8)
    pr.compare_rows()
    pr.check_index()
    pr.close()
