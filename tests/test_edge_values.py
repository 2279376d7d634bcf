"""GPU against the oracle on edge values of the update and on non-default
table configurations.

* The dim-1 grid of tests/test_division.py (the oracle pinned there to
  exact arithmetic): den = 0, subnormal denominators and gradients, squares
  that overflow; the GPU rows and accumulators must equal the oracle's bit
  for bit (NaN on both sides counts as equal).
* eps = 0 with gradients whose mean square underflows (rows become
  infinities) and a subnormal eps with all-zero gradients (rows unchanged),
  at dim 64 with repeated keys.
* Tables opened with a seed other than the default and max load 0.9 / 0.5:
  the seed enters every initial row, the load the index layout.
* A probe chain longer than the index allows (keys crafted to share one home
  bucket): the call fails as a whole with MLKV_EFULL.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2504_01506_amd import mlkv, workloads as W
from _harness import Pair, dev, dev_keys, log, record
from test_division import EPS, GRADS

pytestmark = pytest.mark.gpu


def bits_equal_nan_aware(a: np.ndarray, b: np.ndarray) -> bool:
    both_nan = np.isnan(a) & np.isnan(b)
    return bool(np.all(both_nan | (a.view(np.uint32) == b.view(np.uint32))))


@pytest.mark.parametrize("eps", EPS)
def test_edge_value_grid_bit_exact(eps):
    g1 = np.array(GRADS, dtype=np.float32).reshape(-1, 1)
    g2 = np.array(GRADS[::-1], dtype=np.float32).reshape(-1, 1)
    n = g1.shape[0]
    keys = np.arange(1, n + 1, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    pr = Pair(1, 64)
    pr.get(keys)
    for g in (g1, g2):
        pr.gpu.put_grad(dev_keys(keys), dev(g), 0.01, eps)
        assert pr.ora.put_grad(keys, g, 0.01, eps) == O.OK
        assert pr.gpu.sync() == mlkv.MLKV_OK
        rows = pr.ora.lookup_rows(keys)
        w, st = pr.gpu.read_rows(torch.from_numpy(rows).cuda())
        want_w, want_st = pr.ora.read_rows(rows)
        assert bits_equal_nan_aware(w.cpu().numpy(), want_w), (w.cpu().numpy().ravel(), want_w.ravel())
        assert bits_equal_nan_aware(st.cpu().numpy(), want_st), (st.cpu().numpy(), want_st)
    pr.close()


def test_eps_zero_with_underflowing_gradients_gives_infinite_rows():
    rng = np.random.default_rng(21)
    dim, n = 64, 3000
    pr = Pair(dim, 2000)
    keys = rng.integers(0, 1500, size=n).astype(np.uint64)
    pr.get(keys)
    g = (rng.normal(0, 1, size=(n, dim)) * 1e-23).astype(np.float32)
    g[::7, :5] = 0.0  # some zero columns (0 / 0 where the key's whole column is zero)
    pr.put(keys, g, 0.01, 0.0)
    pr.compare_rows()
    w, _, _, _ = pr.gpu.export()
    assert not np.isfinite(w.cpu().numpy()).all(), "expected infinite rows from den = 0"
    log(f"[edge] eps=0 underflow ok, stats={pr.stats}")
    pr.close()


def test_subnormal_eps_with_zero_gradients_leaves_rows_unchanged():
    rng = np.random.default_rng(22)
    dim, n = 64, 2000
    pr = Pair(dim, 1500)
    keys = rng.integers(0, 1000, size=n).astype(np.uint64)
    pr.get(keys)
    w0, _, _, _ = pr.gpu.export()
    pr.put(keys, np.zeros((n, dim), dtype=np.float32), 0.01, 1e-40)
    pr.compare_rows()
    w1, st1, _, _ = pr.gpu.export()
    assert torch.equal(w0.view(torch.int32), w1.view(torch.int32))
    assert torch.all(st1 == 0)
    # then ordinary gradients with the same subnormal eps, and with eps = 0
    for eps in (1e-40, 0.0):
        pr.put(keys, rng.normal(0, 0.01, size=(n, dim)).astype(np.float32), 0.01, eps)
    pr.compare_rows()
    pr.close()


def test_huge_and_subnormal_gradients_with_duplicates():
    rng = np.random.default_rng(23)
    dim, n = 16, 4000
    pr = Pair(dim, 1000)
    keys = rng.integers(0, 600, size=n).astype(np.uint64)
    pr.get(keys)
    scale = rng.choice(np.array([1e-41, 1e-30, 1.0, 1e18, 3e30]), size=(n, 1))
    g = (rng.normal(0, 1, size=(n, dim)) * scale).astype(np.float32)
    pr.put(keys, g, 0.01, 1e-8)
    pr.compare_rows()
    pr.close()


@pytest.mark.parametrize("seed,max_load", [(1, 0.9), (0xDEADBEEFCAFEF00D, 0.5)])
@pytest.mark.parametrize("name,scale,steps", [("tiny", 1.0, 4), ("dlrm", 0.01, 3), ("kg", 0.002, 3)])
def test_configs_with_other_seed_and_load(name, scale, steps, seed, max_load):
    wl = W.make(name, scale=scale, steps=steps)
    pr = Pair(wl.dim, wl.capacity, seed=seed, max_load=max_load)
    pre = wl.prefill_keys()
    if pre.size:
        pr.prefill(pre)
    for s in range(steps):
        keys = wl.keys(s)
        pr.get(keys)
        pr.put(keys, wl.grads(s), wl.lr, wl.eps)
    pr.compare_rows()
    pr.check_index()
    # the seed must matter: a row of the default seed differs
    k = np.array([wl.keys(0)[0]], dtype=np.uint64)
    d = O.OracleTable(wl.dim, 8)
    _, w_default = d.get(k)
    d.close()
    _, w_seeded = pr.ora.get(k)
    assert not np.array_equal(w_default, w_seeded)
    record(f"{name}@{scale}x{steps} seed={seed:#x} load={max_load}", pr.stats)
    pr.close()


# ---- a probe chain longer than the index allows -----------------------------
M64 = (1 << 64) - 1
FMIX_C1, FMIX_C2 = 0xFF51AFD7ED558CCD, 0xC4CEB9FE1A85EC53
MAX_PROBE_BUCKETS = 4096  # buckets a probe visits before the call reports overflow


def fmix64_inverse(h: int) -> int:
    """Inverse of the index's 64-bit finaliser (xor-shift 33, multiply, ...):
    the keys whose home bucket the test chooses."""
    x = h ^ (h >> 33)
    x = (x * pow(FMIX_C2, -1, 1 << 64)) & M64
    x ^= x >> 33
    x = (x * pow(FMIX_C1, -1, 1 << 64)) & M64
    return x ^ (x >> 33)


def fmix64(k: int) -> int:
    k ^= k >> 33
    k = (k * FMIX_C1) & M64
    k ^= k >> 33
    k = (k * FMIX_C2) & M64
    return k ^ (k >> 33)


def colliding_keys(count: int, nb_log2: int, bucket: int, rng) -> np.ndarray:
    out = set()
    while len(out) < count:
        low = int(rng.integers(0, 1 << (64 - nb_log2), dtype=np.uint64))
        k = fmix64_inverse((bucket << (64 - nb_log2)) | low)
        if k != M64:
            out.add(k)
    return np.array(sorted(out), dtype=np.uint64)


def test_fmix64_inverse_round_trips():
    rng = np.random.default_rng(5)
    for _ in range(100):
        h = int(rng.integers(0, 1 << 63)) * 2 + 1
        assert fmix64(fmix64_inverse(h)) == h


def test_probe_chain_overflow_fails_the_whole_call():
    rng = np.random.default_rng(24)
    cap = 40000
    t = mlkv.Table(2, cap, max_load=0.9)
    nb_log2 = int(np.log2(t.num_slots // 8))
    assert (1 << nb_log2) > MAX_PROBE_BUCKETS
    keys = colliding_keys(8 * MAX_PROBE_BUCKETS + 1, nb_log2, 5, rng)
    fill, extra = keys[:-1], keys[-1:]
    t.get(dev_keys(fill), None)      # fills the 4096 buckets of the chain exactly
    assert t.sync() == mlkv.MLKV_OK and t.size == fill.size
    _, _, sk0, sr0 = t.export(0)
    t.get(dev_keys(extra), None)     # one more key with the same home bucket
    assert t.sync() == mlkv.MLKV_EFULL
    assert t.size == fill.size
    _, _, sk1, sr1 = t.export(0)
    assert torch.equal(sk0, sk1) and torch.equal(sr0, sr1), "a failed call changed the index"
    g = torch.zeros((1, 2), device="cuda")
    t.put_grad(dev_keys(extra), g, 0.1, 0.0)
    assert t.sync() == mlkv.MLKV_EFULL
    # other keys still insert, and the chain's keys still map to their rows
    other = colliding_keys(1, nb_log2, 6000, rng)  # home bucket outside the chain
    t.get(dev_keys(other), None)
    assert t.sync() == mlkv.MLKV_OK and t.size == fill.size + 1
    rows = t.lookup_rows(dev_keys(fill)).cpu().numpy()
    assert np.array_equal(np.sort(rows), np.arange(fill.size))
    assert np.array_equal(rows, np.arange(fill.size))  # fill was ascending: rows in key order
    t.close()
