"""Synthetic workload generators: reproducible, and shaped as stated."""
import numpy as np
import pytest

from paper_2504_01506_amd import workloads as W


def test_zipf_sampler_matches_exact_pmf_small_support():
    rng = np.random.default_rng(0)
    for s in (0.99, 1.05, 1.1, 2.0):
        n = 50
        z = W.ZipfSampler(n, s)
        x = z.sample(rng, 400_000)
        assert x.min() >= 1 and x.max() <= n
        p = np.arange(1, n + 1, dtype=np.float64) ** -s
        p /= p.sum()
        f = np.bincount(x, minlength=n + 1)[1:] / x.size
        # chi-square against the exact finite-support pmf
        chi2 = np.sum((f - p) ** 2 / p) * x.size
        assert chi2 < 100, (s, chi2)   # 49 dof: mean 49, sd ~10


def test_harmonic_sum_head_plus_tail_is_accurate():
    for s in (0.99, 1.1):
        n = 3_000_000
        exact = float(np.sum(np.arange(1, n + 1, dtype=np.float64) ** -s))
        assert abs(W.ZipfSampler.harmonic(n, s) - exact) < 1e-9 * exact


def test_streams_reproduce_from_their_seeds():
    a = W.make("dlrm", scale=0.01)
    b = W.make("dlrm", scale=0.01)
    assert np.array_equal(a.keys(3), b.keys(3))
    assert np.array_equal(a.grads(3), b.grads(3))
    assert not np.array_equal(a.keys(3), a.keys(4))


def test_tiny_shape():
    t = W.make("tiny")
    k = t.keys(0)
    assert k.dtype == np.uint64 and k.size == 4096
    assert not np.any(k == W.EMPTY_KEY)
    ids = np.arange(100_000, dtype=np.uint64)
    assert np.unique(t.id_to_key(ids)).size == ids.size      # bijective key map
    g = t.grads(0)
    assert g.shape == (4096, 16) and g.dtype == np.float32
    assert abs(float(g.std()) - 0.01) < 0.0005


def test_dlrm_shape_full_size_structure():
    d = W.make("dlrm")
    assert d.sizes.sum() == 10_000_000 and d.sizes.size == 26
    assert d.sizes.min() >= 1000 and d.sizes.max() <= 2_000_000
    k = d.keys(0)
    assert k.size == 212_992
    f = (k >> np.uint64(40)).astype(np.int64).reshape(8192, 26)
    assert np.all(f == np.arange(26)[None, :])             # sample-major layout
    ids = (k & np.uint64((1 << 40) - 1)).reshape(8192, 26)
    assert np.all(ids < d.sizes[None, :].astype(np.uint64))
    pre = d.prefill_keys()
    assert pre.size == 10_000_000 and np.all(pre[1:] > pre[:-1])


def test_kg_gnn_large_scaled_shapes():
    kg = W.make("kg", scale=0.01)
    k = kg.keys(0)
    assert k.size == 3 * kg.edges and k.max() < kg.nent
    gnn = W.make("gnn", scale=0.01)
    assert gnn.keys(0).size == gnn.n
    lg = W.make("large", scale=0.01)
    pre = lg.prefill_keys()
    assert np.all(pre[1:] > pre[:-1])
    assert abs(pre.size - lg.fill) < 0.01 * lg.fill
    miss = ~np.isin(lg.keys(0), pre)
    assert 0.12 < miss.mean() < 0.18


@pytest.mark.slow
def test_gnn_full_size_duplicate_fraction_about_30_percent():
    g = W.make("gnn")
    k = g.keys(0)
    dup = 1.0 - np.unique(k).size / k.size
    assert 0.25 < dup < 0.35


def test_kv_mix_shapes_and_skew():
    for name in ("kv-uniform", "kv-zipf"):
        wl = W.make(name, scale=0.01)
        k = wl.keys(0)
        v = wl.values(0)
        pre = wl.prefill_keys()
        assert k.dtype == np.uint64 and k.size == wl.n and wl.n % 2 == 0
        assert v.shape == (wl.n // 2, wl.dim) and v.dtype == np.float32
        assert pre.size == wl.capacity and np.all(np.diff(pre.astype(np.float64)) >= 0)
        assert np.isin(k, pre).all()  # every operation hits a prefilled record
        assert np.array_equal(k, wl.keys(0)) and not np.array_equal(k, wl.keys(1))
    u = W.make("kv-uniform", scale=0.01).keys(0)
    z = W.make("kv-zipf", scale=0.01).keys(0)
    # the skewed mix repeats keys far more than the uniform one
    assert np.unique(z).size < 0.7 * np.unique(u).size
