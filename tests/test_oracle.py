"""Pins of the CPU oracle against things other than itself.

Each test fixes part of the oracle by an independent fact: a published test
vector, a library routine that reduces to the same mathematics in a special
case, brute force on tiny inputs, a closed form, or an invariant that a wrong
sign, a dropped term or a swapped operand would break.
"""
import math
import os

import numpy as np
import pytest

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_hex(name):
    vals = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                vals.append(int(line, 16))
    return vals


# --------------------------------------------------------------------------
# init: SplitMix64 finaliser (published vectors) and the value map
# --------------------------------------------------------------------------
def test_mix64_matches_published_splitmix64_sequence():
    want = _golden_hex("splitmix64_seed0.txt")
    state, got = 0, []
    for _ in want:
        state = (state + 0x9E3779B97F4A7C15) & (2**64 - 1)
        got.append(O.mix64(state))
    assert got == want


def test_init_values_lie_on_the_stated_grid_and_range():
    # every value is the fp32 product of an integer t in [-2^23, 2^23) with the
    # fp32 constant 0.01f * 2^-23, so it lies in [-0.01f, 0.01f)
    step = np.float32(0.01) * np.float32(2.0**-23)
    keys = [0, 1, 2, 12345, 2**40 + 7, 2**63 + 11]
    for k in keys:
        for c in range(64):
            v = np.float32(O.init_value(O.DEFAULT_SEED, k, c))
            t = int(round(float(v) / float(step)))
            assert -(2**23) <= t < 2**23
            assert np.float32(np.float32(t) * step) == v
            assert -np.float32(0.01) <= v < np.float32(0.01)


def test_init_columns_follow_the_splitmix64_stream():
    # Column c of a key's initial row is output c+1 of the reference SplitMix64
    # generator (state += 0x9E3779B97F4A7C15, then mix64) started from the state
    # mix64(key ^ seed) - gamma; the top 24 bits of that output, centred, scaled
    # by 0.01f * 2^-23, give the value.
    gamma = 0x9E3779B97F4A7C15
    step = np.float32(0.01) * np.float32(2.0**-23)
    for seed, key in [(O.DEFAULT_SEED, 0), (1, 2**40 + 3), (2**63, 123456789)]:
        state = (O.mix64(key ^ seed) - gamma) & (2**64 - 1)
        for c in range(40):
            state = (state + gamma) & (2**64 - 1)
            h = O.mix64(state)
            v = np.float32(np.float32((h >> 40) - 2**23) * step)
            assert v == np.float32(O.init_value(seed, key, c)), (seed, key, c)


def test_init_statistics_uniform_on_pm_001():
    vals = np.array([O.init_value(7, k, c) for k in range(2000) for c in range(16)], dtype=np.float64)
    assert vals.min() >= -0.01 and vals.max() < 0.01
    assert abs(vals.mean()) < 3 * 0.02 / math.sqrt(12 * vals.size) * 2
    assert abs(vals.var() - 0.02**2 / 12) < 0.05 * 0.02**2 / 12
    # a uniform variable has its quartiles at -0.005, 0, 0.005
    q = np.quantile(vals, [0.25, 0.5, 0.75])
    assert np.allclose(q, [-0.005, 0.0, 0.005], atol=5e-4)


def test_init_depends_only_on_seed_key_and_column():
    a = O.OracleTable(8, 100, seed=99)
    b = O.OracleTable(8, 100, seed=99)
    c = O.OracleTable(8, 100, seed=100)
    _, oa = a.get([10, 20, 30])
    _, ob = b.get([30, 999, 20, 10])       # other order, other rows
    _, oc = c.get([10, 20, 30])
    assert np.array_equal(oa[0], ob[3]) and np.array_equal(oa[1], ob[2]) and np.array_equal(oa[2], ob[0])
    assert not np.array_equal(oa, oc)
    assert not np.array_equal(oa[0, :4], oa[0, 4:])


# --------------------------------------------------------------------------
# resolve: brute-force list model of the row-assignment rule (R1)
# --------------------------------------------------------------------------
class ListModel:
    """Key -> row as a Python list of pairs; the rule written in its plainest form."""

    def __init__(self, cap):
        self.pairs = []
        self.cap = cap

    def rows(self, keys):
        known = {k for k, _ in self.pairs}
        new = sorted(set(k for k in keys if k not in known))
        if len(self.pairs) + len(new) > self.cap:
            return None
        for k in new:
            self.pairs.append((k, len(self.pairs)))
        return [next(r for kk, r in self.pairs if kk == k) for k in keys]


@pytest.mark.parametrize("seed", range(20))
def test_row_assignment_matches_list_model(seed):
    rng = np.random.default_rng(seed)
    cap = int(rng.integers(5, 40))
    t = O.OracleTable(3, cap)
    m = ListModel(cap)
    for _ in range(6):
        n = int(rng.integers(0, 12))
        keys = rng.integers(0, 30, size=n).astype(np.uint64)
        want = m.rows([int(k) for k in keys])
        before = t.size
        rc, _ = t.get(keys)
        if want is None:
            assert rc == O.EFULL and t.size == before
            continue
        assert rc == O.OK
        assert t.lookup_rows(keys).tolist() == want
        assert t.size == len(m.pairs)
    # bijection onto [0, size)
    allk = np.array(sorted(k for k, _ in m.pairs), dtype=np.uint64)
    rows = t.lookup_rows(allk)
    assert sorted(rows.tolist()) == list(range(t.size))
    assert t.row_keys(rows).tolist() == allk.tolist()


def test_lookup_never_inserts():
    t = O.OracleTable(2, 10)
    assert t.lookup_rows([1, 2, 3]).tolist() == [-1, -1, -1]
    assert t.size == 0


def test_prefill_sorted_equals_inserting_through_get():
    keys = np.array([3, 8, 9, 100, 2**41], dtype=np.uint64)
    a = O.OracleTable(4, 10)
    b = O.OracleTable(4, 10)
    assert a.prefill_sorted(keys) == O.OK
    assert b.get(keys, want_out=False)[0] == O.OK
    probe = np.array([100, 3, 7, 2**41], dtype=np.uint64)
    assert a.lookup_rows(probe).tolist() == b.lookup_rows(probe).tolist()
    ra, oa = a.get(probe)
    rb, ob = b.get(probe)
    assert ra == rb == O.OK and np.array_equal(oa, ob)
    assert a.size == b.size == 6


def test_errors_leave_the_table_unchanged():
    t = O.OracleTable(2, 3)
    assert t.get([1, 2])[0] == O.OK
    g = np.ones((3, 2), np.float32)
    assert t.get([5, 6, 7])[0] == O.EFULL
    assert t.put_grad([8, 9, 1], g, 0.1, 0.0) == O.EFULL
    assert t.size == 2
    _, st = t.read_rows([0, 1])
    assert st.tolist() == [0.0, 0.0]
    assert t.get([1, 0xFFFFFFFFFFFFFFFF])[0] == O.EINVAL
    assert t.put_grad([1], g[:1], float("nan"), 0.0) == O.EINVAL
    assert t.put_grad([1], g[:1], 0.1, -1.0) == O.EINVAL
    assert t.put_grad([1], g[:1], 0.1, float("inf")) == O.EINVAL
    assert t.size == 2
    assert t.get([3])[0] == O.OK and t.size == 3     # exactly at capacity is fine
    with pytest.raises(ValueError):
        O.OracleTable(0, 10)
    with pytest.raises(ValueError):
        O.OracleTable(4, 0)


# --------------------------------------------------------------------------
# Adagrad: library special cases (torch.optim.Adagrad), closed form, invariants
# --------------------------------------------------------------------------
torch = pytest.importorskip("torch")


def test_dim1_equals_torch_adagrad_dense():
    rng = np.random.default_rng(1)
    lr, eps = 0.05, 1e-8
    t = O.OracleTable(1, 4)
    _, w0 = t.get([42])
    p = torch.nn.Parameter(torch.tensor(w0[0].copy()))
    opt = torch.optim.Adagrad([p], lr=lr, eps=eps)
    for _ in range(25):
        g = rng.normal(0, 0.3, size=1).astype(np.float32)
        assert t.put_grad([42], g.reshape(1, 1), lr, eps) == O.OK
        p.grad = torch.tensor(g)
        opt.step()
    w, st = t.read_rows([0])
    np.testing.assert_allclose(w[0], p.detach().numpy(), rtol=2e-6, atol=0)
    np.testing.assert_allclose(st[0], opt.state[p]["sum"].numpy()[0], rtol=2e-6)


def test_constant_rows_equal_elementwise_adagrad_pins_mean_over_dim():
    # If every element of a gradient row is the same value g, mean(g^2) = g^2 and
    # row-wise Adagrad coincides with element-wise Adagrad. Summing instead of
    # averaging over the row would make G eight times larger here.
    rng = np.random.default_rng(2)
    D, lr, eps = 8, 0.02, 1e-8
    t = O.OracleTable(D, 4)
    _, w0 = t.get([5])
    p = torch.nn.Parameter(torch.tensor(w0[0].copy()))
    opt = torch.optim.Adagrad([p], lr=lr, eps=eps)
    for _ in range(10):
        gv = np.float32(rng.normal(0, 0.1))
        g = np.full((1, D), gv, np.float32)
        assert t.put_grad([5], g, lr, eps) == O.OK
        p.grad = torch.tensor(g[0])
        opt.step()
    w, st = t.read_rows([0])
    np.testing.assert_allclose(w[0], p.detach().numpy(), rtol=2e-6)
    np.testing.assert_allclose(st[0], opt.state[p]["sum"].numpy()[0], rtol=2e-6)


def test_duplicates_sum_then_one_step_like_torch_sparse_adagrad():
    # torch's sparse Adagrad coalesces (sums) duplicate indices before its step.
    rng = np.random.default_rng(3)
    lr, eps = 0.1, 1e-8
    keys = np.array([7, 3, 7, 7, 9, 3, 11], dtype=np.uint64)
    t = O.OracleTable(1, 16)
    _, w0 = t.get(np.array([3, 7, 9, 11], np.uint64))
    emb = torch.nn.Embedding(4, 1, sparse=True)
    with torch.no_grad():
        emb.weight.copy_(torch.tensor(w0))
    opt = torch.optim.Adagrad(emb.parameters(), lr=lr, eps=eps)
    idx_of = {3: 0, 7: 1, 9: 2, 11: 3}
    for _ in range(5):
        g = rng.normal(0, 0.2, size=(keys.size, 1)).astype(np.float32)
        assert t.put_grad(keys, g, lr, eps) == O.OK
        idx = torch.tensor([idx_of[int(k)] for k in keys])
        opt.zero_grad()
        out = emb(idx)
        out.backward(torch.tensor(g))
        opt.step()
    w, st = t.read_rows([0, 1, 2, 3])
    np.testing.assert_allclose(w[:, 0], emb.weight.detach().numpy()[:, 0], rtol=3e-6)


def test_closed_form_constant_gradient():
    # one key, the same gradient row every step, G0 = 0:
    #   G_t = t * m,   w_t = w_0 - lr * g * sum_{k=1..t} 1 / (sqrt(k m) + eps)
    D, lr, eps, T = 16, 0.01, 1e-3, 40
    g = (np.arange(D, dtype=np.float32) - 7.5) * np.float32(0.01)
    m = float(np.mean(g.astype(np.float64) ** 2))
    t = O.OracleTable(D, 2)
    _, w0 = t.get([1])
    for _ in range(T):
        assert t.put_grad([1], g.reshape(1, D), lr, eps) == O.OK
    w, st = t.read_rows([0])
    s = sum(1.0 / (math.sqrt(k * m) + eps) for k in range(1, T + 1))
    want = w0[0].astype(np.float64) - lr * g.astype(np.float64) * s
    np.testing.assert_allclose(st[0], T * m, rtol=1e-5)
    np.testing.assert_allclose(w[0], want, rtol=1e-4, atol=1e-7)


@pytest.mark.parametrize("k", [-3, 2, 5])
def test_scale_invariance_with_zero_eps(k):
    # with eps = 0 the step is invariant to scaling gradients by 2^k (exact in
    # IEEE arithmetic), while G scales by 4^k.
    rng = np.random.default_rng(4)
    D = 12
    keys = rng.integers(0, 20, size=60).astype(np.uint64)
    a = O.OracleTable(D, 64)
    b = O.OracleTable(D, 64)
    for step in range(4):
        g = rng.normal(0, 0.01, size=(keys.size, D)).astype(np.float32)
        assert a.put_grad(keys, g, 0.03, 0.0) == O.OK
        assert b.put_grad(keys, g * np.float32(2.0**k), 0.03, 0.0) == O.OK
    rows = np.arange(a.size)
    wa, sa = a.read_rows(rows)
    wb, sb = b.read_rows(rows)
    assert np.array_equal(wa, wb)
    assert np.array_equal(sa * np.float32(4.0**k), sb)


def test_accumulator_never_decreases_and_get_after_put_sees_update():
    rng = np.random.default_rng(5)
    D = 6
    t = O.OracleTable(D, 50)
    prev = None
    for step in range(5):
        keys = rng.integers(0, 30, size=40).astype(np.uint64)
        rc, before = t.get(keys)
        g = rng.normal(0, 0.01, size=(keys.size, D)).astype(np.float32)
        assert t.put_grad(keys, g, 0.01, 1e-8) == O.OK
        rc, after = t.get(keys)
        assert not np.array_equal(before, after)
        _, st = t.read_rows(np.arange(t.size))
        if prev is not None:
            assert np.all(st[: prev.size] >= prev)
        prev = st


def _exact_sum_f32(col):
    return np.float32(math.fsum(float(x) for x in col))


def test_segment_sum_all_same_key_is_the_full_sum_and_permutation_invariant():
    rng = np.random.default_rng(6)
    D, n, lr, eps = 5, 300, 0.01, 1e-8
    g = rng.normal(0, 0.01, size=(n, D)).astype(np.float32)
    a = O.OracleTable(D, 4)
    _, w0 = a.get([77])
    assert a.put_grad(np.full(n, 77, np.uint64), g, lr, eps) == O.OK
    w, st = a.read_rows([0])
    gs = np.array([_exact_sum_f32(g[:, c]) for c in range(D)], np.float32)
    m = np.float32(np.sum(gs.astype(np.float64) ** 2) / D)
    den = np.float32(np.sqrt(np.float32(0) + m)) + np.float32(eps)
    want = w0[0] - np.float32(lr) * (gs / den)
    np.testing.assert_allclose(w[0], want, rtol=1e-6)
    # the same batch in another order gives the same result
    perm = rng.permutation(n)
    b = O.OracleTable(D, 4)
    b.get([77])
    assert b.put_grad(np.full(n, 77, np.uint64), g[perm], lr, eps) == O.OK
    wb, stb = b.read_rows([0])
    np.testing.assert_allclose(wb, w, rtol=1e-7)
    np.testing.assert_allclose(stb, st, rtol=1e-7)


def test_segment_sum_all_distinct_is_identity():
    # all keys distinct: each row sees exactly its own gradient row; compare
    # with torch's element-wise Adagrad on rows whose elements are equal.
    rng = np.random.default_rng(7)
    D, n, lr, eps = 4, 50, 0.02, 1e-8
    keys = np.arange(1000, 1000 + n, dtype=np.uint64)
    t = O.OracleTable(D, n)
    _, w0 = t.get(keys)
    gv = rng.normal(0, 0.05, size=n).astype(np.float32)
    g = np.repeat(gv[:, None], D, axis=1)
    assert t.put_grad(keys, g, lr, eps) == O.OK
    _, w = t.get(keys)
    p = torch.nn.Parameter(torch.tensor(w0.copy()))
    opt = torch.optim.Adagrad([p], lr=lr, eps=eps)
    p.grad = torch.tensor(g)
    opt.step()
    np.testing.assert_allclose(w, p.detach().numpy(), rtol=2e-6)


# ---- Put (batch upsert) and the SGD variant of the Rmw ----------------------

@pytest.mark.parametrize("seed", range(10))
def test_put_matches_a_dict_model_last_position_wins(seed):
    rng = np.random.default_rng(100 + seed)
    dim, cap = 3, 60
    t = O.OracleTable(dim, cap)
    rows_model = ListModel(cap)
    vals = {}  # key -> row values the plain dict model holds
    for _ in range(5):
        n = int(rng.integers(1, 15))
        keys = rng.integers(0, 40, size=n).astype(np.uint64)
        v = rng.normal(size=(n, dim)).astype(np.float32)
        want_rows = rows_model.rows([int(k) for k in keys])
        assert want_rows is not None
        assert t.put(keys, v) == O.OK
        for i, k in enumerate(keys.tolist()):   # sequential upserts: later positions overwrite
            vals[k] = v[i].copy()
        assert t.lookup_rows(keys).tolist() == want_rows
        ks = np.array(sorted(vals), dtype=np.uint64)
        rc, got = t.get(ks)
        assert rc == O.OK
        assert np.array_equal(got, np.stack([vals[k] for k in ks.tolist()]))


def test_put_keeps_the_accumulator_of_existing_keys_and_zeroes_new_ones():
    t = O.OracleTable(2, 10)
    g = np.array([[0.5, -0.5]], np.float32)
    assert t.put_grad(np.array([4], np.uint64), g, 0.1, 1e-8) == O.OK
    _, st0 = t.read_rows([0])
    assert st0[0] > 0
    assert t.put(np.array([4, 9], np.uint64), np.ones((2, 2), np.float32)) == O.OK
    w, st = t.read_rows([0, 1])
    assert st[0] == st0[0] and st[1] == 0.0
    assert np.array_equal(w, np.ones((2, 2), np.float32))


def test_put_errors_leave_the_table_unchanged():
    t = O.OracleTable(2, 3)
    assert t.put(np.array([1, 2], np.uint64), np.zeros((2, 2), np.float32)) == O.OK
    assert t.put(np.array([3, 4], np.uint64), np.ones((2, 2), np.float32)) == O.EFULL
    assert t.put(np.array([1, O_RESERVED], np.uint64), np.ones((2, 2), np.float32)) == O.EINVAL
    assert t.size == 2
    _, w = t.get(np.array([1, 2], np.uint64))
    assert np.array_equal(w, np.zeros((2, 2), np.float32))


O_RESERVED = np.uint64(0xFFFFFFFFFFFFFFFF)


@pytest.mark.parametrize("dim", [1, 8])
def test_sgd_equals_torch_sparse_sgd_with_duplicates(dim):
    # torch's sparse SGD coalesces (sums) duplicate indices, then w -= lr * g
    rng = np.random.default_rng(7 + dim)
    lr = 0.05
    keys = np.array([7, 3, 7, 7, 9, 3, 11], dtype=np.uint64)
    t = O.OracleTable(dim, 16)
    _, w0 = t.get(np.array([3, 7, 9, 11], np.uint64))
    emb = torch.nn.Embedding(4, dim, sparse=True)
    with torch.no_grad():
        emb.weight.copy_(torch.tensor(w0))
    opt = torch.optim.SGD(emb.parameters(), lr=lr)
    idx_of = {3: 0, 7: 1, 9: 2, 11: 3}
    for _ in range(5):
        g = rng.normal(0, 0.2, size=(keys.size, dim)).astype(np.float32)
        assert t.put_grad_sgd(keys, g, lr) == O.OK
        idx = torch.tensor([idx_of[int(k)] for k in keys])
        opt.zero_grad()
        emb(idx).backward(torch.tensor(g))
        opt.step()
    w, st = t.read_rows([0, 1, 2, 3])
    np.testing.assert_allclose(w, emb.weight.detach().numpy(), rtol=2e-6, atol=1e-9)
    assert np.all(st == 0)   # the SGD step leaves the Adagrad accumulators alone


def test_sgd_closed_form_with_exact_sums():
    # k copies of the same power-of-two gradient sum exactly, so the step is
    # w1 = w0 - lr * (k * g) bit for bit
    t = O.OracleTable(4, 8)
    _, w0 = t.get(np.array([5], np.uint64))
    k, gval, lr = 6, 0.25, 0.5
    keys = np.full(k, 5, np.uint64)
    assert t.put_grad_sgd(keys, np.full((k, 4), gval, np.float32), lr) == O.OK
    w, _ = t.read_rows([0])
    want = (w0[0] - np.float32(lr) * np.float32(k * gval)).astype(np.float32)
    assert np.array_equal(w[0], want)


# --------------------------------------------------------------------------
# bounded staleness (Sec. III-C1): closed forms of the per-key counts
# --------------------------------------------------------------------------
def _blocked_keys(keys, blocked):
    return {int(k) for k, b in zip(keys, blocked) if b}


@pytest.mark.parametrize("bound", [0, 1, 3])
def test_staleness_bound_serves_exactly_bound_plus_one_gets_before_a_put(bound):
    # a key fetched again and again without any put is served bound + 1 times
    # (the stale-synchronous window), then blocked until one put completes
    t = O.OracleTable(4, 16, staleness_bound=bound)
    k = np.array([42], np.uint64)
    for _ in range(bound + 1):
        rc, _, bl = t.get_bounded(k)
        assert rc == O.OK and bl[0] == 0
    for _ in range(3):
        rc, _, bl = t.get_bounded(k)
        assert rc == O.OK and bl[0] == 1   # blocked gets do not count
    # one put call completes one get, however often it holds the key
    assert t.put_grad(np.repeat(k, 2), np.zeros((2, 4), np.float32), 0.1, 1e-8) == O.OK
    rc, _, bl = t.get_bounded(k)
    assert rc == O.OK and bl[0] == 0
    rc, _, bl = t.get_bounded(k)
    assert bl[0] == 1


def test_bsp_pipeline_blocks_exactly_the_keys_shared_with_the_pending_step():
    # bound 0 with get(s) issued before put(s-1): the blocked keys are the
    # intersection of the two batches; once put(s-1) is done a second get of
    # the blocked keys is served. Strictly alternating get and put never blocks.
    rng = np.random.default_rng(7)
    t = O.OracleTable(4, 4096, staleness_bound=0)
    batches = [rng.integers(0, 300, size=200).astype(np.uint64) for _ in range(6)]
    assert not t.get_bounded(batches[0])[2].any()
    for s in range(1, 6):
        rc, _, bl = t.get_bounded(batches[s])
        assert rc == O.OK
        want = set(int(x) for x in batches[s]) & set(int(x) for x in batches[s - 1])
        assert want and _blocked_keys(batches[s], bl) == want
        g = np.zeros((batches[s - 1].size, 4), np.float32)
        assert t.put_grad(batches[s - 1], g, 0.1, 1e-8) == O.OK
        again = batches[s][bl == 1]
        rc, _, bl2 = t.get_bounded(again)
        assert rc == O.OK and not bl2.any()
    t2 = O.OracleTable(4, 4096, staleness_bound=0)
    for s in range(6):
        rc, _, bl = t2.get_bounded(batches[s])
        assert rc == O.OK and not bl.any()
        assert t2.put(batches[s], np.zeros((batches[s].size, 4), np.float32)) == O.OK


def test_bound_one_three_deep_pipeline_blocks_the_triple_intersection():
    # bound 1, gets of steps 0, 1, 2 before any put: the third get blocks the
    # keys present in all three batches and nothing else
    rng = np.random.default_rng(11)
    t = O.OracleTable(4, 4096, staleness_bound=1)
    b = [rng.integers(0, 120, size=100).astype(np.uint64) for _ in range(3)]
    for s in range(2):
        rc, _, bl = t.get_bounded(b[s])
        assert rc == O.OK and not bl.any()
    rc, _, bl = t.get_bounded(b[2])
    want = set(int(x) for x in b[0]) & set(int(x) for x in b[1]) & set(int(x) for x in b[2])
    assert _blocked_keys(b[2], bl) == want


def test_staleness_duplicates_in_one_call_count_once_and_rows_match_an_untracked_table():
    # a key repeated within one get is served at every position and counted
    # once; served rows are exactly those of a table without a bound that saw
    # the same served calls
    rng = np.random.default_rng(3)
    dim = 8
    t = O.OracleTable(dim, 1024, staleness_bound=0)
    u = O.OracleTable(dim, 1024)
    keys = np.repeat(np.array([9, 4, 9, 1], np.uint64), 25)
    rc, out, bl = t.get_bounded(keys)
    assert rc == O.OK and not bl.any()
    rc2, out2 = u.get(keys)
    assert np.array_equal(out, out2)
    rows = t.lookup_rows(np.array([9, 4, 1], np.uint64))
    assert list(t.staleness(rows)) == [1, 1, 1]
    g = rng.normal(0, 0.01, size=(keys.size, dim)).astype(np.float32)
    assert t.put_grad(keys, g, 0.01, 1e-8) == O.OK and u.put_grad(keys, g, 0.01, 1e-8) == O.OK
    assert list(t.staleness(rows)) == [0, 0, 0]
    rc, out, bl = t.get_bounded(keys)
    assert not bl.any() and np.array_equal(out, u.get(keys)[1])


def test_staleness_blocked_rows_are_untouched_and_counts_floor_at_zero():
    t = O.OracleTable(4, 64, staleness_bound=0)
    k = np.array([1, 2], np.uint64)
    t.get_bounded(k)
    sentinel = np.full((2, 4), 7.0, np.float32)
    rc, out, bl = t.get_bounded(k, out=sentinel.copy())
    assert list(bl) == [1, 1] and np.array_equal(out, sentinel)
    # puts on keys without pending gets (and a new key) leave counts at 0
    assert t.put(np.array([1, 2, 3], np.uint64), np.zeros((3, 4), np.float32)) == O.OK
    assert t.put(np.array([1, 2, 3], np.uint64), np.zeros((3, 4), np.float32)) == O.OK
    assert list(t.staleness(t.lookup_rows(np.array([1, 2, 3], np.uint64)))) == [0, 0, 0]
    # a plain get is refused on a bounded table; a failed call changes no count
    assert t.get(k)[0] == O.EINVAL
    t3 = O.OracleTable(4, 3, staleness_bound=0)
    assert t3.get_bounded(np.array([1, 2], np.uint64))[0] == O.OK
    assert t3.get_bounded(np.array([1, 5, 6], np.uint64))[0] == O.EFULL
    assert list(t3.staleness([0, 1])) == [1, 1] and t3.size == 2


# --------------------------------------------------------------------------
# Lookahead with the table in memory: insert ahead, count nothing
# --------------------------------------------------------------------------
def test_lookahead_then_get_equals_get_alone_and_moves_no_count():
    rng = np.random.default_rng(21)
    keys = rng.integers(0, 500, size=800).astype(np.uint64)
    later = rng.integers(0, 700, size=600).astype(np.uint64)
    a = O.OracleTable(4, 2000)
    b = O.OracleTable(4, 2000)
    assert a.get(keys)[0] == O.OK and b.get(keys)[0] == O.OK
    # rows of the keys a lookahead inserts: the R1 rule on the lookahead's
    # own batch (ascending among its missing keys), the same as an
    # insert-only get
    assert a.lookahead(later) == O.OK
    assert b.get(later, want_out=False)[0] == O.OK
    assert a.size == b.size
    assert np.array_equal(a.lookup_rows(later), b.lookup_rows(later))
    assert np.array_equal(a.get(later)[1], b.get(later)[1])
    # bounded table: a lookahead neither blocks nor counts
    t = O.OracleTable(4, 2000, staleness_bound=0)
    k = np.array([1, 2, 3], np.uint64)
    assert t.lookahead(k) == O.OK
    assert list(t.staleness(t.lookup_rows(k))) == [0, 0, 0]
    assert not t.get_bounded(k)[2].any()
    assert t.lookahead(k) == O.OK
    assert list(t.staleness(t.lookup_rows(k))) == [1, 1, 1]
    # failures leave the table unchanged
    full = O.OracleTable(4, 3)
    assert full.lookahead(np.array([1, 2, 3, 4], np.uint64)) == O.EFULL and full.size == 0
    assert full.lookahead(np.array([1, 2**64 - 1], np.uint64)) == O.EINVAL
