"""The get of the next batch and put_grad of the current one in one call
(mlkv_get_put_grad: the order of asynchronous training, Sec. II, kept within
a staleness bound, Sec. III-C1), against the CPU oracle, which takes the get
and then the put; and against a twin table that issues the two calls one
after the other.

Bar: as in the parity tests (get outputs and rows bit-exact until updated,
then within 1e-5 row-scaled; blocked flags, staleness counts and key -> row
exact); against the twin table every row, accumulator and count is
bit-identical, since the same arithmetic runs on each row in the same order.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2504_01506_amd import mlkv
from _harness import Pair, dev, dev_keys, log

pytestmark = pytest.mark.gpu


def _keys(rng, n, space, zipf=False):
    ids = (rng.zipf(1.2, size=n) % space) if zipf else rng.integers(0, space, size=n)
    k = ids.astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15) + np.uint64(7)
    k[k == np.uint64(mlkv.MLKV_RESERVED_KEY)] = np.uint64(3)
    return k


@pytest.mark.parametrize("bound", [None, 0, 1, 3])
@pytest.mark.parametrize("dim", [8, 64, 130])
def test_pipelined_steps_match_the_oracle(bound, dim):
    # a training loop: batch t+1's get, then batch t's put, in one call;
    # positions the bound blocks are fetched again once the put is done
    rng = np.random.default_rng(7 + dim + (bound or 0) * 100)
    pr = Pair(dim, 60_000, staleness_bound=bound)
    cur = _keys(rng, 5000, 20_000, zipf=True)
    if bound is None:
        pr.get(cur)
    else:
        pr.get_bounded(cur)
    nblocked = 0
    for s in range(8):
        n = 4097 if s == 3 else int(rng.integers(500, 9000))
        nxt = _keys(rng, n, 20_000, zipf=(s % 2 == 0))
        g = rng.normal(0, 0.01, size=(cur.size, dim)).astype(np.float32)
        bl = pr.get_put_grad(nxt, cur, g, 0.01, 1e-8)
        if bl is not None and bl.any():
            nblocked += int(bl.sum())
            again = pr.get_bounded(nxt[bl == 1])
            assert not again.any()  # the put they waited for is done
        if bound is not None and s % 3 == 2:
            pr.compare_staleness()
        cur = nxt
    pr.put(cur, rng.normal(0, 0.01, size=(cur.size, dim)).astype(np.float32), 0.01, 1e-8)
    if bound is not None:
        counts = pr.compare_staleness()
        assert int(counts.max()) == 0
    if bound == 0:
        assert nblocked > 0
    pr.compare_rows()
    pr.check_index()
    log(f"[pipelined] bound {bound} dim {dim}: {nblocked} blocked, size {pr.ora.size} stats={pr.stats}")
    pr.close()


def _export(t):
    w, st = t.read_rows(torch.arange(t.size, dtype=torch.int64, device="cuda"))
    return w.cpu().numpy().view(np.uint32), st.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("kind", ["plain", "radix", "tiered", "bounded1"])
def test_pipelined_calls_equal_the_calls_in_order(kind):
    # two GPU tables with the same calls: one issues each get with the put of
    # the batch before it in one call, the other as two calls; every bit must
    # agree
    rng = np.random.default_rng(31)
    dim, cap = 64, 400_000
    kw = {}
    if kind == "radix":
        kw["dedup"] = "radix"
    elif kind == "tiered":
        kw["cache_rows"] = 60_000
    elif kind == "bounded1":
        kw["staleness_bound"] = 1
    a = mlkv.Table(dim, cap, **kw)
    b = mlkv.Table(dim, cap, **kw)
    bounded = kind == "bounded1"
    cur = dev_keys(_keys(rng, 50_000, 300_000, zipf=True))
    for t in (a, b):
        if bounded:
            t.get_bounded(cur, None)
        else:
            t.get(cur, None)
    for s in range(6):
        nxt = dev_keys(_keys(rng, int(rng.integers(20_000, 80_000)), 300_000, zipf=(s % 2 == 1)))
        g = dev(rng.normal(0, 0.01, size=(cur.numel(), dim)).astype(np.float32))
        oa = torch.empty((nxt.numel(), dim), dtype=torch.float32, device="cuda")
        ob = torch.empty_like(oa)
        if kind == "tiered":
            a.lookahead(nxt)
            b.lookahead(nxt)
        bla = a.get_put_grad(nxt, oa, cur, g, 0.01, 1e-8)
        if bounded:
            blb = b.get_bounded(nxt, ob)
        else:
            b.get(nxt, ob)
        b.put_grad(cur, g, 0.01, 1e-8)
        assert a.sync() == mlkv.MLKV_OK and b.sync() == mlkv.MLKV_OK
        if bounded:
            assert torch.equal(bla, blb)
            served = (bla == 0).unsqueeze(1)
            assert torch.equal(torch.where(served, oa, 0.0).view(torch.int32),
                               torch.where(served, ob, 0.0).view(torch.int32))
        else:
            assert torch.equal(oa.view(torch.int32), ob.view(torch.int32))
        cur = nxt
    assert a.size == b.size
    wa, sa = _export(a)
    wb, sb = _export(b)
    assert np.array_equal(wa, wb) and np.array_equal(sa, sb)
    if bounded:
        rows = torch.arange(a.size, dtype=torch.int64, device="cuda")
        assert torch.equal(a.read_staleness(rows), b.read_staleness(rows))
    assert torch.equal(a.lookup_rows(cur), b.lookup_rows(cur))
    log(f"[pipelined] {kind}: twin tables identical, size {a.size}")
    a.close()
    b.close()


def test_a_put_key_absent_before_the_call_fails_the_put_alone():
    rng = np.random.default_rng(41)
    dim = 16
    pr = Pair(dim, 10_000)
    known = _keys(rng, 2000, 5000)
    pr.get(known)
    w0, s0 = _export(pr.gpu)
    # a put key never inserted; then one that this call's get inserts
    for case, bad in enumerate((np.uint64(0x5151515151), np.uint64(0xABCDEF12345))):
        nxt = _keys(rng, 1500, 9000)
        if case == 1:
            nxt[7] = bad
        put = known.copy()
        put[100] = bad
        g = rng.normal(0, 0.01, size=(put.size, dim)).astype(np.float32)
        out = torch.empty((nxt.size, dim), dtype=torch.float32, device="cuda")
        pr.gpu.get_put_grad(dev_keys(nxt), out, dev_keys(put), dev(g), 0.01, 1e-8)
        assert pr.gpu.sync() == mlkv.MLKV_EINVAL
        assert "absent" in mlkv.mlkv_last_error()
        # the get was applied (the oracle takes it alone), the put was not
        rc, want = pr.ora.get(nxt)
        assert rc == O.OK
        pr.compare_get(nxt, out.cpu().numpy(), want)
        w1, s1 = _export(pr.gpu)
        n0 = w0.shape[0]
        assert np.array_equal(w1[:n0], w0) and np.array_equal(s1[:n0], s0)
        w0, s0 = w1, s1
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_a_reserved_key_fails_only_its_own_part():
    rng = np.random.default_rng(43)
    dim = 8
    pr = Pair(dim, 10_000)
    known = _keys(rng, 1000, 3000)
    pr.get(known)
    g = rng.normal(0, 0.01, size=(known.size, dim)).astype(np.float32)
    res = np.uint64(mlkv.MLKV_RESERVED_KEY)
    # the reserved key in the put: the get is applied, the put is not
    nxt = _keys(rng, 800, 6000)
    put = known.copy()
    put[5] = res
    out = torch.empty((nxt.size, dim), dtype=torch.float32, device="cuda")
    pr.gpu.get_put_grad(dev_keys(nxt), out, dev_keys(put), dev(g), 0.01, 1e-8)
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    assert "reserved" in mlkv.mlkv_last_error()
    rc, want = pr.ora.get(nxt)
    assert rc == O.OK
    pr.compare_get(nxt, out.cpu().numpy(), want)
    pr.compare_rows()
    # the reserved key in the get: the put is applied, the get is not
    nxt2 = _keys(rng, 900, 8000)
    nxt2[3] = res
    out2 = torch.empty((nxt2.size, dim), dtype=torch.float32, device="cuda")
    size0 = pr.gpu.size
    pr.gpu.get_put_grad(dev_keys(nxt2), out2, dev_keys(known), dev(g), 0.01, 1e-8)
    assert pr.gpu.sync() == mlkv.MLKV_EINVAL
    assert pr.gpu.size == size0
    assert pr.ora.put_grad(known, g, 0.01, 1e-8) == O.OK
    pr.updated[pr.ora.lookup_rows(known)] = True
    pr.compare_rows()
    pr.check_index()
    pr.close()


def test_one_part_empty_is_the_other_call():
    rng = np.random.default_rng(47)
    dim = 32
    pr = Pair(dim, 20_000)
    k = _keys(rng, 3000, 10_000)
    g = rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32)
    # no put: a get
    out = torch.empty((k.size, dim), dtype=torch.float32, device="cuda")
    empty = torch.empty(0, dtype=torch.int64, device="cuda")
    pr.gpu.get_put_grad(dev_keys(k), out, empty, torch.empty((0, dim), device="cuda"), 0.01, 1e-8)
    rc, want = pr.ora.get(k)
    assert rc == O.OK and pr.gpu.sync() == mlkv.MLKV_OK
    pr.compare_get(k, out.cpu().numpy(), want)
    # no get: a put
    pr.gpu.get_put_grad(empty, None, dev_keys(k), dev(g), 0.01, 1e-8)
    assert pr.ora.put_grad(k, g, 0.01, 1e-8) == O.OK
    assert pr.gpu.sync() == mlkv.MLKV_OK
    pr.updated[pr.ora.lookup_rows(k)] = True
    pr.compare_rows()
    pr.close()


def test_work_waiting_for_the_get_done_event_sees_the_rows():
    # a second stream waits for the event, then copies the rows out while the
    # put's row updates may still run
    rng = np.random.default_rng(53)
    dim = 64
    pr = Pair(dim, 100_000)
    cur = _keys(rng, 40_000, 60_000, zipf=True)
    pr.get(cur)
    side = torch.cuda.Stream()  # default priority
    for _ in range(3):
        nxt = _keys(rng, 40_000, 60_000, zipf=True)
        g = rng.normal(0, 0.01, size=(cur.size, dim)).astype(np.float32)
        out = torch.empty((nxt.size, dim), dtype=torch.float32, device="cuda")
        copy = torch.empty_like(out)
        done = torch.cuda.Event()
        kd, pd, gd = dev_keys(nxt), dev_keys(cur), dev(g)
        pr.gpu.get_put_grad(kd, out, pd, gd, 0.01, 1e-8, get_done=done)
        with torch.cuda.stream(side):
            side.wait_event(done)
            copy.copy_(out)
        side.synchronize()
        rc, want = pr.ora.get(nxt)
        assert rc == O.OK and pr.ora.put_grad(cur, g, 0.01, 1e-8) == O.OK
        assert pr.gpu.sync() == mlkv.MLKV_OK
        pr.compare_get(nxt, copy.cpu().numpy(), want)
        pr.updated[pr.ora.lookup_rows(cur)] = True
        cur = nxt
    pr.compare_rows()
    pr.close()


def test_argument_checks_leave_the_table_alone():
    # each refused call returns MLKV_EINVAL before queuing anything: the table
    # answers the next call as if the refused ones had not been made
    rng = np.random.default_rng(59)
    dim = 16
    pr = Pair(dim, 20_000, staleness_bound=1)
    k = _keys(rng, 2000, 8000)
    pr.get_bounded(k)
    h = pr.gpu.h
    kd, gd = dev_keys(k), dev(rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32))
    out = torch.empty((k.size, dim), dtype=torch.float32, device="cuda")
    bl = torch.empty(k.size, dtype=torch.uint8, device="cuda")
    call = mlkv.mlkv_get_put_grad
    assert call(h, kd, k.size, out, None, kd, gd, k.size, 0.01, 1e-8) == mlkv.MLKV_EINVAL  # no blocked flags
    assert "blocked" in mlkv.mlkv_last_error()
    assert call(h, kd, -1, out, bl, kd, gd, k.size, 0.01, 1e-8) == mlkv.MLKV_EINVAL
    assert call(h, kd, k.size, out, bl, kd, gd, -1, 0.01, 1e-8) == mlkv.MLKV_EINVAL
    assert call(h, kd, k.size, out, bl, kd, gd, k.size, float("nan"), 1e-8) == mlkv.MLKV_EINVAL
    assert call(h, kd, k.size, out, bl, kd, gd, k.size, 0.01, -1.0) == mlkv.MLKV_EINVAL
    assert call(h, kd, k.size, out, bl, kd, None, k.size, 0.01, 1e-8) == mlkv.MLKV_EINVAL
    assert call(h, None, k.size, out, bl, kd, gd, k.size, 0.01, 1e-8) == mlkv.MLKV_EINVAL
    assert pr.gpu.sync() == mlkv.MLKV_OK
    # the same table goes on as the oracle does
    nxt = _keys(rng, 1500, 8000)
    bl2 = pr.get_put_grad(nxt, k, rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32), 0.01, 1e-8)
    assert bl2 is not None
    pr.compare_staleness()
    pr.compare_rows()
    pr.close()
