"""Calls issued on streams other than the default one, and two tables whose
calls run on two streams at the same time, against the CPU oracle.

Calls on one table are ordered on its stream; tables share no device state
(each has its own index, rows, scratch and control block), so the kernels of
two tables may overlap. Bar as in the parity tests: get outputs and rows
bit-exact until updated, then within 1e-5 row-scaled; key -> row exact."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2504_01506_amd import mlkv
from _harness import Pair, dev, dev_keys, log

pytestmark = pytest.mark.gpu


def test_one_table_on_a_side_stream():
    rng = np.random.default_rng(21)
    dim = 32
    side = torch.cuda.Stream()  # default priority
    with torch.cuda.stream(side):
        pr = Pair(dim, 50_000)
        for _ in range(4):
            k = rng.integers(0, 30_000, size=9_000).astype(np.uint64) * np.uint64(2654435761)
            pr.get(k)
            pr.put(k, rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32), 0.01, 1e-8)
            pr.lookahead(k[::2].copy())
        pr.compare_rows()
        pr.check_index()
        log(f"[streams] side stream: size {pr.ora.size} stats={pr.stats}")
        pr.close()


@pytest.mark.parametrize("second", ["hash", "radix", "tiered"])
def test_two_tables_on_two_streams_at_once(second):
    rng = np.random.default_rng(22)
    dim = 16
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    prs = [Pair(dim, 60_000),
           Pair(dim, 60_000, dedup="radix" if second == "radix" else "hash",
                cache_rows=5_000 if second == "tiered" else None)]
    gets = []   # (pair, keys, device output, oracle output)
    held = []   # device buffers in use on a side stream until it is synchronized
    for step in range(5):
        for j, (pr, st) in enumerate(zip(prs, streams)):
            k = rng.integers(0, 40_000, size=12_000).astype(np.uint64) * np.uint64(40503) + np.uint64(j)
            g = rng.normal(0, 0.01, size=(k.size, dim)).astype(np.float32)
            with torch.cuda.stream(st):
                kd, gd = dev_keys(k), dev(g)
                out = torch.empty((k.size, dim), dtype=torch.float32, device="cuda")
                if second == "tiered" and j == 1:
                    pr.gpu.lookahead(kd)
                pr.gpu.get(kd, out)
                pr.gpu.put_grad(kd, gd, 0.01, 1e-8)
            held += [kd, gd]
            if second == "tiered" and j == 1:
                assert pr.ora.lookahead(k) == O.OK
            rc, want = pr.ora.get(k)
            assert rc == O.OK
            assert pr.ora.put_grad(k, g, 0.01, 1e-8) == O.OK
            gets.append((pr, k, out, want))
    for pr, st in zip(prs, streams):
        assert pr.gpu.sync(st) == mlkv.MLKV_OK
    for pr, k, out, want in gets:   # the rows each put changed
        pr.updated[pr.ora.lookup_rows(k)] = True
    for pr, k, out, want in gets:
        pr.compare_get(k, out.cpu().numpy(), want)
    for pr in prs:
        pr.compare_rows()
        pr.check_index()
        log(f"[streams] two streams ({second}): size {pr.ora.size} stats={pr.stats}")
        pr.close()
