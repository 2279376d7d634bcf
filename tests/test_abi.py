"""The C ABI library loads, exports every symbol the header declares, and
rejects bad arguments on the host (no GPU needed for any of this)."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mlkv.h")
LIB = os.path.join(ROOT, "paper_2504_01506_amd", "libmlkv.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mlkv_[a-z_]+)\s*\(", src)))


def test_header_declares_the_calls():
    names = declared_functions()
    for want in ("mlkv_open", "mlkv_get", "mlkv_put_grad", "mlkv_sync", "mlkv_close"):
        assert want in names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2504_01506_amd import build
        build.build()
    from paper_2504_01506_amd import mlkv
    return mlkv.load()


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (mlkv_[a-z_]+)", out))
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    for f in declared_functions():
        assert hasattr(lib, f)


def test_binding_exposes_the_same_names(lib):
    from paper_2504_01506_amd import mlkv
    for f in declared_functions():
        assert callable(getattr(mlkv, f)), f


def test_host_side_validation_without_a_gpu(lib):
    from paper_2504_01506_amd import mlkv
    assert lib.mlkv_open(0, 10) is None
    assert "dim" in mlkv.last_error()
    assert lib.mlkv_open(16, 0) is None
    assert lib.mlkv_open(16, 2**32) is None
    assert lib.mlkv_open_ex(16, 100, 1, 0.0) is None
    assert lib.mlkv_open_ex(16, 100, 1, float("nan")) is None
    assert lib.mlkv_open_ex(2000, 100, 1, 0.5) is None
    assert lib.mlkv_get(None, None, 10, None, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_put_grad(None, None, None, 10, 0.1, 0.0, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_sync(None, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_size(None) == -1
    assert lib.mlkv_num_slots(None) == -1
    assert lib.mlkv_open_bounded(16, 100, 1, 0.5, -1) is None
    assert "staleness_bound" in mlkv.last_error()
    assert lib.mlkv_open_bounded(16, 100, 1, 0.5, 2**24 - 1) is None
    assert lib.mlkv_get_bounded(None, None, 10, None, None, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_read_staleness(None, None, 10, None, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_lookahead(None, None, 10, None) == mlkv.MLKV_EINVAL
    assert lib.mlkv_get_put_grad(None, None, 10, None, None, None, None, 10, 0.1, 0.0, None, None) == mlkv.MLKV_EINVAL
    lib.mlkv_close(None)  # no-op


def test_single_hip_runtime_in_process(lib):
    from paper_2504_01506_amd import mlkv
    rts = mlkv.hip_runtimes_loaded()
    assert len(rts) <= 1, rts
