"""ctypes binding of the CPU oracle (``liboracle.so``).

TEST INFRASTRUCTURE ONLY: the plain CPU definition of the batched embedding
get / put_grad path that the GPU library is checked against. Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import this
module. It imports nothing from the GPU library's package.

Every function follows the C definitions in ``mlkv_oracle.cpp``; see that file
for the passages of the paper (MLKV, arXiv 2504.01506) each step restates.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mlkv_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, EFULL = 0, -1, -2
DEFAULT_SEED = 0x4D4C4B56  # same documented default as the library's open call

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with g++ (no GPU code, no shared headers)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-o", _LIB + ".tmp", _SRC]
        subprocess.check_call(cmd)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    lib = ctypes.CDLL(_LIB)
    P, I32, I64, U64, F32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                             ctypes.c_uint64, ctypes.c_float)
    sig = {
        "oracle_abi_version": (ctypes.c_int, []),
        "oracle_open": (P, [I32, I64, U64]),
        "oracle_open_bounded": (P, [I32, I64, U64, I64]),
        "oracle_get_bounded": (ctypes.c_int, [P, P, I64, P, P]),
        "oracle_staleness": (ctypes.c_int, [P, P, I64, P]),
        "oracle_lookahead": (ctypes.c_int, [P, P, I64]),
        "oracle_close": (None, [P]),
        "oracle_size": (I64, [P]),
        "oracle_init_value": (F32, [U64, U64, I32]),
        "oracle_mix64": (U64, [U64]),
        "oracle_prefill_sorted": (ctypes.c_int, [P, P, I64]),
        "oracle_get": (ctypes.c_int, [P, P, I64, P]),
        "oracle_put_grad": (ctypes.c_int, [P, P, P, I64, F32, F32]),
        "oracle_put": (ctypes.c_int, [P, P, P, I64]),
        "oracle_put_grad_sgd": (ctypes.c_int, [P, P, P, I64, F32]),
        "oracle_lookup_rows": (ctypes.c_int, [P, P, I64, P]),
        "oracle_read_rows": (ctypes.c_int, [P, P, I64, P, P]),
        "oracle_row_keys": (ctypes.c_int, [P, P, I64, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _keys(keys):
    k = np.ascontiguousarray(keys, dtype=np.uint64)
    return k


def init_value(seed: int, key: int, c: int) -> float:
    return float(np.float32(_load().oracle_init_value(seed, key, c)))


def mix64(z: int) -> int:
    return int(_load().oracle_mix64(z))


class OracleTable:
    """One embedding table: plain CPU definition, single-threaded."""

    def __init__(self, dim: int, capacity: int, seed: int = DEFAULT_SEED, staleness_bound: int | None = None):
        self._lib = _load()
        self.dim = int(dim)
        self.capacity = int(capacity)
        self.seed = int(seed)
        self.staleness_bound = staleness_bound
        if staleness_bound is None:
            h = self._lib.oracle_open(self.dim, self.capacity, self.seed)
        else:
            h = self._lib.oracle_open_bounded(self.dim, self.capacity, self.seed, int(staleness_bound))
        if not h:
            raise ValueError("oracle_open rejected its arguments")
        self._h = h

    def close(self):
        if self._h:
            self._lib.oracle_close(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def size(self) -> int:
        return int(self._lib.oracle_size(self._h))

    def prefill_sorted(self, keys) -> int:
        k = _keys(keys)
        return self._lib.oracle_prefill_sorted(self._h, _ptr(k), k.size)

    def get(self, keys, want_out: bool = True):
        """Returns (rc, out[n, dim] float32 or None)."""
        k = _keys(keys)
        out = np.empty((k.size, self.dim), dtype=np.float32) if want_out else None
        rc = self._lib.oracle_get(self._h, _ptr(k), k.size, _ptr(out))
        return rc, out

    def get_bounded(self, keys, out=None):
        """Get under the staleness bound. Returns (rc, out, blocked[n] uint8);
        rows of blocked positions keep what `out` held (zeros if not given)."""
        k = _keys(keys)
        if out is None:
            out = np.zeros((k.size, self.dim), dtype=np.float32)
        out = np.ascontiguousarray(out, dtype=np.float32)
        blocked = np.zeros(k.size, dtype=np.uint8)
        rc = self._lib.oracle_get_bounded(self._h, _ptr(k), k.size, _ptr(out), _ptr(blocked))
        return rc, out, blocked

    def lookahead(self, keys) -> int:
        """Insert the missing keys ahead of their gets; no output, no counts."""
        k = _keys(keys)
        return self._lib.oracle_lookahead(self._h, _ptr(k), k.size)

    def staleness(self, rows):
        """Per-row staleness counts (gets served not yet matched by a put)."""
        r = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty(r.size, dtype=np.uint32)
        rc = self._lib.oracle_staleness(self._h, _ptr(r), r.size, _ptr(out))
        if rc != OK:
            raise ValueError(f"oracle_staleness rc={rc}")
        return out

    def put_grad(self, keys, grads, lr: float, eps: float) -> int:
        k = _keys(keys)
        g = np.ascontiguousarray(grads, dtype=np.float32)
        if g.size != k.size * self.dim:
            raise ValueError("grads must hold n * dim values")
        return self._lib.oracle_put_grad(self._h, _ptr(k), _ptr(g), k.size,
                                         ctypes.c_float(lr), ctypes.c_float(eps))


    def put(self, keys, values) -> int:
        """Batch upsert: the value at a key's last position wins."""
        k = _keys(keys)
        v = np.ascontiguousarray(values, dtype=np.float32)
        if v.size != k.size * self.dim:
            raise ValueError("values must hold n * dim values")
        return self._lib.oracle_put(self._h, _ptr(k), _ptr(v), k.size)

    def put_grad_sgd(self, keys, grads, lr: float) -> int:
        """Sum duplicate gradients, then one plain SGD step per key."""
        k = _keys(keys)
        g = np.ascontiguousarray(grads, dtype=np.float32)
        if g.size != k.size * self.dim:
            raise ValueError("grads must hold n * dim values")
        return self._lib.oracle_put_grad_sgd(self._h, _ptr(k), _ptr(g), k.size, float(lr))

    def lookup_rows(self, keys):
        k = _keys(keys)
        rows = np.empty(k.size, dtype=np.int64)
        rc = self._lib.oracle_lookup_rows(self._h, _ptr(k), k.size, _ptr(rows))
        if rc != OK:
            raise ValueError(f"oracle_lookup_rows rc={rc}")
        return rows

    def read_rows(self, rows):
        r = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty((r.size, self.dim), dtype=np.float32)
        st = np.empty(r.size, dtype=np.float32)
        rc = self._lib.oracle_read_rows(self._h, _ptr(r), r.size, _ptr(out), _ptr(st))
        if rc != OK:
            raise ValueError(f"oracle_read_rows rc={rc}")
        return out, st

    def row_keys(self, rows):
        r = np.ascontiguousarray(rows, dtype=np.int64)
        out = np.empty(r.size, dtype=np.uint64)
        rc = self._lib.oracle_row_keys(self._h, _ptr(r), r.size, _ptr(out))
        if rc != OK:
            raise ValueError(f"oracle_row_keys rc={rc}")
        return out
