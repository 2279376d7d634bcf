"""ctypes binding of libmlkv.so (see include/mlkv.h for the contract).

Functions carry the C names and only marshal arguments: torch tensors are
passed as device pointers and torch streams as hipStream_t. Every step of the
get / put_grad path runs in the library's HIP kernels; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loads the HIP runtime that libmlkv binds to (same soname)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmlkv.so")

MLKV_OK, MLKV_EINVAL, MLKV_EFULL, MLKV_ENOMEM, MLKV_EDEVICE = 0, -1, -2, -3, -4
MLKV_DEFAULT_SEED = 0x4D4C4B56
MLKV_RESERVED_KEY = 0xFFFFFFFFFFFFFFFF

MLKV_NUM_KERNELS = 10
MLKV_DEDUP_HASH, MLKV_DEDUP_RADIX = 0, 1
DEDUP_MODES = {"hash": MLKV_DEDUP_HASH, "radix": MLKV_DEDUP_RADIX}
MLKV_NOALLOC_MAX_KEYS = 65536

_lib = None


class MlkvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


def load() -> ctypes.CDLL:
    """Loads libmlkv.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(or python paper_2504_01506_amd/build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, F32, INT = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_float, ctypes.c_int)
    sig = {
        "mlkv_open": (P, [I32, I64]),
        "mlkv_open_ex": (P, [I32, I64, U64, F32]),
        "mlkv_open_bounded": (P, [I32, I64, U64, F32, I64]),
        "mlkv_open_tiered": (P, [I32, I64, U64, F32, I64]),
        "mlkv_cache_stats": (INT, [P, P]),
        "mlkv_get": (INT, [P, P, I64, P, P]),
        "mlkv_get_bounded": (INT, [P, P, I64, P, P, P]),
        "mlkv_get_noalloc": (INT, [P, P, I64, P, P]),
        "mlkv_lookahead": (INT, [P, P, I64, P]),
        "mlkv_read_staleness": (INT, [P, P, I64, P, P]),
        "mlkv_put_grad": (INT, [P, P, P, I64, F32, F32, P]),
        "mlkv_put_grad_sgd": (INT, [P, P, P, I64, F32, P]),
        "mlkv_get_put_grad": (INT, [P, P, I64, P, P, P, P, I64, F32, F32, P, P]),
        "mlkv_put": (INT, [P, P, P, I64, P]),
        "mlkv_sync": (INT, [P, P]),
        "mlkv_size": (I64, [P]),
        "mlkv_num_slots": (I64, [P]),
        "mlkv_reserve": (INT, [P, I64]),
        "mlkv_set_dedup": (INT, [P, INT]),
        "mlkv_close": (None, [P]),
        "mlkv_last_error": (ctypes.c_char_p, []),
        "mlkv_lookup_rows": (INT, [P, P, I64, P, P]),
        "mlkv_export": (INT, [P, I64, P, P, P, P, P]),
        "mlkv_read_rows": (INT, [P, P, I64, P, P, P]),
        "mlkv_profile_enable": (INT, [P, INT]),
        "mlkv_profile_read": (INT, [P, P, P]),
        "mlkv_kernel_name": (ctypes.c_char_p, [INT]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def hip_runtimes_loaded() -> list[str]:
    """Paths of every libamdhip64 mapped into this process (must be exactly one)."""
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            if "libamdhip64" in line:
                paths.add(line.split()[-1])
    return sorted(paths)


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def last_error() -> str:
    return load().mlkv_last_error().decode()


def _check(rc: int):
    if rc != MLKV_OK:
        raise MlkvError(rc, last_error())


# ---- the C calls, same names ------------------------------------------------
def mlkv_open(dim: int, capacity: int) -> int:
    h = load().mlkv_open(dim, capacity)
    if not h:
        raise MlkvError(MLKV_EINVAL, last_error())
    return h


def mlkv_open_ex(dim: int, capacity: int, seed: int, max_load: float) -> int:
    h = load().mlkv_open_ex(dim, capacity, seed, max_load)
    if not h:
        raise MlkvError(MLKV_EINVAL, last_error())
    return h


def mlkv_open_bounded(dim: int, capacity: int, seed: int, max_load: float, staleness_bound: int) -> int:
    h = load().mlkv_open_bounded(dim, capacity, seed, max_load, staleness_bound)
    if not h:
        raise MlkvError(MLKV_EINVAL, last_error())
    return h


def mlkv_open_tiered(dim: int, capacity: int, seed: int, max_load: float, cache_rows: int) -> int:
    h = load().mlkv_open_tiered(dim, capacity, seed, max_load, cache_rows)
    if not h:
        raise MlkvError(MLKV_EINVAL, last_error())
    return h


def mlkv_cache_stats(t: int) -> dict:
    """{loaded, evicted, written_back, filled, cache_rows} of a tiered table."""
    out = (ctypes.c_int64 * 5)()
    _check(load().mlkv_cache_stats(t, out))
    return dict(zip(("loaded", "evicted", "written_back", "filled", "cache_rows"), list(out)))


def mlkv_get(t: int, keys, n: int, out, stream=None) -> int:
    return load().mlkv_get(t, _ptr(keys), n, _ptr(out), _stream(stream))


def mlkv_get_noalloc(t: int, keys, n: int, out, stream=None) -> int:
    return load().mlkv_get_noalloc(t, _ptr(keys), n, _ptr(out), _stream(stream))


def mlkv_get_bounded(t: int, keys, n: int, out, blocked, stream=None) -> int:
    return load().mlkv_get_bounded(t, _ptr(keys), n, _ptr(out), _ptr(blocked), _stream(stream))


def mlkv_lookahead(t: int, keys, n: int, stream=None) -> int:
    return load().mlkv_lookahead(t, _ptr(keys), n, _stream(stream))


def mlkv_read_staleness(t: int, rows, n: int, out, stream=None) -> int:
    return load().mlkv_read_staleness(t, _ptr(rows), n, _ptr(out), _stream(stream))


def mlkv_put_grad(t: int, keys, grads, n: int, lr: float, eps: float, stream=None) -> int:
    return load().mlkv_put_grad(t, _ptr(keys), _ptr(grads), n, lr, eps, _stream(stream))


def mlkv_get_put_grad(t: int, get_keys, n_get: int, out, blocked, put_keys, grads, n_put: int, lr: float,
                      eps: float, get_done=None, stream=None) -> int:
    ev = None
    if get_done is not None:  # a torch.cuda.Event: its hipEvent_t exists once it has been recorded
        if not get_done.cuda_event:
            get_done.record()
        ev = get_done.cuda_event
    return load().mlkv_get_put_grad(t, _ptr(get_keys), n_get, _ptr(out), _ptr(blocked), _ptr(put_keys),
                                    _ptr(grads), n_put, lr, eps, ev, _stream(stream))


def mlkv_put_grad_sgd(t: int, keys, grads, n: int, lr: float, stream=None) -> int:
    return load().mlkv_put_grad_sgd(t, _ptr(keys), _ptr(grads), n, lr, _stream(stream))


def mlkv_put(t: int, keys, values, n: int, stream=None) -> int:
    return load().mlkv_put(t, _ptr(keys), _ptr(values), n, _stream(stream))


def mlkv_sync(t: int, stream=None) -> int:
    return load().mlkv_sync(t, _stream(stream))


def mlkv_size(t: int) -> int:
    return load().mlkv_size(t)


def mlkv_num_slots(t: int) -> int:
    return load().mlkv_num_slots(t)


def mlkv_reserve(t: int, n: int) -> int:
    return load().mlkv_reserve(t, n)


def mlkv_set_dedup(t: int, mode: int) -> int:
    return load().mlkv_set_dedup(t, mode)


def mlkv_close(t: int) -> None:
    load().mlkv_close(t)


def mlkv_last_error() -> str:
    return last_error()


def mlkv_lookup_rows(t: int, keys, n: int, rows_out, stream=None) -> int:
    return load().mlkv_lookup_rows(t, _ptr(keys), n, _ptr(rows_out), _stream(stream))


def mlkv_export(t: int, nrows: int, rows_out=None, state_out=None, slot_keys_out=None,
                slot_rows_out=None, stream=None) -> int:
    return load().mlkv_export(t, nrows, _ptr(rows_out), _ptr(state_out), _ptr(slot_keys_out),
                              _ptr(slot_rows_out), _stream(stream))


def mlkv_read_rows(t: int, rows, n: int, rows_out=None, state_out=None, stream=None) -> int:
    return load().mlkv_read_rows(t, _ptr(rows), n, _ptr(rows_out), _ptr(state_out), _stream(stream))


def mlkv_profile_enable(t: int, enable: bool) -> int:
    return load().mlkv_profile_enable(t, 1 if enable else 0)


def mlkv_profile_read(t: int):
    """{kernel name: (total ms, launches)} of the launches since the last read."""
    ms = (ctypes.c_double * MLKV_NUM_KERNELS)()
    cnt = (ctypes.c_int64 * MLKV_NUM_KERNELS)()
    _check(load().mlkv_profile_read(t, ms, cnt))
    return {mlkv_kernel_name(k): (ms[k], cnt[k]) for k in range(MLKV_NUM_KERNELS)}


def mlkv_kernel_name(kernel: int) -> str:
    r = load().mlkv_kernel_name(kernel)
    return r.decode() if r else None


# ---- a small object wrapper over the same calls -----------------------------
class Table:
    """One embedding table on the current GPU. Keys are uint64 (stored in an
    int64 tensor), rows fp32. Methods raise MlkvError on a non-zero code."""

    def __init__(self, dim: int, capacity: int, seed: int = MLKV_DEFAULT_SEED, max_load: float = 0.75,
                 staleness_bound: int | None = None, cache_rows: int | None = None, dedup: str = "hash"):
        self.dim = int(dim)
        self.capacity = int(capacity)
        self.staleness_bound = staleness_bound
        self.cache_rows = cache_rows
        if staleness_bound is not None and cache_rows is not None:
            raise ValueError("a table is either bounded or tiered here")
        if cache_rows is not None:
            self.h = mlkv_open_tiered(self.dim, self.capacity, seed, max_load, int(cache_rows))
        elif staleness_bound is None:
            self.h = mlkv_open_ex(self.dim, self.capacity, seed, max_load)
        else:
            self.h = mlkv_open_bounded(self.dim, self.capacity, seed, max_load, int(staleness_bound))
        if dedup != "hash":
            self.set_dedup(dedup)

    def set_dedup(self, mode: str):
        """How puts find equal keys: "hash" (partition + LDS grouping) or "radix"
        (radix sort by row + run-length encoding); results are the same."""
        _check(mlkv_set_dedup(self.h, DEDUP_MODES[mode]))

    def close(self):
        if self.h:
            mlkv_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def get(self, keys: torch.Tensor, out: torch.Tensor | None = None, stream=None):
        _check(mlkv_get(self.h, keys, keys.numel(), out, stream))
        return out

    def get_bounded(self, keys: torch.Tensor, out: torch.Tensor | None = None,
                    blocked: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """Get under the table's staleness bound; returns the uint8 blocked flags."""
        if blocked is None:
            blocked = torch.empty(keys.numel(), dtype=torch.uint8, device=keys.device)
        _check(mlkv_get_bounded(self.h, keys, keys.numel(), out, blocked, stream))
        return blocked

    def lookahead(self, keys: torch.Tensor, stream=None):
        """Insert the missing keys ahead of their gets (no output, no staleness count);
        on a tiered table, also bring their rows into the HBM cache."""
        _check(mlkv_lookahead(self.h, keys, keys.numel(), stream))

    def cache_stats(self) -> dict:
        return mlkv_cache_stats(self.h)

    def read_staleness(self, rows: torch.Tensor, stream=None) -> torch.Tensor:
        """Staleness counts (int32 view of uint32) of the given row ids (int64)."""
        out = torch.empty(rows.numel(), dtype=torch.int32, device=rows.device)
        _check(mlkv_read_staleness(self.h, rows, rows.numel(), out, stream))
        return out

    def put_grad(self, keys: torch.Tensor, grads: torch.Tensor, lr: float, eps: float, stream=None):
        _check(mlkv_put_grad(self.h, keys, grads, keys.numel(), lr, eps, stream))

    def get_put_grad(self, get_keys: torch.Tensor, out: torch.Tensor | None, put_keys: torch.Tensor,
                     grads: torch.Tensor, lr: float, eps: float, blocked: torch.Tensor | None = None,
                     get_done: torch.cuda.Event | None = None, stream=None):
        """The get of get_keys, then put_grad of put_keys, in one call (every put
        key must be in the table before the call); get_done, if given, is
        recorded once the rows are in `out`. Returns the blocked flags on a
        table with a staleness bound, else None."""
        if blocked is None and self.staleness_bound is not None:
            blocked = torch.empty(get_keys.numel(), dtype=torch.uint8, device=get_keys.device)
        _check(mlkv_get_put_grad(self.h, get_keys, get_keys.numel(), out, blocked, put_keys, grads,
                                 put_keys.numel(), lr, eps, get_done, stream))
        return blocked

    def put_grad_sgd(self, keys: torch.Tensor, grads: torch.Tensor, lr: float, stream=None):
        _check(mlkv_put_grad_sgd(self.h, keys, grads, keys.numel(), lr, stream))

    def put(self, keys: torch.Tensor, values: torch.Tensor, stream=None):
        _check(mlkv_put(self.h, keys, values, keys.numel(), stream))

    def sync(self, stream=None) -> int:
        return mlkv_sync(self.h, stream)

    @property
    def size(self) -> int:
        return mlkv_size(self.h)

    def reserve(self, n: int):
        """Size the per-call scratch for calls of up to n keys (no allocation on later calls)."""
        _check(mlkv_reserve(self.h, int(n)))

    @property
    def num_slots(self) -> int:
        return mlkv_num_slots(self.h)

    def lookup_rows(self, keys: torch.Tensor, stream=None) -> torch.Tensor:
        out = torch.empty(keys.numel(), dtype=torch.int64, device=keys.device)
        _check(mlkv_lookup_rows(self.h, keys, keys.numel(), out, stream))
        return out

    def read_rows(self, rows: torch.Tensor, stream=None):
        """(values[len(rows), dim], accumulators[len(rows)]) of the given row ids (int64)."""
        w = torch.empty((rows.numel(), self.dim), dtype=torch.float32, device=rows.device)
        st = torch.empty(rows.numel(), dtype=torch.float32, device=rows.device)
        _check(mlkv_read_rows(self.h, rows, rows.numel(), w, st, stream))
        return w, st

    def export(self, nrows: int | None = None, stream=None):
        """(rows[nrows, dim], state[nrows], slot_keys[num_slots] int64, slot_rows[num_slots] int32)."""
        if nrows is None:
            nrows = self.size
        dev = torch.device("cuda", torch.cuda.current_device())
        rows = torch.empty((nrows, self.dim), dtype=torch.float32, device=dev)
        st = torch.empty(nrows, dtype=torch.float32, device=dev)
        ns = self.num_slots
        sk = torch.empty(ns, dtype=torch.int64, device=dev)
        sr = torch.empty(ns, dtype=torch.int32, device=dev)
        _check(mlkv_export(self.h, nrows, rows, st, sk, sr, stream))
        return rows, st, sk, sr
