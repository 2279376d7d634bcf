"""Seeded synthetic workloads shaped like the paper's embedding tables.

This module only draws inputs (keys, gradients, prefill key sets). It holds
none of the get / put_grad arithmetic, and both the GPU library's tests and
the CPU oracle's tests feed the very same arrays to each side.

The paper's datasets (Table II: Criteo, WikiKG2 / Freebase86M, Papers100M,
eBay) are not available here; these generators stand in for them with the
shapes the paper lists and skew models of the same kind:

* ``tiny``  100k-row fp32 table, dim 16, keys are a seeded 64-bit hash of the
  ids, 4096 lookups per step drawn Zipf(1.05), table starts empty.
* ``dlrm``  26 sparse features, row counts log-uniform in [1e3, 2e6] summing
  to 10M, dim 64, key = feature << 40 | id, 8192 samples x 26 features per
  step (sample-major), per-feature Zipf(1.1), table prefilled.
* ``kg``    4M entities, dim 400, per step 50k (head, tail) pairs drawn by
  power-law degree (exponent 2.1) plus 50k uniform negative tails, prefilled.
* ``gnn``   20M nodes, dim 128, 1M node ids per step drawn by power-law
  degree (exponent 2.0, degree cap tuned so about 30% of lookups repeat).
* ``large`` 200M-row capacity, dim 128, half filled, 1M keys per step drawn
  Zipf(0.99) over a 300M-id space so that about 15% of lookups miss.
* ``kv-uniform`` / ``kv-zipf``  the key-value mix of the paper's NoSQL test
  (Sec. IV: half reads, half writes, uniform or skewed access): 10M records
  of 16-byte values (dim 4) prefilled; per step 2^20 operations, the first
  half gets and the second half puts (upserts of existing records with new
  values), record ids uniform or Zipf(0.99) (the usual YCSB skew constant).

Gradients are N(0, 0.01) fp32; lr = 0.01 and eps = 1e-8 everywhere.
Every draw comes from numpy's PCG64 seeded by a SeedSequence keyed on
(base seed, config, stream kind, step), so any step can be regenerated alone.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

BASE_SEED = 0x250401506
EMPTY_KEY = np.uint64(0xFFFFFFFFFFFFFFFF)
_CFG_INDEX = {"tiny": 0, "dlrm": 1, "kg": 2, "gnn": 3, "large": 4, "kv-uniform": 5, "kv-zipf": 6}
_KIND = {"struct": 0, "keys": 1, "grads": 2, "prefill": 3, "values": 4}

M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def rng_for(cfg: str, kind: str, step: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([BASE_SEED & 0xFFFFFFFF, BASE_SEED >> 32,
                                 _CFG_INDEX[cfg], _KIND[kind], int(step)])
    return np.random.Generator(np.random.PCG64(ss))


def _splitmix_finalize(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function on a uint64 array (a bijection on 64-bit
    words; used here only to turn ids into scattered 64-bit keys and into
    per-rank coin flips)."""
    z = np.asarray(z, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= np.uint64(0xBF58476D1CE4E5B9)
        z ^= z >> np.uint64(27)
        z *= np.uint64(0x94D049BB133111EB)
        z ^= z >> np.uint64(31)
    return z


# ----------------------------------------------------------------------------
# Zipf over a finite support {1..N}, P(r) proportional to r^-s, by
# rejection-inversion (Hoermann & Derflinger 1996). Works for s < 1 too.
# ----------------------------------------------------------------------------
class ZipfSampler:
    def __init__(self, n: int, s: float):
        if n < 1 or s <= 0 or abs(s - 1.0) < 1e-12:
            raise ValueError("need n >= 1 and s > 0, s != 1")
        self.n = int(n)
        self.s = float(s)
        self._lo = self._H(1.5) - 1.0          # bottom of the accepted band for rank 1
        self._hi = self._H(self.n + 0.5)

    def _H(self, x):
        # integral of t^-s from 1 to x
        a = 1.0 - self.s
        return np.expm1(a * np.log(x)) / a

    def _Hinv(self, y):
        a = 1.0 - self.s
        return np.exp(np.log1p(a * y) / a)

    def sample(self, rng: np.random.Generator, size: int) -> np.ndarray:
        """Ranks in [1, n] (int64)."""
        out = np.empty(size, dtype=np.int64)
        filled = 0
        while filled < size:
            m = size - filled
            m = int(m * 1.1) + 16
            u = self._hi + rng.random(m) * (self._lo - self._hi)
            x = self._Hinv(u)
            k = np.floor(x + 0.5)
            k = np.clip(k, 1, self.n)
            ok = u >= self._H(k + 0.5) - np.power(k, -self.s)
            acc = k[ok].astype(np.int64)
            take = min(acc.size, size - filled)
            out[filled:filled + take] = acc[:take]
            filled += take
        return out

    @staticmethod
    def harmonic(n: int, s: float) -> float:
        """sum_{r=1..n} r^-s: exact head plus midpoint-rule integral for the tail."""
        head = min(n, 1_000_000)
        r = np.arange(1, head + 1, dtype=np.float64)
        total = float(np.sum(r ** -s))
        if n > head:
            a = 1.0 - s
            lo, hi = head + 0.5, n + 0.5
            total += (hi ** a - lo ** a) / a
        return total


def affine_bijection(rng: np.random.Generator, n: int):
    """(a * r + b) mod n with gcd(a, n) = 1: scatters hot ranks over ids."""
    if n == 1:
        return 1, 0
    while True:
        a = int(rng.integers(1, n))
        if math.gcd(a, n) == 1:
            break
    b = int(rng.integers(0, n))
    return a, b


def apply_bijection(ranks0: np.ndarray, ab, n: int) -> np.ndarray:
    a, b = ab
    r = ranks0.astype(np.uint64)
    return (r * np.uint64(a) + np.uint64(b)) % np.uint64(n)


def loguniform_sizes(rng: np.random.Generator, k: int, lo: float, hi: float, total: int) -> np.ndarray:
    """k sizes log-uniform in [lo, hi], rescaled (with clipping) to sum to total."""
    v = np.exp(rng.uniform(math.log(lo), math.log(hi), size=k))
    for _ in range(200):
        clipped = (v <= lo) | (v >= hi)
        free = ~clipped
        rest = total - v[clipped].sum()
        f = rest / v[free].sum()
        v_new = v.copy()
        v_new[free] = np.clip(v[free] * f, lo, hi)
        if np.allclose(v_new, v, rtol=0, atol=1e-9):
            break
        v = v_new
    sizes = np.floor(v).astype(np.int64)
    free = np.nonzero((sizes > lo) & (sizes < hi))[0]
    j = free[0] if free.size else int(np.argmin(sizes))
    sizes[j] += total - int(sizes.sum())
    return sizes


def powerlaw_degrees(rng: np.random.Generator, n: int, gamma: float, dmax: int) -> np.ndarray:
    u = 1.0 - rng.random(n)  # (0, 1]
    d = np.floor(u ** (-1.0 / (gamma - 1.0)))
    return np.minimum(d, dmax).astype(np.int64)


def sample_by_weight(rng: np.random.Generator, cum: np.ndarray, size: int) -> np.ndarray:
    t = rng.integers(0, int(cum[-1]), size=size)
    return np.searchsorted(cum, t, side="right").astype(np.int64)


@dataclass
class Workload:
    name: str
    dim: int
    capacity: int
    n: int                     # lookups per step
    steps: int
    lr: float = 0.01
    eps: float = 1e-8
    scale: float = 1.0
    info: dict = field(default_factory=dict)

    # -- to be provided by subclasses ------------------------------------
    def prefill_keys(self) -> np.ndarray:
        return np.empty(0, dtype=np.uint64)

    def keys(self, step: int) -> np.ndarray:
        raise NotImplementedError

    def grads(self, step: int) -> np.ndarray:
        rng = rng_for(self.name, "grads", step)
        g = rng.standard_normal(size=(self.n, self.dim), dtype=np.float32)
        g *= np.float32(0.01)
        return g


class Tiny(Workload):
    def __init__(self, scale: float = 1.0, steps: int = 10):
        super().__init__("tiny", dim=16, capacity=100_000, n=4096, steps=steps, scale=scale)
        rng = rng_for("tiny", "struct")
        self.nids = 100_000
        self.key_seed = np.uint64(int(rng.integers(0, 2**63)))
        self.zipf = ZipfSampler(self.nids, 1.05)
        self.bij = affine_bijection(rng, self.nids)
        self.info = {"ids": self.nids, "alpha": 1.05, "prefill": 0}

    def id_to_key(self, ids: np.ndarray) -> np.ndarray:
        k = _splitmix_finalize(ids.astype(np.uint64) ^ self.key_seed)
        assert not np.any(k == EMPTY_KEY)
        return k

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for("tiny", "keys", step)
        ranks = self.zipf.sample(rng, self.n)
        ids = apply_bijection(ranks - 1, self.bij, self.nids)
        return self.id_to_key(ids)


class Dlrm(Workload):
    FEATURES = 26
    SAMPLES = 8192

    def __init__(self, scale: float = 1.0, steps: int = 100):
        total = int(round(10_000_000 * scale))
        samples = max(1, int(round(self.SAMPLES * scale)))
        super().__init__("dlrm", dim=64, capacity=total, n=samples * self.FEATURES,
                         steps=steps, scale=scale)
        self.samples = samples
        rng = rng_for("dlrm", "struct")
        lo, hi = 1e3 * scale, 2e6 * scale
        lo = max(lo, 1.0)
        self.sizes = loguniform_sizes(rng, self.FEATURES, lo, hi, total)
        self.zipf = [ZipfSampler(int(s), 1.1) for s in self.sizes]
        self.bij = [affine_bijection(rng, int(s)) for s in self.sizes]
        self.info = {"features": self.FEATURES, "samples": samples, "alpha": 1.1,
                     "rows_min": int(self.sizes.min()), "rows_max": int(self.sizes.max()),
                     "prefill": total}

    def prefill_keys(self) -> np.ndarray:
        parts = [(np.uint64(f) << np.uint64(40)) | np.arange(int(s), dtype=np.uint64)
                 for f, s in enumerate(self.sizes)]
        return np.concatenate(parts)  # already ascending: feature-major, then id

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for("dlrm", "keys", step)
        out = np.empty((self.samples, self.FEATURES), dtype=np.uint64)
        for f in range(self.FEATURES):
            ranks = self.zipf[f].sample(rng, self.samples)
            ids = apply_bijection(ranks - 1, self.bij[f], int(self.sizes[f]))
            out[:, f] = (np.uint64(f) << np.uint64(40)) | ids
        return out.reshape(-1)  # sample-major


class Kg(Workload):
    def __init__(self, scale: float = 1.0, steps: int = 50):
        nent = int(round(4_000_000 * scale))
        edges = max(1, int(round(50_000 * scale)))
        super().__init__("kg", dim=400, capacity=nent, n=3 * edges, steps=steps, scale=scale)
        self.nent = nent
        self.edges = edges
        rng = rng_for("kg", "struct")
        deg = powerlaw_degrees(rng, nent, 2.1, nent)
        self.cum = np.cumsum(deg)
        self.info = {"entities": nent, "edges": edges, "gamma": 2.1,
                     "max_degree": int(deg.max()), "prefill": nent}

    def prefill_keys(self) -> np.ndarray:
        return np.arange(self.nent, dtype=np.uint64)

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for("kg", "keys", step)
        h = sample_by_weight(rng, self.cum, self.edges)
        t = sample_by_weight(rng, self.cum, self.edges)
        neg = rng.integers(0, self.nent, size=self.edges)
        return np.stack([h, t, neg], axis=1).reshape(-1).astype(np.uint64)


class Gnn(Workload):
    DMAX = 700

    def __init__(self, scale: float = 1.0, steps: int = 20):
        nodes = int(round(20_000_000 * scale))
        n = max(1, int(round(1_000_000 * scale)))
        super().__init__("gnn", dim=128, capacity=nodes, n=n, steps=steps, scale=scale)
        self.nodes = nodes
        rng = rng_for("gnn", "struct")
        deg = powerlaw_degrees(rng, nodes, 2.0, self.DMAX)
        self.cum = np.cumsum(deg)
        self.info = {"nodes": nodes, "gamma": 2.0, "dmax": self.DMAX, "prefill": nodes}

    def prefill_keys(self) -> np.ndarray:
        return np.arange(self.nodes, dtype=np.uint64)

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for("gnn", "keys", step)
        return sample_by_weight(rng, self.cum, self.n).astype(np.uint64)


class Large(Workload):
    ALPHA = 0.99

    def __init__(self, scale: float = 1.0, steps: int = 20, target_miss: float = 0.15):
        cap = int(round(200_000_000 * scale))
        space = int(round(300_000_000 * scale))
        fill = int(round(100_000_000 * scale))
        n = max(1, int(round(1_000_000 * scale)))
        super().__init__("large", dim=128, capacity=cap, n=n, steps=steps, scale=scale)
        self.space = space
        self.fill = fill
        rng = rng_for("large", "struct")
        self.zipf = ZipfSampler(space, self.ALPHA)
        self.bij = affine_bijection(rng, space)
        self.coin_seed = np.uint64(int(rng.integers(0, 2**63)))
        self.head = self._choose_head(target_miss)
        self.q = (fill - self.head) / (space - self.head)
        self.info = {"id_space": space, "alpha": self.ALPHA, "prefill_target": fill,
                     "hot_head": self.head, "coin_q": self.q,
                     "expected_miss": self._miss(self.head)}

    def _miss(self, k: int) -> float:
        hn = ZipfSampler.harmonic(self.space, self.ALPHA)
        hk = ZipfSampler.harmonic(k, self.ALPHA) if k > 0 else 0.0
        q = (self.fill - k) / (self.space - k)
        return (1.0 - hk / hn) * (1.0 - q)

    def _choose_head(self, target: float) -> int:
        lo, hi = 1, self.fill
        for _ in range(60):
            mid = (lo + hi) // 2
            if self._miss(mid) > target:
                lo = mid + 1
            else:
                hi = mid
            if lo >= hi:
                break
        return lo

    def _coin(self, ranks0: np.ndarray) -> np.ndarray:
        h = _splitmix_finalize(ranks0.astype(np.uint64) ^ self.coin_seed)
        return (h >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)

    def prefill_keys(self) -> np.ndarray:
        parts = []
        chunk = 10_000_000
        for start in range(0, self.space, chunk):
            r0 = np.arange(start, min(start + chunk, self.space), dtype=np.int64)
            keep = (r0 < self.head) | (self._coin(r0) < self.q)
            parts.append(apply_bijection(r0[keep], self.bij, self.space))
        ids = np.concatenate(parts)
        ids.sort()
        return ids

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for("large", "keys", step)
        ranks = self.zipf.sample(rng, self.n)
        return apply_bijection(ranks - 1, self.bij, self.space)


class KvMix(Workload):
    """Half gets, half puts over prefilled records: keys(step)[:n // 2] are
    read, keys(step)[n // 2:] are written with values(step)."""

    ALPHA = 0.99

    def __init__(self, skew: str, scale: float = 1.0, steps: int = 100):
        name = f"kv-{skew}"
        records = max(1000, int(round(10_000_000 * scale)))
        n = max(2, int(round((1 << 20) * scale)) // 2 * 2)
        super().__init__(name, dim=4, capacity=records, n=n, steps=steps, scale=scale)
        rng = rng_for(name, "struct")
        self.records = records
        self.key_seed = np.uint64(int(rng.integers(0, 2**63)))
        self.zipf = ZipfSampler(records, self.ALPHA) if skew == "zipf" else None
        self.bij = affine_bijection(rng, records)
        self.info = {"records": records, "skew": skew, "alpha": self.ALPHA if self.zipf else 0.0,
                     "reads": n // 2, "writes": n - n // 2}

    def id_to_key(self, ids: np.ndarray) -> np.ndarray:
        k = _splitmix_finalize(ids.astype(np.uint64) ^ self.key_seed)
        assert not np.any(k == EMPTY_KEY)
        return k

    def prefill_keys(self) -> np.ndarray:
        return np.sort(self.id_to_key(np.arange(self.records, dtype=np.int64)))

    def keys(self, step: int) -> np.ndarray:
        rng = rng_for(self.name, "keys", step)
        if self.zipf is None:
            ids = rng.integers(0, self.records, size=self.n)
        else:
            ids = apply_bijection(self.zipf.sample(rng, self.n) - 1, self.bij, self.records)
        return self.id_to_key(ids)

    def values(self, step: int) -> np.ndarray:
        rng = rng_for(self.name, "values", step)
        return rng.standard_normal(size=(self.n - self.n // 2, self.dim), dtype=np.float32)


class KvUniform(KvMix):
    def __init__(self, scale: float = 1.0, steps: int = 100):
        super().__init__("uniform", scale, steps)


class KvZipf(KvMix):
    def __init__(self, scale: float = 1.0, steps: int = 100):
        super().__init__("zipf", scale, steps)


CONFIGS = {"tiny": Tiny, "dlrm": Dlrm, "kg": Kg, "gnn": Gnn, "large": Large,
           "kv-uniform": KvUniform, "kv-zipf": KvZipf}


def make(name: str, scale: float = 1.0, steps: int | None = None) -> Workload:
    cls = CONFIGS[name]
    if steps is None:
        return cls(scale=scale)
    return cls(scale=scale, steps=steps)
