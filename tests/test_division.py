"""The oracle's row-wise Adagrad step on edge values, pinned to exact
arithmetic (CPU).

At dim 1 with one position per key, the step is (fp32 operations, each
correctly rounded):

    m = RN(g^2);  G' = RN(G + m);  den = RN(RN(sqrt(G')) + eps)
    q = RN(g / den);  p = RN(lr * q);  w' = RN(w - p)

Each rounding is computed here from exact rationals (Fraction), with the
IEEE special cases written out: g / 0 is an infinity of the sign of g, 0 / 0
and inf - inf are NaN, overflow rounds to an infinity. The grid covers the
values where a division through a reciprocal goes wrong: den = 0 (eps = 0
with an underflowing m), subnormal denominators and gradients, huge
gradients whose square overflows, and ordinary values. The GPU library is
compared with the oracle on the same grid in tests/test_edge_values.py.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O

F32_MAX = Fraction(float(np.finfo(np.float32).max))
# the largest finite float32 plus half an ulp: values at or above round to inf
F32_OVF = F32_MAX + Fraction(2) ** (127 - 24)


def rn32(v) -> float:
    """Round an exact rational (or an IEEE special value) to float32, ties to even."""
    if isinstance(v, float):  # inf or nan passed through
        return float(np.float32(v))
    if v == 0:
        return 0.0
    if abs(v) >= F32_OVF:
        return math.copysign(math.inf, v)
    f = np.float32(float(v))  # within an ulp; pick the nearest of the neighbours
    cands = {f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))}
    best = None
    for c in cands:
        if not np.isfinite(c):
            continue
        d = abs(Fraction(float(c)) - v)
        key = (d, int(np.array(c).view(np.uint32)) & 1)  # on a tie the even significand wins
        if best is None or key < best[0]:
            best = (key, c)
    return float(best[1])


def add(a: float, b: float) -> float:
    if not (math.isfinite(a) and math.isfinite(b)):
        return float(np.float32(a) + np.float32(b))  # inf / nan rules
    return rn32(Fraction(a) + Fraction(b))


def mul(a: float, b: float) -> float:
    if not (math.isfinite(a) and math.isfinite(b)):
        with np.errstate(invalid="ignore"):
            return float(np.float32(a) * np.float32(b))
    return rn32(Fraction(a) * Fraction(b))


def div(a: float, b: float) -> float:
    if math.isnan(a) or math.isnan(b):
        return math.nan
    if b == 0:
        return math.nan if a == 0 else math.copysign(math.inf, a) * math.copysign(1.0, b)
    if math.isinf(a) or math.isinf(b):
        with np.errstate(invalid="ignore"):
            return float(np.float32(a) / np.float32(b))
    return rn32(Fraction(a) / Fraction(b))


def sqrt32(x: float) -> float:
    """Correctly rounded float32 square root: the float64 root of a float32
    rounds correctly to float32 (53 >= 2 * 24 + 2)."""
    if math.isnan(x) or x < 0:
        return math.nan
    return float(np.float32(math.sqrt(x)))


def adagrad_exact(w: float, G: float, g: float, lr: float, eps: float):
    lr, eps = float(np.float32(lr)), float(np.float32(eps))  # the call takes fp32 arguments
    m = rn32(Fraction(g) ** 2) if math.isfinite(g) else math.inf
    Gn = add(G, m)
    den = add(sqrt32(Gn), eps)
    q = div(g, den)
    p = mul(lr, q)
    return add(w, -p if not math.isnan(p) else math.nan), Gn


GRADS = [0.0, 1e-45, -1e-45, 1e-40, -3e-39, 1e-23, -1e-23, 1e-3, -0.02, 3e19, -1e30, 3e38]
EPS = [0.0, 1e-45, 1e-40, 1e-8]


def same(a: float, b: float) -> bool:
    return (math.isnan(a) and math.isnan(b)) or (np.float32(a).view(np.uint32) == np.float32(b).view(np.uint32))


@pytest.mark.parametrize("eps", EPS)
def test_two_adagrad_steps_on_edge_values_match_exact_arithmetic(eps):
    lr = 0.01
    g1 = np.array(GRADS, dtype=np.float32)
    g2 = np.array(GRADS[::-1], dtype=np.float32)  # the second step sees another grid order
    n = g1.size
    keys = np.arange(1, n + 1, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    t = O.OracleTable(1, 64)
    rc, w0 = t.get(keys)
    assert rc == O.OK
    assert t.put_grad(keys, g1.reshape(n, 1), lr, eps) == O.OK
    assert t.put_grad(keys, g2.reshape(n, 1), lr, eps) == O.OK
    w, G = t.read_rows(t.lookup_rows(keys))
    t.close()
    for i in range(n):
        wa, Ga = adagrad_exact(float(w0[i, 0]), 0.0, float(g1[i]), lr, eps)
        wb, Gb = adagrad_exact(wa, Ga, float(g2[i]), lr, eps)
        assert same(float(w[i, 0]), wb), (i, g1[i], g2[i], eps, w[i, 0], wb)
        assert same(float(G[i]), Gb), (i, G[i], Gb)


def test_zero_denominator_gives_signed_infinities_and_nan():
    # eps = 0 and a gradient whose square underflows: den = 0, g / den = +-inf
    # (w becomes -+inf); a zero gradient gives 0 / 0 = NaN
    t = O.OracleTable(1, 8)
    keys = np.array([11, 12, 13], dtype=np.uint64)
    t.get(keys)
    g = np.array([[1e-23], [-1e-23], [0.0]], dtype=np.float32)
    assert t.put_grad(keys, g, 0.01, 0.0) == O.OK
    w, G = t.read_rows(t.lookup_rows(keys))
    t.close()
    assert w[0, 0] == -np.inf and w[1, 0] == np.inf and np.isnan(w[2, 0])
    assert np.all(G == 0)


def test_subnormal_eps_with_zero_gradient_leaves_the_row_unchanged():
    t = O.OracleTable(4, 8)
    keys = np.array([5, 6], dtype=np.uint64)
    _, w0 = t.get(keys)
    assert t.put_grad(keys, np.zeros((2, 4), dtype=np.float32), 0.01, 1e-40) == O.OK
    w, G = t.read_rows(t.lookup_rows(keys))
    t.close()
    assert np.array_equal(w.view(np.uint32), w0.view(np.uint32)) and np.all(G == 0)
