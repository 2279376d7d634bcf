"""The Adagrad kernels divide a row by one denominator through a correctly
rounded reciprocal y = RN(1/den) and one FMA correction per element:

    q0 = RN(g * y);  r = RN(g - den * q0);  q = RN(q0 + r * y)

(r and q each from one FMA, a single rounding). By Markstein's analysis of
this correction step, q = RN(g / den) when nothing underflows or overflows.
These CPU tests check that with exact rational arithmetic, on float32 inputs
of the kind the kernels see (gradient sums, denominators sqrt(G) + eps), on
adversarial significands and on random bit patterns; the oracle divides
directly.
"""
from fractions import Fraction

import numpy as np


def rn32(v: Fraction) -> np.float32:
    """Round an exact rational to the nearest float32, ties to even."""
    f = np.float32(float(v))
    cands = {f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))}
    best = None
    for c in cands:
        d = abs(Fraction(float(c)) - v)
        key = (d, int(np.array(c).view(np.uint32)) & 1)  # on a tie the even significand wins
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def markstein(g: np.float32, den: np.float32) -> np.float32:
    y = rn32(Fraction(1) / Fraction(float(den)))
    q0 = rn32(Fraction(float(g)) * Fraction(float(y)))
    r = rn32(Fraction(float(g)) - Fraction(float(den)) * Fraction(float(q0)))  # one FMA
    return rn32(Fraction(float(q0)) + Fraction(float(r)) * Fraction(float(y)))  # one FMA


def direct(g, den):
    return rn32(Fraction(float(g)) / Fraction(float(den)))


def test_random_gradient_like_quotients():
    rng = np.random.default_rng(0)
    g = (rng.normal(0, 0.01, 3000) * rng.choice([1, 3, 30], 3000)).astype(np.float32)
    den = (np.sqrt(rng.uniform(1e-6, 1.0, 3000)) + 1e-8).astype(np.float32)
    for a, b in zip(g, den):
        assert markstein(a, b) == direct(a, b), (a, b)


def test_adversarial_significands():
    # all-ones and near-power-of-two significands, where reciprocals round badly
    sig = [1.0, 1.0 + 2 ** -23, 2.0 - 2 ** -23, 1.5, 1.0 + 2 ** -12, 2.0 - 2 ** -12, 1.3333333, 1.9999999]
    vals = [np.float32(s * 2.0 ** e) for s in sig for e in (-20, -7, -1, 0, 3)]
    for a in vals:
        for b in vals:
            for sgn in (1, -1):
                aa = np.float32(sgn * a)
                assert markstein(aa, b) == direct(aa, b), (aa, b)


def test_random_bit_patterns():
    rng = np.random.default_rng(1)
    # significands uniformly random, exponents in the range the update meets
    for _ in range(3000):
        a = np.float32(rng.uniform(1, 2) * 2.0 ** int(rng.integers(-30, 10)))
        b = np.float32(rng.uniform(1, 2) * 2.0 ** int(rng.integers(-15, 5)))
        assert markstein(a, b) == direct(a, b), (a, b)
