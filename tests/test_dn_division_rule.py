"""The fast binary32 division behind the projection of normalized data, checked exactly.

The device normalizes a = fl32(x - mean) by den = fl32(std + 1e-7) without the IEEE
division sequence: with rd = fl32(1/den), q = fl32(a rd), the residual a - den q (exact
in one fma) and the result fl32(q + residual rd) (one fma).  Markstein's theorem (IBM J.
Res. Develop. 34(1), 1990) makes that the correctly rounded a/den when nothing underflows
or overflows; the device uses it for den in [2^-24, 2^24] and 2^-100 <= |a| <= 2^100.
Here the two fmas are evaluated in exact rational arithmetic and compared with numpy's
IEEE binary32 division, on cases built to put a/den next to a rounding boundary (a the
rounding of den times a midpoint between floats, and its neighbours) and on random ones,
at the ends of the ranges too.
"""
from fractions import Fraction

import numpy as np


def rn32(v):
    """Round a Fraction to binary32, to nearest, ties to even (normal range only)."""
    f = np.float32(float(v))   # float() rounds once to fp64; fix up below
    # search the neighbours of the fp64-then-fp32 guess for the exact nearest
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = None
    for c in cands:
        d = abs(Fraction(float(c)) - v)
        key = (d, int(np.array([c]).view(np.uint32)[0]) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def fast_div(a, den):
    a, den = np.float32(a), np.float32(den)
    rd = np.float32(1.0) / den
    q = np.float32(a * rd)
    r = rn32(Fraction(float(a)) - Fraction(float(den)) * Fraction(float(q)))
    return rn32(Fraction(float(q)) + Fraction(float(r)) * Fraction(float(rd)))


def cases():
    rng = np.random.default_rng(1234)
    out = []
    for _ in range(1500):
        den = np.float32(rng.uniform(1.0, 2.0))
        if rng.integers(4) == 0:
            den = np.float32(2.0) - np.float32(rng.integers(1, 256)) * np.float32(2.0 ** -23)
        m = 1.0 + float(int(rng.integers(0, 2 ** 24)) | 1) / 2.0 ** 24   # a midpoint
        a = np.float32(float(den) * m)
        for sa, sd in [(0, 0), (int(rng.integers(-99, 99)), int(rng.integers(-24, 24))),
                       (-99, 24), (99, -24), (-99, -24)]:
            for aa in (a, np.nextafter(a, np.float32(0)), np.nextafter(a, np.float32(4))):
                out.append((np.float32(np.ldexp(aa, sa)), np.float32(np.ldexp(den, sd))))
    for _ in range(3000):
        a = np.float32(rng.uniform(1, 2) * 2.0 ** rng.integers(-100, 99)) * (1 - 2 * rng.integers(2))
        den = np.float32(rng.uniform(1, 2) * 2.0 ** rng.integers(-24, 23))
        out.append((a, den))
    return out


def test_fast_division_is_correctly_rounded():
    n = 0
    with np.errstate(all="ignore"):
        for a, den in cases():
            ad = abs(float(a))
            if not (2.0 ** -100 <= ad <= 2.0 ** 100 and 2.0 ** -24 <= float(den) <= 2.0 ** 24):
                continue
            want = np.float32(a) / np.float32(den)
            got = fast_div(a, den)
            assert got == want, (a, den, got, want)
            n += 1
    assert n > 15000
