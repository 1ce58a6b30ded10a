"""Pins of the oracle's projection (eq. (6)-(8)) against brute-force nearest
search, the paper's worked example, constructed ties, special values and the
textbook special cases (fixed point, powers of two)."""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK, TABLE1_BK, read_golden

ALPHAS = [1.0, 0.37, 2.0 ** -5, 1.7e-3, 3.1]


def decode_codes(codes, b, ks):
    table = np.array([oracle.decode(c, b, ks) for c in range(256)])
    return table[codes]


def special_inputs():
    f = np.float32
    vals = [0.0, -0.0, np.inf, -np.inf, np.nan, f(1e-45), f(-1e-45), f(1.17e-38), f(3.4e38),
            f(-3.4e38), f(0.5), f(-0.5), f(1.5), f(-2.5)]
    return np.array(vals, dtype=np.float32)


def random_bit_patterns(seed, n):
    r = np.random.default_rng([7, seed])
    return r.integers(0, 2 ** 32, size=n, dtype=np.uint64).astype(np.uint32).view(np.float32)


def midpoint_inputs(b, ks):
    """Exact midpoints between neighbouring set values and their fp32 neighbours."""
    v = oracle.valueset(b, ks)
    mids = ((v[1:] + v[:-1]) / 2).astype(np.float32)
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(-np.inf))
    m = np.concatenate([mids, up, dn, v.astype(np.float32)])
    return np.concatenate([m, -m])


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_project_equals_bruteforce(b, ks):
    x = np.concatenate([random_bit_patterns(b * 10 + ks, 20000), special_inputs(),
                        midpoint_inputs(b, ks),
                        np.random.default_rng(b).standard_normal(20000).astype(np.float32) * 3])
    for alpha in ALPHAS:
        a = oracle.project(x, alpha, b, ks)
        bf = oracle.project_bruteforce(x, alpha, b, ks)
        np.testing.assert_array_equal(a, bf)


@pytest.mark.parametrize("b,ks", TABLE1_BK)
def test_scaled_midpoints_tie_to_larger_magnitude(b, ks):
    """Constructed ties: alpha a power of two, so x/alpha is exactly a midpoint."""
    v = oracle.valueset(b, ks)
    alpha = 2.0 ** -3
    mids = (v[1:] + v[:-1]) / 2
    x = (mids * alpha).astype(np.float32)
    q = decode_codes(oracle.project(x, alpha, b, ks), b, ks)
    np.testing.assert_array_equal(q, v[1:])
    qn = decode_codes(oracle.project(-x, alpha, b, ks), b, ks)
    np.testing.assert_array_equal(qn, -v[1:])


def test_paper_projection_example():
    for b, k, v, pv in read_golden("projection_example.txt"):
        b, k, v, pv = int(b), int(k), float(v), float(pv)
        assert oracle.project_value(np.float32(v), 1.0, b, k + 1) == pv


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_special_values(b, ks):
    C = oracle.C(b, ks)
    pv = lambda x, a=1.0: oracle.project_value(x, a, b, ks)
    assert pv(np.inf) == C and pv(-np.inf) == -C
    assert pv(3.4e38) == C
    s = pv(np.nan)
    assert s == 0.0 and not np.signbit(s)
    s = pv(-0.0)
    assert s == 0.0 and not np.signbit(s)
    assert pv(1e-45) == 0.0
    # invalid scales give +0
    for a in [0.0, -1.0, np.inf, np.nan]:
        assert pv(1.0, a) == 0.0
    # sign symmetry
    x = np.random.default_rng(3).standard_normal(2000).astype(np.float32) * 4
    pos = decode_codes(oracle.project(x, 0.7, b, ks), b, ks)
    neg = decode_codes(oracle.project(-x, 0.7, b, ks), b, ks)
    np.testing.assert_array_equal(pos, -neg)


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_idempotent_and_monotone(b, ks):
    alpha = 2.0 ** -2
    codes = np.arange(2 ** b, dtype=np.uint8)
    deq = oracle.dequantize(codes, alpha, b, ks)
    back = oracle.project(deq, alpha, b, ks)
    canon = np.array([oracle.encode(oracle.decode(c, b, ks), b, ks) for c in codes])
    np.testing.assert_array_equal(back, canon)
    x = np.sort(np.random.default_rng(5).standard_normal(5000).astype(np.float32) * 5)
    q = decode_codes(oracle.project(x, 0.9, b, ks), b, ks)
    assert np.all(np.diff(q) >= 0)


@pytest.mark.parametrize("b", range(2, 9))
def test_fixed_point_special_case(b):
    """k = b-2 is linear quantization: truncate to [-C, C] then round (Sec. 3.1)."""
    k = b - 2
    x = np.random.default_rng(b).standard_normal(20000).astype(np.float32) * 2
    alpha = np.float32(0.3)
    v = (x / alpha).astype(np.float32).astype(np.float64)
    C = (2 ** (b - 1) - 1) / 2.0 ** k
    a = np.minimum(np.abs(v), C)
    expect = np.sign(v) * np.floor(a * 2 ** k + 0.5) / 2 ** k
    q = decode_codes(oracle.project(x, alpha, b, k + 1), b, k + 1)
    np.testing.assert_array_equal(q, expect + 0.0)


@pytest.mark.parametrize("b", range(2, 7))
def test_power_of_two_special_case(b):
    """k = 0: nearest of {0, 1, 2, 4, ...}; the cell boundaries are 0.5 and 1.5 * 2^e."""
    x = np.abs(np.random.default_rng(b).standard_normal(20000)).astype(np.float32) * 6
    top = 2 ** (2 ** (b - 1) - 2)
    a = np.minimum(x.astype(np.float64), top)
    e = np.floor(np.log2(np.maximum(a, 1e-300)))
    p = 2.0 ** e
    expect = np.where(a < 0.5, 0.0, np.where(a < 1.0, 1.0, np.where(a >= 1.5 * p, 2 * p, p)))
    expect = np.minimum(expect, top)
    q = decode_codes(oracle.project(x, 1.0, b, 1), b, 1)
    np.testing.assert_array_equal(q, expect)


def test_subnormal_quotients():
    """Subnormal inputs and tiny scales stay exact (no flush to zero)."""
    b, ks = 5, 3
    x = np.array([1e-45, 3e-45, 1e-40, 5.9e-39], dtype=np.float32)
    alpha = np.float32(1e-44)
    bf = oracle.project_bruteforce(x, alpha, b, ks)
    np.testing.assert_array_equal(oracle.project(x, alpha, b, ks), bf)
    assert oracle.project_value(x[1], alpha, b, ks) != 0.0
