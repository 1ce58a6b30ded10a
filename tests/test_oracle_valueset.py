"""Pins of the oracle's value set (eq. (4)-(5)) against things the paper and
standard formats fix independently of the oracle's enumeration."""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK, read_golden


def minifloat_values(b, k_sig):
    """Independent construction: an IEEE-like minifloat with b-k-1 exponent bits,
    k mantissa bits, exponent bias 1, subnormals, every exponent finite."""
    k = k_sig - 1
    ebits = b - k - 1
    vals = set()
    for e in range(0, 1 << ebits):
        for f in range(0, 1 << k):
            if e == 0:
                vals.add(f / 2.0 ** k)                       # 0.f * 2^(1 - bias)
            else:
                vals.add((1 + f / 2.0 ** k) * 2.0 ** (e - 1))  # 1.f * 2^(e - bias)
    return np.array(sorted(vals))


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_cardinality_and_minifloat(b, ks):
    v = oracle.valueset(b, ks)
    assert v.size == 2 ** (b - 1)                 # 2^b - 1 values with the negatives
    assert oracle.full_valueset(b, ks).size == 2 ** b - 1
    assert np.all(np.diff(v) > 0) and v[0] == 0.0
    np.testing.assert_array_equal(v, minifloat_values(b, ks))


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_closed_forms(b, ks):
    k = ks - 1
    N = 2 ** (b - k - 1) - 1
    v = oracle.valueset(b, ks)
    assert oracle.N(b, ks) == N
    assert v[-1] == 2.0 ** N - 2.0 ** (N - k - 1)   # C = max(xi_N * Omega_N)
    assert oracle.C(b, ks) == v[-1]
    # the smallest positive step is xi_0 = 2^-k (eq. (5)); for k = 0 the first value is 1
    assert v[1] == 2.0 ** -k


@pytest.mark.parametrize("b", range(2, 9))
def test_linear_special_case(b):
    """k = b-2: the set is Q_l(alpha, b) of eq. (2) up to the scale 2^-k (Sec. 3.2)."""
    k = b - 2
    v = oracle.valueset(b, k + 1)
    np.testing.assert_array_equal(v * 2.0 ** k, np.arange(0, 2 ** (b - 1)))


@pytest.mark.parametrize("b", range(2, 9))
def test_pot_special_case(b):
    """k = 0: powers of two {0, 2^0, ..., 2^(2^(b-1)-2)} (Sec. 3.2; eq. (3) with the
    top exponent read as 2^(b-1)-2 so that the set has 2^b - 1 members)."""
    v = oracle.valueset(b, 1)
    expect = [0.0] + [2.0 ** e for e in range(0, 2 ** (b - 1) - 1)]
    np.testing.assert_array_equal(v, np.array(expect))


def test_ternary_special_case():
    np.testing.assert_array_equal(oracle.full_valueset(2, 1), [-1.0, 0.0, 1.0])


def test_intro_two_significant_bits_example():
    g = {row[0]: [float(t) for t in row[1:]] for row in read_golden("intro_two_sb_set.txt")}
    s = set(g["base"])
    for sh in g["shifts"]:
        s |= {v * 2 ** sh for v in g["shifted"]}
    pos = np.array(sorted(s))
    full = np.concatenate([-pos[:0:-1], pos])
    assert full.size == int(g["count"][0])
    np.testing.assert_array_equal(pos[-6:], g["listed_tail"])
    # two significant bits in five bits is ESB(5, k=1) scaled by 2
    np.testing.assert_array_equal(2.0 * oracle.valueset(5, 2), pos)


def test_esb41_is_ocp_fp4_e2m1():
    e2m1 = np.array([float(t) for t in read_golden("ocp_fp4_e2m1.txt")[0]])
    np.testing.assert_array_equal(oracle.valueset(4, 2), e2m1)


def test_invalid_parameters():
    for b, ks in [(1, 1), (9, 2), (4, 0), (4, 4), (3, 3)]:
        with pytest.raises(ValueError):
            oracle.valueset(b, ks)
