"""Pins of the oracle's ESB float format (eq. (14)) and its multiplication rule (eq. (15))."""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK, TABLE1_BK


def fields(code, b, k_sig):
    k = k_sig - 1
    ebits = b - k - 1
    return (code >> (b - 1)) & 1, (code >> k) & ((1 << ebits) - 1), code & ((1 << k) - 1)


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_decode_all_codes_is_signed_set(b, ks):
    vals = np.array([oracle.decode(c, b, ks) for c in range(2 ** b)])
    full = oracle.full_valueset(b, ks)
    np.testing.assert_array_equal(np.unique(vals), full)
    # every nonzero member has exactly one code; zero has two (sign 0 and sign 1)
    u, cnt = np.unique(vals, return_counts=True)
    assert cnt[u == 0.0][0] == 2 and np.all(cnt[u != 0.0] == 1)


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_encode_roundtrip_and_canonical_zero(b, ks):
    N = oracle.N(b, ks)
    k = ks - 1
    zero = N << k
    for c in range(2 ** b):
        q = oracle.decode(c, b, ks)
        e = oracle.encode(q, b, ks)
        if q == 0.0:
            assert e == zero                      # +0, sign bit 0
        else:
            assert e == c
    assert oracle.encode(0.3, 4, 2) == -1          # not a member


def test_code_layout_examples():
    """Layout sign | exponent | fraction with the all-ones exponent subnormal (eq. (14))."""
    assert oracle.encode(0.0, 4, 2) == 0b0110
    assert oracle.encode(0.5, 4, 2) == 0b0111
    assert oracle.encode(1.0, 4, 2) == 0b0000
    assert oracle.encode(6.0, 4, 2) == 0b0101
    assert oracle.encode(-6.0, 4, 2) == 0b1101
    assert oracle.encode(5.0, 5, 3) == 0b01001


@pytest.mark.parametrize("b,ks", TABLE1_BK)
def test_multiplication_rule_eq15(b, ks):
    """q_i q_j = (-1)^(sb_i xor sb_j) * (zeta_i + 0.f_i)(zeta_j + 0.f_j) * 2^(e_i zeta_i + e_j zeta_j)."""
    k = ks - 1
    emax = 2 ** (b - k - 1) - 1
    codes = np.arange(2 ** b)
    sb, e, f = fields(codes, b, ks)
    zeta = (e != emax).astype(np.int64)
    frac = zeta + f / 2.0 ** k
    dec = np.array([oracle.decode(int(c), b, ks) for c in codes])
    prod_rule = ((-1.0) ** (sb[:, None] ^ sb[None, :]) * (frac[:, None] * frac[None, :])
                 * 2.0 ** (e[:, None] * zeta[:, None] + e[None, :] * zeta[None, :]))
    np.testing.assert_array_equal(prod_rule, dec[:, None] * dec[None, :])
    # the fraction product needs at most (k+1) x (k+1) significant bits
    fi = (frac * 2 ** k).astype(np.int64)
    assert fi.max() < 2 ** (k + 1)
