"""CPU model of the projection kernel's fast path (reciprocal multiply, rounding
on the bit pattern, exact fallback within 4 ulps of a cell midpoint), checked
against the oracle: whenever the model does not ask for the fallback, its code
must equal the oracle's.  This tests the error argument of the fast path on
many more inputs than the GPU tests take."""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK


def fast_model(x, alpha, b, ks):
    with np.errstate(over="ignore", invalid="ignore"):
        return _fast_model(x, alpha, b, ks)


def _fast_model(x, alpha, b, ks):
    k = ks - 1
    N = 2 ** (b - k - 1) - 1
    zero = N << k
    sign_bit = 1 << (b - 1)
    C = np.float32(oracle.C(b, ks))
    c_code = ((N - 1) << k) | ((1 << k) - 1)
    r = np.float32(1.0) / np.float32(alpha)
    q0 = (x.astype(np.float32) * r).astype(np.float32)
    qb = q0.view(np.uint32)
    ab = qb & np.uint32(0x7FFFFFFF)
    small = ab < np.uint32(0x3F800000)
    w = np.where(small, ab.view(np.float32) + np.float32(1.0), ab.view(np.float32)).astype(np.float32)
    wb = w.view(np.uint32).astype(np.int64)
    shA = 23 - k
    half = 1 << (shA - 1)
    c = ((wb + half) >> shA) - (127 << k)
    d = wb & ((half << 1) - 1)
    risky = np.abs(d - half) <= 4
    code = np.where(small, (zero + c) & (sign_bit - 1), c)
    code = np.where(ab.astype(np.int64) >= int(C.view(np.uint32)), c_code, code)
    code = np.where(ab > np.uint32(0x7F800000), zero, code)
    code = np.where((code != zero) & (qb >> np.uint32(31) == 1), code | sign_bit, code)
    return code.astype(np.uint8), risky


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_fast_model_agrees_when_not_risky(b, ks):
    r = np.random.default_rng([51, b, ks])
    v = oracle.valueset(b, ks)
    mids = (v[1:] + v[:-1]) / 2
    total_risky = 0
    for alpha in np.concatenate([r.uniform(1e-3, 3.0, 6), [0.37, 1.0 / 3]]).astype(np.float32):
        base = (mids * np.float64(alpha)).astype(np.float32).view(np.uint32).astype(np.int64)
        near = (base[:, None] + np.arange(-64, 65)[None, :]).ravel().astype(np.uint32).view(np.float32)
        x = np.concatenate([near, -near, (r.standard_normal(200000) * 2 * alpha).astype(np.float32),
                            r.integers(0, 2 ** 32, 100000, dtype=np.uint64).astype(np.uint32).view(np.float32)])
        code, risky = fast_model(x, alpha, b, ks)
        ref = oracle.project(x, alpha, b, ks)
        ok = ~risky
        np.testing.assert_array_equal(code[ok], ref[ok])
        total_risky += int(risky.sum())
    assert total_risky > 0      # the near-midpoint inputs do exercise the fallback
