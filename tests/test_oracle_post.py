"""Pins of the oracle's fused post-processing (Sec. 4.2, eq. (16), then the projection).

* Without affine, residual or ReLU it is the plain projection of y (pinned against brute
  force elsewhere), and z is y.
* The affine step is one rounding of a*y + b: checked in exact rational arithmetic on
  random values and on cancellation cases b = -fl32(a*y), where rounding a*y first would
  give exactly 0.
* The residual is one binary32 addition; ReLU maps negatives and NaN to +0 (whose code is
  the all-ones exponent with a zero fraction).
* Eq. (16): a BN and a DN folded into per-channel (a, b) give, after the projection with
  the next layer's alpha, the codes of the unfused fp64 chain, except where that chain
  lies within rounding distance of a cell midpoint.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def rn32(v):
    f = np.float32(float(v))
    best = None
    for c in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        key = (abs(Fraction(float(c)) - v), int(np.array([c]).view(np.uint32)[0]) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_identity_post_is_the_projection():
    r = np.random.default_rng(1)
    y = (r.standard_normal((37, 53)) * 3).astype(np.float32)
    y[0, :5] = [0.0, -0.0, np.nan, np.inf, -np.inf]
    for (b, ks, alpha) in [(4, 2, 0.7), (5, 3, 0.3), (8, 5, 0.05), (3, 1, 1.0)]:
        z, codes = oracle.post(y, b, ks, alpha)
        np.testing.assert_array_equal(codes, oracle.project(y, alpha, b, ks))
        same = ~np.isnan(y)
        assert np.array_equal(z[same], y[same]) and np.isnan(z[~same]).all()


def test_affine_is_one_rounding():
    r = np.random.default_rng(2)
    rows, cols = 40, 30
    y = (r.standard_normal((rows, cols)) * 2).astype(np.float32)
    a = (r.standard_normal(cols) * 1.5).astype(np.float32)
    bias = (r.standard_normal(cols)).astype(np.float32)
    # cancellation rows: b = -fl32(a*y) makes the result the rounding error of a*y
    bias_c = np.array([-(np.float32(a[j] * y[0, j])) for j in range(cols)], dtype=np.float32)
    for bb in (bias, bias_c):
        z, _ = oracle.post(y, 4, 2, 1.0, a=a, bias=bb)
        for i in range(rows if bb is bias else 1):
            for j in range(cols):
                want = rn32(Fraction(float(a[j])) * Fraction(float(y[i, j])) + Fraction(float(bb[j])))
                assert z[i, j] == want, (i, j, z[i, j], want)
    z, _ = oracle.post(y[:1], 4, 2, 1.0, a=a, bias=bias_c)
    assert np.count_nonzero(z) > cols // 2   # two roundings would give zeros here


def test_residual_and_relu():
    r = np.random.default_rng(3)
    y = r.standard_normal((20, 64)).astype(np.float32)
    res = r.standard_normal((20, 64)).astype(np.float32)
    y[0, 0] = np.nan
    z, codes = oracle.post(y, 5, 3, 0.25, res=res)
    ok = ~np.isnan(y)
    np.testing.assert_array_equal(z[ok], (y + res)[ok])
    z, codes = oracle.post(y, 5, 3, 0.25, res=res, relu=True)
    assert np.isnan(z).sum() == 0 and (z >= 0).all()
    pos = (y + res) > 0
    np.testing.assert_array_equal(z[pos], (y + res)[pos])
    assert (z[~pos] == 0).all()
    assert (codes[~pos] == oracle.encode(0.0, 5, 3)).all()   # the code of +0
    np.testing.assert_array_equal(codes, oracle.project(z, 0.25, 5, 3))


@pytest.mark.parametrize("b,ks", [(4, 2), (5, 3), (6, 3)])
def test_eq16_folding_of_bn_and_dn(b, ks):
    r = np.random.default_rng([4, b, ks])
    rows, cols = 64, 48
    y = (r.standard_normal((rows, cols)) * 0.8 + 0.1).astype(np.float32)
    gamma = r.uniform(0.5, 1.5, cols)
    beta = r.standard_normal(cols) * 0.1
    mu_b = r.standard_normal(cols) * 0.2
    sd_b = r.uniform(0.5, 2.0, cols)
    mu_d, sd_d, eps = 0.05, 1.3, 1e-7
    alpha_next = np.float32(0.6)
    # unfused chain in fp64: BN, then DN
    t = gamma * (y.astype(np.float64) - mu_b) / sd_b + beta
    t = (t - mu_d) / (sd_d + eps)
    # folded constants (a, b) of eq. (16), rounded to binary32
    a = (gamma / sd_b / (sd_d + eps)).astype(np.float32)
    bb = ((beta - gamma * mu_b / sd_b - mu_d) / (sd_d + eps)).astype(np.float32)
    z, codes = oracle.post(y, b, ks, alpha_next, a=a, bias=bb)
    # a, b rounded to binary32 (half an ulp each) and the fma's one rounding
    scale = np.abs(a.astype(np.float64) * y) + np.abs(bb.astype(np.float64))
    assert (np.abs(z - t) <= 2.0 ** -22 * scale).all()
    # codes of the exact chain: nearest set value to t/alpha (ties up), clipped
    q = np.asarray(oracle.valueset(b, ks), dtype=np.float64)
    v = np.abs(t) / np.float64(alpha_next)
    mids = (q[1:] + q[:-1]) / 2
    cell = np.searchsorted(mids, v, side="right")
    near = np.min(np.abs(v[..., None] - mids), axis=-1) <= 1e-5 * np.maximum(v, 1.0)
    qz = oracle.dequantize(codes, 1.0, b, ks)
    same = np.abs(qz.astype(np.float64)) == q[cell]
    assert (same | near).all()
    assert same.mean() > 0.99
