"""Oracle pins for data normalization (Sec. 3.4, the DN equation) and the projection of
normalized data (Alg. 1: ESB(DN(W))).

* The statistics equal numpy's float64 mean and population standard deviation (a library
  routine) on data with a large offset, and reduce to the obvious values on constant data
  and a single element.
* With mean 0 and a standard deviation whose fl32(std + 1e-7) is exactly 1, the projection
  of normalized data is the plain projection (already pinned against brute force).
* Otherwise it is the plain projection of x-hat, with x-hat formed by binary32 IEEE
  arithmetic (numpy float32), and x-hat has mean ~0 and standard deviation ~1."""
import numpy as np

import oracle


def test_dn_stats_match_numpy():
    r = np.random.default_rng(3)
    for (loc, scale, n) in [(0.0, 1.0, 10007), (1000.0, 0.01, 5000), (-3.5, 250.0, 777)]:
        x = (loc + scale * r.standard_normal(n)).astype(np.float32)
        m, s = oracle.dn_stats(x)
        xd = x.astype(np.float64)
        assert abs(m - xd.mean()) <= 1e-12 * max(abs(xd.mean()), scale)
        assert abs(s - xd.std()) <= 1e-10 * xd.std()


def test_dn_stats_special_cases():
    m, s = oracle.dn_stats(np.full(100, 2.5, np.float32))
    assert m == 2.5 and s == 0.0
    m, s = oracle.dn_stats(np.array([-7.25], np.float32))
    assert m == -7.25 and s == 0.0
    m, s = oracle.dn_stats(np.array([1.0, 3.0], np.float32))
    assert m == 2.0 and s == 1.0


def test_project_dn_identity_case_is_plain_projection():
    x = np.random.default_rng(4).standard_normal(20000).astype(np.float32)
    std = np.float32(1.0) - np.float32(2.0 ** -23)
    assert np.float32(std + np.float32(1e-7)) == np.float32(1.0)
    for (b, ks, alpha) in [(4, 2, 0.4871), (5, 3, 0.3), (3, 1, 1.1)]:
        np.testing.assert_array_equal(oracle.project_dn(x, 0.0, std, alpha, b, ks),
                                      oracle.project(x, alpha, b, ks))


def test_project_dn_is_projection_of_normalized_data():
    r = np.random.default_rng(5)
    x = (12.0 + 0.7 * r.standard_normal(30000)).astype(np.float32)
    m, s = oracle.dn_stats(x)
    m32, s32 = np.float32(m), np.float32(s)
    xh = (x - m32) / np.float32(s32 + np.float32(1e-7))
    assert xh.dtype == np.float32
    assert abs(float(xh.astype(np.float64).mean())) < 1e-3
    assert abs(float(xh.astype(np.float64).std()) - 1.0) < 1e-3
    for (b, ks, alpha) in [(4, 2, 0.4871), (5, 3, 0.3)]:
        np.testing.assert_array_equal(oracle.project_dn(x, m32, s32, alpha, b, ks),
                                      oracle.project(xh, alpha, b, ks))
