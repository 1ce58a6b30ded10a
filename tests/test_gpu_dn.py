"""GPU data normalization and analytic aligner vs the oracle (Sec. 3.4, eq. (9)).

esb_dn_stats: the binary32 mean and standard deviation within one ulp of the
oracle's long-double statistics rounded to binary32 (the device sums in fp64 in
another order, so the last rounding may fall on the other side).
esb_project_dn: bit-exact codes against the oracle given the same binary32
statistics.  esb_dda_normal: D within 1e-10 relative of the oracle's fp64
closed form (device erfc/exp differ from the C library's in the last bits; the
cell sums cancel by at most a factor 1e3 for the finest formats), the chosen
scale the grid's argmin, and Table 1 regenerated on the device.
"""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK, read_golden
from gpuutil import assert_rel, dev, host, log, scalar

pytestmark = pytest.mark.gpu

TABLE1 = [(int(b), int(k), float(d), float(a)) for b, k, d, a in read_golden("table1_dda.txt")]
# Table 1 lists the smallest-scale local minimum for these two rows; the global
# minimum on (0, 3] lies at a larger scale (pinned on the oracle alone).
NONCONVEX_ROWS = {(4, 0), (5, 1)}


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def ulps(a, b):
    a = np.array([a], dtype=np.float32).view(np.int32)[0].astype(np.int64)
    b = np.array([b], dtype=np.float32).view(np.int32)[0].astype(np.int64)
    return abs(a - b)


def stats_inputs():
    r = np.random.default_rng(505)
    yield "weights_n64x3x3x64", (r.standard_normal(36864) * 0.05 + 0.001).astype(np.float32)
    yield "offset_mean", (r.standard_normal(300001) + 100.0).astype(np.float32)
    yield "uniform_2^22+7", r.uniform(-3, 5, (1 << 22) + 7).astype(np.float32)
    yield "one", np.array([1.25], dtype=np.float32)
    yield "tiny_ragged", r.standard_normal(1000).astype(np.float32)
    yield "constant", np.full(4099, 0.7, dtype=np.float32)
    yield "heavy_tail", (r.standard_t(3, 1 << 20)).astype(np.float32)


@pytest.mark.parametrize("name", [n for n, _ in stats_inputs()])
def test_dn_stats(esb, name):
    x = dict(stats_inputs())[name]
    log("dn_stats %s len=%d" % (name, x.size))
    got = host(esb.esb_dn_stats(dev(x)))
    m, s = oracle.dn_stats(x)
    assert ulps(got[0], np.float32(m)) <= 1, (got[0], m)
    assert ulps(got[1], np.float32(s)) <= 1, (got[1], s)


def test_dn_stats_empty(esb):
    torch = pytest.importorskip("torch")
    got = host(esb.esb_dn_stats(torch.empty(0, dtype=torch.float32, device="cuda")))
    assert np.isnan(got).all()


def test_dn_stats_workspace_reuse(esb):
    """Two calls on one workspace (stale partials must not leak into the second)."""
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(9)
    a = r.standard_normal(1 << 21).astype(np.float32) * 3 + 1
    b = r.standard_normal(5000).astype(np.float32)
    ws = torch.empty(int(esb.lib().esb_dn_workspace_size(a.size)), dtype=torch.uint8,
                     device="cuda")
    for x in (a, b):
        got = host(esb.esb_dn_stats(dev(x), workspace=ws))
        m, s = oracle.dn_stats(x)
        assert ulps(got[0], np.float32(m)) <= 1 and ulps(got[1], np.float32(s)) <= 1


def mixed(seed):
    r = np.random.default_rng(seed)
    x = (r.standard_normal(50000) * 0.07 + 0.002).astype(np.float32)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, 3.4e38, -3.4e38, 0.002],
                        dtype=np.float32)
    bits = r.integers(0, 2 ** 32, size=20000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    edges = np.array([2.0 ** -100, 2.0 ** 100, 2.0 ** -101, 2.0 ** 101], dtype=np.float32)
    edges = np.concatenate([edges, np.nextafter(edges, np.float32(0)),
                            np.nextafter(edges, np.float32(np.inf))])
    return np.concatenate([x, specials, x[:777] * np.float32(40), bits, edges, -edges,
                           edges + np.float32(0.002)])


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_project_dn_given_stats(esb, b, ks):
    x = mixed(b * 10 + ks)
    xd = dev(x)
    for mean, std, alpha in [(0.002, 0.07, 1.2), (-0.5, 3.0, 0.4871), (0.0, 1e-9, 2.0),
                             (0.0, 0.0, 1.0), (0.0, 2.0 ** 24 - 1, 0.03), (1.0, 2.0 ** 25, 1e-6),
                             (0.0, -1e-7, 1.0), (0.0, -2.0, 0.5), (0.3, np.inf, 1.0)]:
        st = dev(np.array([mean, std], dtype=np.float32))
        log("project_dn b=%d k_sig=%d mean=%g std=%g alpha=%g" % (b, ks, mean, std, alpha))
        got = host(esb.esb_project_dn(xd, st, scalar(alpha), b, ks))
        np.testing.assert_array_equal(got, oracle.project_dn(x, mean, std, alpha, b, ks))


@pytest.mark.parametrize("b,ks", [(3, 1), (4, 2), (5, 3), (6, 4), (8, 5)])
def test_alg1_chain(esb, b, ks):
    """W -> device statistics -> device analytic alpha -> device codes, each step checked."""
    r = np.random.default_rng([77, b, ks])
    w = (r.standard_normal(3 * 3 * 64 * 64 + 17) * 0.03 - 0.004).astype(np.float32)
    wd = dev(w)
    st = esb.esb_dn_stats(wd)
    grid = np.linspace(0.01, 4.0, 2000).astype(np.float32)
    alpha, D = esb.esb_dda_normal(b, ks, dev(grid))
    codes = host(esb.esb_project_dn(wd, st, alpha, b, ks))
    sh = host(st)
    a = float(host(alpha)[0])
    m, s = oracle.dn_stats(w)
    assert ulps(sh[0], np.float32(m)) <= 1 and ulps(sh[1], np.float32(s)) <= 1
    Do = np.array([oracle.dda_normal(g, b, ks) for g in grid])
    assert a == grid[int(np.argmin(Do))] or abs(Do[grid == a][0] - Do.min()) <= 1e-10 * Do.min()
    np.testing.assert_array_equal(codes, oracle.project_dn(w, sh[0], sh[1], a, b, ks))


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_dda_normal_objective(esb, b, ks):
    grid = np.concatenate([np.linspace(0.003, 3.5, 1500), [0.4871, 1e-3, 7.5]]).astype(np.float32)
    log("dda_normal b=%d k_sig=%d G=%d" % (b, ks, grid.size))
    torch = pytest.importorskip("torch")
    dD = torch.empty(grid.size, dtype=torch.float64, device="cuda")
    alpha, D = esb.esb_dda_normal(b, ks, dev(grid), dD_out=dD)
    Dg = host(D)
    Do = np.array([oracle.dda_normal(g, b, ks) for g in grid])
    assert_rel(Dg, Do, 1e-10, "D b=%d k_sig=%d" % (b, ks))
    dDo = np.array([oracle.dda_normal_deriv(g, b, ks) for g in grid])
    # the slope crosses zero: compare against the scale of its terms, not itself
    np.testing.assert_allclose(host(dD), dDo, rtol=1e-10, atol=1e-12)
    j = int(np.argmin(Dg))
    assert host(alpha)[0] == grid[j]
    jo = int(np.argmin(Do))
    assert j == jo or abs(Do[j] - Do[jo]) <= 1e-10 * Do[jo]


@pytest.mark.parametrize("b,k,dda,alpha_star", TABLE1)
def test_table1_on_device(esb, b, k, dda, alpha_star):
    """Table 1 (b, k, DDA, alpha*) from the device objective; paper k = k_sig - 1."""
    ks = k + 1
    torch = pytest.importorskip("torch")
    around = np.array([alpha_star, alpha_star - 2e-4, alpha_star + 2e-4], dtype=np.float32)
    dD = torch.empty(3, dtype=torch.float64, device="cuda")
    _, D1 = esb.esb_dda_normal(b, ks, dev(around), dD_out=dD)
    assert abs(2 * host(D1)[0] - dda) <= 0.5e-4 + 1e-6
    s = host(dD)
    assert s[1] < 0 < s[2]   # alpha* is where the slope changes sign
    grid = np.linspace(0.005, 3.0, 6000).astype(np.float32)
    alpha, _ = esb.esb_dda_normal(b, ks, dev(grid))
    a = float(host(alpha)[0])
    if (b, k) in NONCONVEX_ROWS:
        assert a > alpha_star + 0.01
    else:
        assert abs(a - alpha_star) <= 1e-3, (a, alpha_star)


def test_dda_normal_invalid_candidates(esb):
    grid = np.array([np.nan, -1.0, 0.0, 1.1, np.inf, 0.9, 1.1], dtype=np.float32)
    alpha, D = esb.esb_dda_normal(4, 2, dev(grid))
    Dg = host(D)
    assert np.isnan(Dg[[0, 1, 2, 4]]).all()
    assert np.isfinite(Dg[[3, 5, 6]]).all()
    assert Dg[3] == Dg[6]
    want = grid[3] if Dg[3] <= Dg[5] else grid[5]
    assert host(alpha)[0] == want
    alpha, D = esb.esb_dda_normal(4, 2, dev(np.array([np.nan, -2.0], dtype=np.float32)))
    assert np.isnan(host(D)).all() and np.isnan(host(alpha)[0])


@pytest.mark.parametrize("length", [1, 1000, 300001])
def test_dn_unaligned(esb, length):
    """Statistics and normalized projection on an x that starts 4 bytes past a 16-byte
    boundary (the scalar-load kernels) and codes at an odd address."""
    torch = pytest.importorskip("torch")
    r = np.random.default_rng([31, length])
    x = (r.standard_normal(length) * 0.4 - 0.03).astype(np.float32)
    log("dn unaligned len=%d" % length)
    xd = dev(np.concatenate([[np.float32(7)], x]))[1:]
    assert xd.data_ptr() % 16 != 0
    st = esb.esb_dn_stats(xd)
    got = host(st)
    m, s = oracle.dn_stats(x)
    assert ulps(got[0], np.float32(m)) <= 1 and ulps(got[1], np.float32(s)) <= 1
    codes = torch.empty(length + 1, dtype=torch.uint8, device="cuda")[1:]
    esb.esb_project_dn(xd, st, scalar(0.9), 4, 2, codes=codes)
    np.testing.assert_array_equal(host(codes), oracle.project_dn(x, got[0], got[1], 0.9, 4, 2))
