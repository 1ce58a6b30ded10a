"""The aligner with a plan (esb_dda_plan, esb_dda_align_planned): candidates
2^E factors[j] with E the binary exponent of a device scale (2^(E-1) <= |scale|
< 2^E), the plan's tables shifted in the exponent instead of rebuilt.  Checked
against the oracle's DDA over grid[j] = ldexp(factors[j], E) computed in NumPy
(alpha exact, D within 1e-9 relative), and against esb_dda_align over that same
grid (alpha and every D_j bit-identical), including scales whose shifted tables
would leave the normal range (the call then rebuilds them) and scales that are
not finite."""
import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
REL = 1e-9
NEAR = 1e-10


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def scaled_grid(factors, scale):
    e = int(np.frexp(np.float32(abs(scale)))[1]) if scale != 0 else 0
    return np.ldexp(factors.astype(np.float32), e).astype(np.float32)


def check_alpha(a, grid, j, Do, what):
    best = Do[j]
    if np.isfinite(best) and best > 0:
        near = np.flatnonzero(~np.isnan(Do) & (Do <= best * (1.0 + NEAR)))
    else:
        near = np.flatnonzero((Do == best) | (np.isnan(Do) & np.isnan(best)))
    if np.all((Do[near] == best) | (np.isnan(Do[near]) & np.isnan(best))):
        assert a == grid[j], (what, a, grid[j])
    else:
        assert a in grid[near], (what, a, grid[near])


def run_both(esb, x, n, ks, factors, plan, scale, what):
    """Planned call, the plain call on the host-computed grid, and the oracle."""
    xd = dev(x)
    G = factors.size
    ap, Dp = esb.esb_dda_align_planned(xd, n, ks, plan, G, scalar(scale))
    grid = scaled_grid(factors, scale)
    aw, Dw = esb.esb_dda_align(xd, n, ks, dev(grid))
    ap, Dp, aw, Dw = host(ap)[0], host(Dp), host(aw)[0], host(Dw)
    assert ap == aw or (np.isnan(ap) and np.isnan(aw)), (what, ap, aw)
    np.testing.assert_array_equal(Dp.view(np.uint64), Dw.view(np.uint64))
    j, Do = oracle.dda(x, n, ks, grid)
    assert_rel(Dp, Do, REL, what)
    check_alpha(ap, grid, j, Do, what)
    return ap, Dp


FORMATS = [(5, 3), (4, 2), (3, 1), (3, 2), (8, 6), (2, 1), (6, 4)]


@pytest.mark.parametrize("n,ks", FORMATS)
def test_planned_matches_oracle(esb, n, ks):
    cmax = oracle.C(n, ks)
    factors = wl.maxabs_grid_factors(cmax, 64)
    plan = esb.esb_dda_plan(n, ks, dev(factors))
    r = np.random.default_rng([51, n, ks])
    for length, spread, relu in [(200_704, 1.0, True), (37_000, 0.02, False), (5, 3.0, False),
                                 (3_211_264, 40.0, True), (0, 1.0, False)]:
        x = (r.standard_normal(length) * spread).astype(np.float32)
        if relu:
            x = np.maximum(x, 0).astype(np.float32)
        scale = float(np.max(np.abs(x))) if length else 0.0
        log("dda planned n=%d k_sig=%d len=%d scale=%g" % (n, ks, length, scale))
        run_both(esb, x, n, ks, factors, plan, scale, "n%d k%d len%d" % (n, ks, length))


def test_one_plan_many_scales(esb):
    """One plan reused across scales 2^-40 .. 2^40 (and one that is not a power of two)."""
    factors = wl.scale_grid(1.0, 64) / np.float32(8.0)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    base = np.random.default_rng(7).standard_normal(60_000).astype(np.float32)
    for e in list(range(-40, 41, 8)) + [3]:
        x = (base * np.float32(2.0 ** e)).astype(np.float32)
        scale = float(np.max(np.abs(x))) * (1.37 if e == 3 else 1.0)
        run_both(esb, x, 5, 3, factors, plan, scale, "e%d" % e)


@pytest.mark.parametrize("scale", [1e-37, 3e-39, 1e36, 3.0e38])
def test_scales_outside_the_plan_range(esb, scale):
    """Scales whose shifted thresholds or candidates would leave the normal fp32 range: the
    call rebuilds the tables and still equals the plain call and the oracle."""
    factors = wl.maxabs_grid_factors(oracle.C(5, 3), 64)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    x = (np.random.default_rng(3).standard_normal(20_000) * scale).astype(np.float32)
    x = np.where(np.isfinite(x), x, 0).astype(np.float32)
    run_both(esb, x, 5, 3, factors, plan, scale, "scale %g" % scale)


@pytest.mark.parametrize("scale", [np.inf, np.nan])
def test_scale_not_finite(esb, scale):
    factors = wl.maxabs_grid_factors(oracle.C(4, 2), 64)
    plan = esb.esb_dda_plan(4, 2, dev(factors))
    x = np.ones(1000, dtype=np.float32)
    a, D = esb.esb_dda_align_planned(dev(x), 4, 2, plan, 64, scalar(scale))
    assert np.isnan(host(a)[0])
    assert np.all(np.isnan(host(D)))


def test_plan_for_other_arguments_is_not_used(esb):
    """A plan built for another format is ignored: the call rebuilds the tables from the
    factors it holds (same results as the plain call on those candidates)."""
    factors = wl.maxabs_grid_factors(oracle.C(4, 2), 64)
    plan = esb.esb_dda_plan(4, 2, dev(factors))
    x = np.abs(np.random.default_rng(9).standard_normal(30_000)).astype(np.float32)
    run_both(esb, x, 5, 3, factors, plan, float(np.max(x)), "foreign plan")


def test_plan_in_a_batch_free_stack_shape(esb):
    """The ResNet18 factors over a layer-sized input at the shapes of the stack (56x56x64 at
    batch 4), with the running maximum as the scale."""
    torch = torch_cuda()
    factors = wl.maxabs_grid_factors(oracle.C(5, 3), 64)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    xd = torch.relu(torch.randn((4, 56, 56, 64), generator=g, device="cuda"))
    x = host(xd)
    m = scalar(0.0)
    esb.esb_absmax(xd, m)
    assert host(m)[0] == np.max(x)
    run_both(esb, x.reshape(-1), 5, 3, factors, plan, float(np.max(x)), "stack shape")
