"""GPU projection (esb_project) vs the oracle: bit-exact codes."""
import numpy as np
import pytest

import oracle
from conftest import ALL_BK
from gpuutil import dev, host, log, scalar
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def mixed_inputs(b, ks, seed):
    r = np.random.default_rng([21, b, ks, seed])
    bits = r.integers(0, 2 ** 32, size=30000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    v = oracle.valueset(b, ks)
    mids = ((v[1:] + v[:-1]) / 2).astype(np.float32)
    around = np.concatenate([mids, np.nextafter(mids, np.float32(np.inf)),
                             np.nextafter(mids, np.float32(-np.inf)), v.astype(np.float32)])
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45, 1.17e-38, 3.4e38,
                         -3.4e38], dtype=np.float32)
    normal = (r.standard_normal(30000) * 2).astype(np.float32)
    return np.concatenate([bits, specials, around, -around, around * np.float32(0.125), normal])


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_project_all_formats(esb, b, ks):
    x = mixed_inputs(b, ks, 0)
    xd = dev(x)
    for alpha in [1.0, 0.125, 0.37, 2.0 ** -5, 1.7e-3, 3.1, 1e-40]:
        log("project b=%d k_sig=%d alpha=%g len=%d" % (b, ks, alpha, x.size))
        got = host(esb.esb_project(xd, scalar(alpha), b, ks))
        np.testing.assert_array_equal(got, oracle.project(x, alpha, b, ks))


@pytest.mark.parametrize("length", [0, 1, 2, 3, 4, 5, 7, 63, 64, 65, 1000, 4097, 1 << 20])
@pytest.mark.parametrize("offset", [0, 1, 3])
def test_project_ragged_and_unaligned(esb, length, offset):
    torch = pytest.importorskip("torch")
    x = (np.random.default_rng(length + offset).standard_normal(length + 8) * 3).astype(np.float32)
    xd = dev(x)[offset:offset + length]
    codes = torch.full((length + 8,), 0xAB, dtype=torch.uint8, device="cuda")
    log("project ragged len=%d offset=%d" % (length, offset))
    esb.esb_project(xd, scalar(0.7), 4, 2, codes=codes[offset:offset + length])
    got = host(codes)
    np.testing.assert_array_equal(got[offset:offset + length],
                                  oracle.project(x[offset:offset + length], 0.7, 4, 2))
    assert (got[:offset] == 0xAB).all() and (got[offset + length:] == 0xAB).all()   # no overrun


@pytest.mark.parametrize("alpha", [0.0, -1.0, float("inf"), float("nan")])
def test_project_invalid_alpha_gives_zero_codes(esb, alpha):
    x = np.linspace(-5, 5, 999).astype(np.float32)
    log("project invalid alpha %r" % alpha)
    got = host(esb.esb_project(dev(x), scalar(alpha), 5, 3))
    np.testing.assert_array_equal(got, oracle.project(x, alpha, 5, 3))
    assert (got == oracle.encode(0.0, 5, 3)).all()


def test_project_subnormal_quotients(esb):
    x = np.array([1e-45, 3e-45, 1e-40, 5.9e-39, -2e-44, 1e-38, 2.5e-44], dtype=np.float32)
    for alpha in [1e-44, 3e-45, 1e-38]:
        for b, ks in [(5, 3), (8, 7), (4, 1)]:
            got = host(esb.esb_project(dev(x), scalar(alpha), b, ks))
            np.testing.assert_array_equal(got, oracle.project(x, alpha, b, ks))


def test_dequantize(esb):
    for b, ks in [(4, 2), (5, 3), (8, 5), (3, 1)]:
        codes = np.arange(256, dtype=np.uint8)
        got = host(esb.esb_dequantize(dev(codes), scalar(0.37), b, ks))
        np.testing.assert_array_equal(got, oracle.dequantize(codes, 0.37, b, ks))


def test_project_full_size_workloads(esb):
    """Every projected tensor of the AlexNet FC and MobileNetV2 block workloads, full size."""
    c = wl.alexnet_fc(0)
    for name, x, b, ks, alpha in [("alexnet W", c["W"], c["nW"], c["ksW"], c["gridW"][9]),
                                  ("alexnet X", c["X"], c["nX"], c["ksX"], c["gridX"][20])]:
        log("project full %s %s" % (name, x.shape))
        got = host(esb.esb_project(dev(x), scalar(alpha), b, ks))
        np.testing.assert_array_equal(got, oracle.project(x, alpha, b, ks))
    m = wl.mobilenetv2_block(0)
    for L in m["layers"]:
        log("project full mobilenet %s %s" % (L["name"], L["x"].shape))
        got = host(esb.esb_project(dev(L["x"]), scalar(m["gridX"][10]), m["n"], m["ks"]))
        np.testing.assert_array_equal(got, oracle.project(L["x"], m["gridX"][10], m["n"], m["ks"]))


@pytest.mark.parametrize("b,ks", [(4, 2), (3, 1), (3, 2), (5, 3), (8, 6), (8, 1), (2, 1)])
def test_project_near_scaled_midpoints(esb, b, ks):
    """x within +-8 ulps of alpha * mu for many non-power-of-two alpha: the region where
    x * fl32(1/alpha) and fl32(x/alpha) can round to different set values."""
    r = np.random.default_rng([41, b, ks])
    v = oracle.valueset(b, ks)
    mids = ((v[1:] + v[:-1]) / 2)
    alphas = np.concatenate([r.uniform(1e-3, 3.0, 24), [1.0 / 3, 0.1, 0.7, 1.1, 2.9]]).astype(np.float32)
    for alpha in alphas:
        base = (mids * np.float64(alpha)).astype(np.float32)
        steps = np.arange(-8, 9, dtype=np.int64)
        bits = (base.view(np.uint32).astype(np.int64)[:, None] + steps[None, :]).ravel()
        x = bits.astype(np.uint32).view(np.float32)
        x = np.concatenate([x, -x])
        got = host(esb.esb_project(dev(x), scalar(float(alpha)), b, ks))
        np.testing.assert_array_equal(got, oracle.project(x, alpha, b, ks))


def test_project_extreme_scales(esb):
    """Scales outside [2^-125, 2^125] use the exact division for every element."""
    z = np.random.default_rng(9).standard_normal(4096)
    for alpha in [1e-39, 2.0 ** -126, 2.0 ** -125, 2.0 ** 125, 3e38]:
        for b, ks in [(4, 2), (8, 7)]:
            with np.errstate(over="ignore"):
                xs = (z * np.float64(alpha)).astype(np.float32)
            got = host(esb.esb_project(dev(xs), scalar(alpha), b, ks))
            np.testing.assert_array_equal(got, oracle.project(xs, alpha, b, ks))
