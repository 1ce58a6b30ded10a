"""Glue kernels between quantized layers (esb_maxpool2d, esb_avgpool_global,
esb_absmax) against plain NumPy definitions: bit-exact (max, the absolute
maximum and a float64 sum in position order divided once are all exactly
defined)."""
import numpy as np
import pytest

from gpuutil import dev, host, log, scalar, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def maxpool_ref(a, R, stride, pad):
    B, H, W, C = a.shape
    P = (H + 2 * pad - R) // stride + 1
    Q = (W + 2 * pad - R) // stride + 1
    out = np.full((B, P, Q, C), -np.inf, dtype=np.float32)
    nan = np.zeros((B, P, Q, C), dtype=bool)
    for p in range(P):
        for q in range(Q):
            h0, w0 = p * stride - pad, q * stride - pad
            win = a[:, max(h0, 0):min(h0 + R, H), max(w0, 0):min(w0 + R, W), :]
            out[:, p, q, :] = np.nanmax(np.where(np.isnan(win), -np.inf, win), axis=(1, 2))
            nan[:, p, q, :] = np.isnan(win).any(axis=(1, 2))
    out[nan] = np.nan
    return out


@pytest.mark.parametrize("shape,R,stride,pad", [
    ((2, 112, 112, 64), 3, 2, 1),      # ResNet18 stem pool
    ((3, 15, 17, 6), 3, 2, 1),         # C % 4 != 0: one channel per thread
    ((2, 9, 8, 8), 2, 2, 0),
    ((1, 7, 7, 12), 3, 1, 1),
    ((2, 5, 6, 4), 5, 3, 2),
])
def test_maxpool(esb, shape, R, stride, pad):
    a = np.random.default_rng(1).standard_normal(shape).astype(np.float32)
    a[0, 1, 2, 1] = np.nan
    log("maxpool %s R=%d stride=%d pad=%d" % (shape, R, stride, pad))
    got = host(esb.esb_maxpool2d(dev(a), R, stride, pad))
    want = maxpool_ref(a, R, stride, pad)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(want))
    np.testing.assert_array_equal(got[~np.isnan(got)], want[~np.isnan(want)])


def test_maxpool_resnet_batch64(esb):
    """The stem pool at batch 64 (64 x 112 x 112 x 64 -> 56 x 56): first and last image."""
    torch = torch_cuda()
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    a = torch.relu(torch.randn((64, 112, 112, 64), generator=g, device="cuda"))
    got = esb.esb_maxpool2d(a, 3, 2, 1)
    for i in (0, 63):
        np.testing.assert_array_equal(host(got[i:i + 1]), maxpool_ref(host(a[i:i + 1]), 3, 2, 1))


@pytest.mark.parametrize("shape", [(64, 7, 7, 512), (3, 5, 5, 7), (1, 1, 1, 1), (2, 49, 1, 3)])
def test_avgpool_global(esb, shape):
    torch = torch_cuda()
    a = np.abs(np.random.default_rng(2).standard_normal(shape)).astype(np.float32)
    a.reshape(-1)[::7] *= 1e-6       # values many binades apart
    B, C = shape[0], shape[-1]
    flat = a.reshape(B, -1, C).astype(np.float64)
    acc = np.zeros((B, C))
    for i in range(flat.shape[1]):
        acc += flat[:, i, :]
    want = (acc / flat.shape[1]).astype(np.float32)
    amax = scalar(0.0)
    got = esb.esb_avgpool_global(dev(a), absmax=amax)
    np.testing.assert_array_equal(host(got).view(np.uint32), want.view(np.uint32))
    assert host(amax)[0] == np.max(np.abs(want))
    del torch


@pytest.mark.parametrize("n,offset", [(0, 0), (1, 0), (7, 1), (1000, 0), (4097, 3),
                                      (12_845_056, 0)])
def test_absmax(esb, n, offset):
    torch = torch_cuda()
    x = np.random.default_rng(n).standard_normal(n + offset).astype(np.float32)
    if n > 10:
        x[offset + n // 2] = -50.0      # the maximum is negative
    xd = dev(x)[offset:]
    m = scalar(0.0)
    esb.esb_absmax(xd, m)
    want = np.max(np.abs(x[offset:])) if n else np.float32(0)
    assert host(m)[0] == want
    big = scalar(1e30)                  # a larger start value stays
    esb.esb_absmax(xd, big)
    assert host(big)[0] == np.float32(1e30)
    del torch


def test_absmax_nan_and_inf(esb):
    x = np.ones(1000, dtype=np.float32)
    x[10] = -np.inf
    m = scalar(0.0)
    esb.esb_absmax(dev(x), m)
    assert host(m)[0] == np.inf
    x[500] = np.nan
    m = scalar(0.0)
    esb.esb_absmax(dev(x), m)
    assert np.isnan(host(m)[0])
