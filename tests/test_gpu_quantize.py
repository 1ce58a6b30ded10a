"""Quantization of one tensor with a plan in one call (esb_quantize_planned): the
planned aligner's alpha and D_j, then the codes of x under that alpha.  Checked bit for
bit against esb_dda_align_planned followed by esb_project (alpha, every D_j, every code)
on the path where each projection block derives alpha itself (up to 2 tiles of 4096
elements per CU: lengths without and with group sums, a tail of len % 4 elements, an
empty tensor) and on the other paths (more tiles, x not 16-byte aligned, 512
candidates); non-finite and zero scales; and the codes of a small case against the
oracle's projection under the chosen alpha."""
import numpy as np
import pytest

import oracle
from gpuutil import dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def activations(seed, n):
    r = np.random.default_rng(seed)
    return np.maximum(r.standard_normal(n), 0.0).astype(np.float32)


def compare(esb, xd, n, ks, plan, G, scale, what):
    a1, D1, c1 = esb.esb_quantize_planned(xd, n, ks, plan, G, scale)
    a0, D0 = esb.esb_dda_align_planned(xd, n, ks, plan, G, scale)
    c0 = esb.esb_project(xd, a0, n, ks)
    a1, a0 = host(a1), host(a0)
    assert a1.view(np.uint32)[0] == a0.view(np.uint32)[0], (what, a1, a0)
    np.testing.assert_array_equal(host(D1).view(np.uint64), host(D0).view(np.uint64))
    np.testing.assert_array_equal(host(c1), host(c0))
    return a1[0], host(c1)


@pytest.mark.parametrize("length", [0, 3, 32771, 200704, 1605632, 12845056])
@pytest.mark.parametrize("fmt", [(5, 3), (4, 2)])
def test_quantize_equals_align_then_project(esb, length, fmt):
    n, ks = fmt
    factors = wl.scale_grid(1.0).astype(np.float32)
    plan = esb.esb_dda_plan(n, ks, dev(factors))
    x = activations(length + n, length)
    log("quantize len=%d fmt=%s" % (length, fmt))
    xd = dev(x) if length else torch_cuda().empty(0, dtype=torch_cuda().float32, device="cuda")
    scale = float(np.abs(x).max()) if length else 1.0
    compare(esb, xd, n, ks, plan, factors.size, scalar(scale), "len %d" % length)


def test_quantize_fallbacks(esb):
    """x one float past a 16-byte boundary, and 512 candidates (the finishing step does
    not fit one block of 256 threads): the finalize kernel, then the projection."""
    factors = wl.scale_grid(1.0).astype(np.float32)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    x = activations(7, 1605633)
    buf = dev(x)
    xu = buf[1:]                               # data_ptr % 16 == 4
    assert xu.data_ptr() % 16 == 4
    log("quantize unaligned")
    compare(esb, xu, 5, 3, plan, 64, scalar(float(np.abs(x[1:]).max())), "unaligned")
    f512 = np.linspace(1.0 / 512, 1.0, 512).astype(np.float32) / 3.0
    plan512 = esb.esb_dda_plan(4, 2, dev(f512))
    log("quantize G=512")
    compare(esb, buf, 4, 2, plan512, 512, scalar(float(np.abs(x).max())), "G 512")


@pytest.mark.parametrize("scale", [float("nan"), float("inf"), 0.0])
def test_quantize_special_scales(esb, scale):
    factors = wl.scale_grid(1.0).astype(np.float32)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    x = activations(11, 40000)
    log("quantize scale=%r" % scale)
    compare(esb, dev(x), 5, 3, plan, factors.size, scalar(scale), "scale %r" % scale)


def test_quantize_codes_match_oracle(esb):
    """The codes are the oracle's projection of x under the alpha the call chose."""
    factors = wl.scale_grid(1.0).astype(np.float32)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    x = np.random.default_rng(3).standard_normal(5003).astype(np.float32)
    a, codes = compare(esb, dev(x), 5, 3, plan, factors.size,
                       scalar(float(np.abs(x).max())), "oracle")
    np.testing.assert_array_equal(codes, oracle.project(x, np.float32(a), 5, 3))


def boundary_lengths():
    """Lengths at the edges of the call's paths: the last block count without group sums
    (32 blocks of 2 rows of 4096 elements), the last projection size that takes the
    finishing step in every block (two tiles of 4096 elements per CU on a 256-CU part),
    and the len % 4 tails around them."""
    out = []
    for base in (32 * 2 * 4096, 2 * 4096 * 256):
        for d in (-4097, -5, -1, 0, 1, 3, 4096):
            out.append(base + d)
    return out


@pytest.mark.parametrize("length", boundary_lengths())
def test_quantize_path_boundaries(esb, length):
    factors = wl.scale_grid(1.0).astype(np.float32)
    plan = esb.esb_dda_plan(5, 3, dev(factors))
    x = activations(length % 1000 + 31, length)
    log("quantize boundary len=%d" % length)
    compare(esb, dev(x), 5, 3, plan, factors.size, scalar(float(np.abs(x).max())),
            "len %d" % length)
