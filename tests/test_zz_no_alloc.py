"""esb_dda_align_noalloc, the DDA for callers that cannot allocate device memory
(its scratch is the library's static per-GPU array), against esb_dda_align with a
caller workspace on the same inputs: the chosen alpha and every D_j bit-identical,
on two calls in a row through the one shared array, the second on a smaller input
(the first call's contents must not leak into it)."""
import numpy as np
import pytest

from gpuutil import dev, host, log, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def both(esb, x, n, ks, grid):
    torch = torch_cuda()
    xd, gd = dev(x), dev(grid)
    a_ws, D_ws = esb.esb_dda_align(xd, n, ks, gd)
    a_na = torch.empty(1, dtype=torch.float32, device="cuda")
    D_na = torch.full((grid.size,), np.nan, dtype=torch.float64, device="cuda")
    esb.esb_dda_align_noalloc(xd, n, ks, gd, a_na, D_na)
    return host(a_ws), host(D_ws), host(a_na), host(D_na)


@pytest.mark.parametrize("order", ["large_then_small", "small_then_large_then_small"])
def test_noalloc_equals_workspace_call(esb, order):
    big = (np.random.default_rng(5).standard_normal(3_000_001) * 0.7).astype(np.float32)
    small = np.maximum(np.random.default_rng(6).standard_normal(40_000), 0).astype(np.float32)
    cases = [(big, 5, 3, wl.scale_grid(0.7)), (small, 4, 2, wl.scale_grid(1.0, 32))]
    if order != "large_then_small":
        cases = [cases[1], cases[0], cases[1]]
    for x, n, ks, grid in cases:
        log("dda noalloc len=%d n=%d k_sig=%d G=%d" % (x.size, n, ks, grid.size))
        a_ws, D_ws, a_na, D_na = both(esb, x, n, ks, grid)
        assert a_na[0] == a_ws[0]
        np.testing.assert_array_equal(D_na.view(np.uint64), D_ws.view(np.uint64))


def test_noalloc_empty_and_without_D(esb):
    torch = torch_cuda()
    grid = dev(wl.scale_grid(1.0))
    a = torch.full((1,), -1.0, dtype=torch.float32, device="cuda")
    esb.esb_dda_align_noalloc(dev(np.zeros(0, dtype=np.float32)), 4, 2, grid, a)
    a_ws, _ = esb.esb_dda_align(dev(np.zeros(0, dtype=np.float32)), 4, 2, grid)
    assert host(a)[0] == host(a_ws)[0]


def test_noalloc_refuses_inputs_beyond_the_scratch(esb):
    torch = torch_cuda()
    x = torch.empty(256, dtype=torch.uint8, device="cuda")   # validation fails before any read
    L = esb.lib()
    import ctypes
    big = 1 << 33
    assert esb.esb_dda_workspace_size(big, 4, 2, 64) > esb.ESB_DDA_NOALLOC_SCRATCH
    st = L.esb_dda_align_noalloc(ctypes.c_void_p(x.data_ptr()), big, 4, 2,
                                 ctypes.c_void_p(x.data_ptr()), 64, ctypes.c_void_p(x.data_ptr()),
                                 None, None)
    assert st == esb.ESB_E_SCRATCH
