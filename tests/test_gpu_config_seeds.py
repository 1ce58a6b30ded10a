"""The four layer workloads end to end on the device, for seeds 0, 1 and 2 of the
synthetic inputs: the scale search (DDA, eq. (13)) of weights and activations,
their projection to ESB codes (eq. (8)) and the contraction over the codes
(eq. (15)), each step compared with the oracle on the same inputs: the chosen
alpha and every code and int32 accumulator bit-exact, scaled outputs within
1e-6 relative.

  tiny GEMM      64x576 N(0, 0.05) times 576x64 ReLU(N(0,1)), ESB(4,1) both;
  ResNet18 conv  3x3 64->64 at 56x56, batch 1, ESB(4,1) both;
  AlexNet FC     9216->4096 at batch 128, W ESB(3,0), X ESB(3,1);
  MobileNetV2    expand 1x1 24->144, depthwise 3x3 on 144, project 1x1 144->24,
                 batch 32 at 56x56, ESB(5,2) everywhere."""
import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, dev, host, log
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
YREL = 1e-6
SEEDS = [0, 1, 2]


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def quantize_both(esb, x, n, ks, grid, what):
    """Device DDA and projection of x, checked against the oracle; returns the device scale
    and codes with the oracle's scale and codes."""
    xd = dev(x)
    a, _ = esb.esb_dda_align(xd, n, ks, dev(grid))
    c = esb.esb_project(xd, a, n, ks)
    j, _ = oracle.dda(x, n, ks, grid)
    oc = oracle.project(x, grid[j], n, ks)
    assert host(a)[0] == grid[j], (what, host(a)[0], grid[j])
    np.testing.assert_array_equal(host(c), oc, err_msg=what)
    return a, c, grid[j], oc


@pytest.mark.parametrize("seed", SEEDS)
def test_tiny_gemm_seed(esb, seed):
    c = wl.tiny_gemm(seed)
    log("config tiny gemm seed %d" % seed)
    aW, cW, oaW, ocW = quantize_both(esb, c["W"], 4, 2, c["gridW"], "W")
    aA, cA, oaA, ocA = quantize_both(esb, c["A"], 4, 2, c["gridA"], "A")
    acc, y = esb.esb_gemm(cW, 4, 2, aW, cA, 4, 2, aA, b_layout=esb.ESB_B_KN)
    st, oacc, oy = oracle.gemm(ocW, ocA, 4, 2, oaW, 4, 2, oaA, b_layout=1)
    assert st == 0
    np.testing.assert_array_equal(host(acc), oacc)
    assert_rel(host(y), oy, YREL, "y")


@pytest.mark.parametrize("seed", SEEDS)
def test_resnet_conv_seed(esb, seed):
    c = wl.resnet_conv3x3(seed)
    log("config resnet conv seed %d" % seed)
    aW, cw, oaW, ocw = quantize_both(esb, c["w"], 4, 2, c["gridW"], "w")
    aX, cx, oaX, ocx = quantize_both(esb, c["x"], 4, 2, c["gridX"], "x")
    acc, y = esb.esb_conv2d(cx, 4, 2, aX, cw, 4, 2, aW, stride=c["stride"], pad=c["pad"])
    st, oacc, oy = oracle.conv2d(ocx, ocw, 4, 2, oaX, 4, 2, oaW, stride=c["stride"], pad=c["pad"])
    assert st == 0
    np.testing.assert_array_equal(host(acc), oacc)
    assert_rel(host(y), oy, YREL, "y")


@pytest.mark.parametrize("seed", SEEDS)
def test_alexnet_fc_seed(esb, seed):
    c = wl.alexnet_fc(seed)
    log("config alexnet fc seed %d" % seed)
    aW, cW, oaW, ocW = quantize_both(esb, c["W"], 3, 1, c["gridW"], "W")
    aX, cX, oaX, ocX = quantize_both(esb, c["X"], 3, 2, c["gridX"], "X")
    acc, y = esb.esb_gemm(cX, 3, 2, aX, cW, 3, 1, aW)
    st, oacc, oy = oracle.gemm(ocX, ocW, 3, 2, oaX, 3, 1, oaW)
    assert st == 0
    np.testing.assert_array_equal(host(acc), oacc)
    assert_rel(host(y), oy, YREL, "y")


@pytest.mark.parametrize("seed", SEEDS)
def test_mobilenet_block_seed(esb, seed):
    m = wl.mobilenetv2_block(seed)
    for L in m["layers"]:
        log("config mobilenet %s seed %d" % (L["name"], seed))
        aW, cw, oaW, ocw = quantize_both(esb, L["w"], 5, 3, m["gridW"], "w " + L["name"])
        aX, cx, oaX, ocx = quantize_both(esb, L["x"], 5, 3, m["gridX"], "x " + L["name"])
        acc, y = esb.esb_conv2d(cx, 5, 3, aX, cw, 5, 3, aW, stride=L["stride"], pad=L["pad"],
                                groups=L["groups"])
        st, oacc, oy = oracle.conv2d(ocx, ocw, 5, 3, oaX, 5, 3, oaW, stride=L["stride"],
                                     pad=L["pad"], groups=L["groups"])
        assert st == 0
        np.testing.assert_array_equal(host(acc), oacc, err_msg=L["name"])
        assert_rel(host(y), oy, YREL, "y " + L["name"])
