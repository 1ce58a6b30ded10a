"""The ResNet18 stack (every convolution and the classifier quantized to ESB(5,2),
per-layer DDA on the device) against the same stack computed by the oracle from
the same input images.

The oracle quantizes every weight tensor and every layer input itself (DDA over
the grid 2^E c_j, E the binary exponent of max|x|, projection) and runs the direct
convolutions; the glue between layers (ReLU, max pool, residual sums, the
float64 average pool) is written again here in NumPy.  Each layer must agree
exactly: the chosen alpha, every code, every int32 accumulator; the fp32
outputs are fl32(s * fl32(acc)) on both sides.  Because each layer's output is
bit-identical, the two stacks stay in lockstep to the logits."""
import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, host, log
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
N, KS = 5, 3


def grid_np(x, cmax):
    """2^E c_j with E the binary exponent of max|x| (the stack's grid rule)."""
    m = np.float32(np.max(np.abs(x)))
    e = int(np.frexp(m)[1]) if m != 0 else 0
    return np.ldexp(wl.maxabs_grid_factors(cmax), e).astype(np.float32)


def quantize_np(x, cmax):
    g = grid_np(x, cmax)
    j, _ = oracle.dda(x, N, KS, g)
    return g[j], oracle.project(x, g[j], N, KS)


def maxpool_np(a):   # 3x3, stride 2, pad 1, NHWC
    B, H, W, C = a.shape
    P = (H + 2 - 3) // 2 + 1
    pad = np.full((B, H + 2, W + 2, C), -np.inf, dtype=np.float32)
    pad[:, 1:-1, 1:-1, :] = a
    out = np.full((B, P, P, C), -np.inf, dtype=np.float32)
    for r in range(3):
        for s in range(3):
            out = np.maximum(out, pad[:, r:r + 2 * P:2, s:s + 2 * P:2, :])
    return out


def avgpool_np(a):   # global average: float64 sum in position order, / HW, one rounding
    B, H, W, C = a.shape
    flat = a.reshape(B, H * W, C).astype(np.float64)
    acc = np.zeros((B, C), dtype=np.float64)
    for i in range(H * W):
        acc += flat[:, i, :]
    return (acc / float(H * W)).astype(np.float32)


@pytest.mark.parametrize("batch", [2])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_resnet18_stack_matches_oracle(batch, seed):
    import torch
    from paper_2109_03513_amd import resnet18
    weights = wl.resnet18_weights(0)
    x = wl.resnet18_input(seed, batch)
    log("resnet18 stack batch=%d seed=%d: GPU forward" % (batch, seed))
    model = resnet18.ResNet18ESB(weights, batch, record=True)
    logits = host(model.forward(torch.from_numpy(x).cuda()))
    cmax = resnet18.value_max(N, KS)
    gpu = {t["name"]: t for t in model.trace}

    def layer(name, a, w, stride, pad, wq, glue=None):
        """The oracle layer; the GPU trace holds its output after the epilogue's glue (ReLU,
        residual), which `glue` applies to the oracle's output in numpy fp32."""
        log("  oracle layer %s input %s" % (name, a.shape))
        alpha, codes = quantize_np(a, cmax)
        t = gpu[name]
        assert host(t["alpha"])[0] == alpha, name
        np.testing.assert_array_equal(host(t["codes"]), codes, err_msg=name)
        if name == "fc":
            st, acc, y = oracle.gemm(codes, wq[1], N, KS, alpha, N, KS, wq[0])
        else:
            st, acc, y = oracle.conv2d(codes, wq[1], N, KS, alpha, N, KS, wq[0],
                                       stride=(stride, stride), pad=(pad, pad))
        assert st == 0
        np.testing.assert_array_equal(host(t["acc"]), acc, err_msg=name)
        z = y if glue is None else glue(y)
        assert_rel(host(t["y"]), z, 1e-6, name)
        return z

    wq = {}
    for name, cin, cout, k, st, pd in wl.RESNET18_CONVS:
        wq[name] = quantize_np(weights[name], cmax)
        L = model.layers[name]
        assert host(L["alpha"])[0] == wq[name][0], name
        np.testing.assert_array_equal(host(L["codes"]), wq[name][1], err_msg=name)
    wq["fc"] = quantize_np(weights["fc"], cmax)
    geo = {name: (st, pd) for name, _, _, _, st, pd in wl.RESNET18_CONVS}

    def conv(name, a, glue=None):
        return layer(name, a, None, geo[name][0], geo[name][1], wq[name], glue)

    def relu(v):
        return np.maximum(v, 0.0).astype(np.float32)

    a = conv("conv1", x, relu)
    a = maxpool_np(a)
    # the fused conv1 + ReLU + pool call wrote exactly the pooled tensor
    np.testing.assert_array_equal(host(gpu["conv1"]["pooled"]).view(np.uint32), a.view(np.uint32))
    for stage in (1, 2, 3, 4):
        for blk in (0, 1):
            p = "l%d.%d." % (stage, blk)
            out = conv(p + "c1", a, relu)
            sc = conv(p + "ds", a) if (p + "ds") in geo else a
            a = conv(p + "c2", out, lambda v: relu(v + sc))
    feat = avgpool_np(a)
    y = layer("fc", feat, None, 1, 0, wq["fc"])
    assert_rel(logits, y, 1e-6, "logits")
    assert np.all(np.isfinite(logits))


def test_resnet18_fused_equals_dda_forward():
    """With the scales of a DDA forward fixed (calibration on the same batch), the fused
    forward (epilogues writing the next layer's codes) gives the same logits bit for bit:
    the epilogue's residual sum and ReLU are the glue's own fp32 operations.  The DDA
    forward on this input (seed 1) is itself compared with the oracle's stack in
    test_resnet18_stack_matches_oracle, so the fused logits are pinned to the oracle too."""
    import torch
    from paper_2109_03513_amd import resnet18
    batch = 2
    weights = wl.resnet18_weights(0)
    x = torch.from_numpy(wl.resnet18_input(1, batch)).cuda()
    model = resnet18.ResNet18ESB(weights, batch)
    log("resnet18 fused: calibration forward")
    ref = host(model.forward(x))
    log("resnet18 fused: fused forward")
    got = host(model.forward_fused(x))
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))
    again = host(model.forward_fused(x))
    np.testing.assert_array_equal(again.view(np.uint32), ref.view(np.uint32))
