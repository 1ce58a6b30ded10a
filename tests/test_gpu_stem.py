"""Convolution + post-processing with a ReLU + max pooling in one call
(esb_conv2d_relu_maxpool): the fused stem kernel (stride 2, C <= 3, 64 output
channels, pool 3 / 2 / 1) and the general path through a workspace, against the
oracle's convolution and post-processing followed by a NumPy max pool: pooled
fp32 outputs and their codes bit-exact, the running maximum equal."""
import numpy as np
import pytest

import oracle
from gpuutil import dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
ALPHA_X, ALPHA_W = 0.61, 0.043


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def pool_ref(z, r, st, pd):
    """Max over windows, positions outside z left out (z >= 0 after the ReLU)."""
    B, H, W, C = z.shape
    P = (H + 2 * pd - r) // st + 1
    Q = (W + 2 * pd - r) // st + 1
    out = np.zeros((B, P, Q, C), dtype=np.float32)
    for i in range(P):
        for j in range(Q):
            h0, w0 = i * st - pd, j * st - pd
            win = z[:, max(h0, 0):min(h0 + r, H), max(w0, 0):min(w0 + r, W), :]
            out[:, i, j, :] = win.max(axis=(1, 2))
    return out


def reference(x, w, fx, fw, stride, pad, a, b, qa, fo, pool):
    st, _, y = oracle.conv2d(x, w, fx[0], fx[1], ALPHA_X, fw[0], fw[1], ALPHA_W, stride=stride,
                             pad=pad, want_acc=False)
    assert st == 0
    K = w.shape[0]
    z, _ = oracle.post(y.reshape(-1, K), fo[0], fo[1], qa, a=a, bias=b, relu=True)
    pooled = pool_ref(z.reshape(y.shape), *pool)
    codes = oracle.project(pooled, qa, fo[0], fo[1])
    return pooled, codes


CASES = [
    # N, H, W, C, K, R, stride, pad, fx, fw, with a/b, fused
    (2, 224, 224, 3, 64, 7, 2, 3, (5, 3), (5, 3), False, True),   # the ResNet18 stem
    (3, 37, 41, 3, 64, 7, 2, 3, (4, 2), (5, 3), True, True),      # ragged tiles
    (2, 30, 30, 2, 64, 5, 2, 2, (3, 1), (4, 2), True, True),      # C = 2, 5 x 5
    (1, 19, 23, 1, 64, 3, 2, 1, (5, 3), (3, 2), False, True),     # C = 1, 3 x 3
    (2, 20, 20, 8, 64, 3, 2, 1, (5, 3), (5, 3), True, False),     # C = 8: general path
    (2, 18, 18, 3, 32, 3, 1, 1, (5, 3), (5, 3), False, False),    # stride 1, K = 32: general
]


@pytest.mark.parametrize("Nb,H,W,C,K,R,st,pd,fx,fw,ab,fused", CASES)
def test_conv_relu_maxpool(esb, Nb, H, W, C, K, R, st, pd, fx, fw, ab, fused):
    torch = torch_cuda()
    x = wl.random_codes(90 + C, (Nb, H, W, C), 8)
    w = wl.random_codes(91 + R, (K, R, R, C), 8)
    r = np.random.default_rng(5)
    a = (r.random(K) + 0.5).astype(np.float32) if ab else None
    b = (r.standard_normal(K) * 0.1).astype(np.float32) if ab else None
    qa = np.float32(0.35)
    fo = (5, 3)
    pooled, codes = reference(x, w, fx, fw, (st, st), (pd, pd), a, b, qa, fo, (3, 2, 1))
    need = esb.esb_conv2d_relu_maxpool_workspace_size(x.shape, w.shape, fx[0], fx[1], fw[0], fw[1],
                                                      stride=(st, st), pad=(pd, pd))
    assert (need == 0) == fused
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda") if need else None
    amax = scalar(0.0)
    log("conv_relu_maxpool %s fused=%s" % ((Nb, H, W, C, K, R, st, pd, fx, fw), fused))
    y, c = esb.esb_conv2d_relu_maxpool(dev(x), fx[0], fx[1], scalar(ALPHA_X), dev(w), fw[0], fw[1],
                                       scalar(ALPHA_W), out_alpha=scalar(qa), out_n=fo[0],
                                       out_k_sig=fo[1], a=None if a is None else dev(a),
                                       b=None if b is None else dev(b), stride=(st, st),
                                       pad=(pd, pd), want_codes=True, absmax=amax, workspace=ws)
    np.testing.assert_array_equal(host(y).view(np.uint32), pooled.view(np.uint32))
    np.testing.assert_array_equal(host(c), codes)
    assert host(amax)[0] == np.max(pooled)


def test_stem_batch64_sampled(esb):
    """The ResNet18 stem at batch 64 (the bench's shape): first and last image."""
    x = wl.random_codes(77, (64, 224, 224, 3), 8)
    w = wl.random_codes(78, (64, 7, 7, 3), 8)
    log("stem batch 64")
    y, _ = esb.esb_conv2d_relu_maxpool(dev(x), 5, 3, scalar(ALPHA_X), dev(w), 5, 3,
                                       scalar(ALPHA_W), stride=(2, 2), pad=(3, 3))
    y = host(y)
    for i in (0, 63):
        pooled, _ = reference(np.ascontiguousarray(x[i:i + 1]), w, (5, 3), (5, 3), (2, 2), (3, 3),
                              None, None, np.float32(1.0), (5, 3), (3, 2, 1))
        np.testing.assert_array_equal(y[i:i + 1].view(np.uint32), pooled.view(np.uint32))


def test_fused_equals_conv_then_pool(esb):
    """The fused call equals esb_conv2d_post (ReLU) followed by esb_maxpool2d, bit for bit."""
    x = dev(wl.random_codes(80, (4, 64, 64, 3), 8))
    w = dev(wl.random_codes(81, (64, 7, 7, 3), 8))
    y, _ = esb.esb_conv2d_relu_maxpool(x, 5, 3, scalar(ALPHA_X), w, 5, 3, scalar(ALPHA_W),
                                       stride=(2, 2), pad=(3, 3))
    _, z, _ = esb.esb_conv2d_post(x, 5, 3, scalar(ALPHA_X), w, 5, 3, scalar(ALPHA_W), None, 5, 3,
                                  relu=True, stride=(2, 2), pad=(3, 3), want_codes=False,
                                  want_y=True)
    p = esb.esb_maxpool2d(z, 3, 2, 1)
    np.testing.assert_array_equal(host(y).view(np.uint32), host(p).view(np.uint32))


@pytest.mark.parametrize("qa", [0.35, 1e-38])
def test_stem_unaligned_outputs_and_scales(esb, qa):
    """Outputs one element past a 16-byte boundary take the per-channel stores, and a
    subnormal output scale takes the exact (division) code path: both bit-exact."""
    torch = torch_cuda()
    Nb, H, W, C, R = 2, 45, 38, 3, 7
    x = wl.random_codes(95, (Nb, H, W, C), 8)
    w = wl.random_codes(96, (64, R, R, C), 8)
    qa = np.float32(qa)
    pooled, codes = reference(x, w, (5, 3), (5, 3), (2, 2), (3, 3), None, None, qa, (5, 3),
                              (3, 2, 1))
    n = pooled.size
    ybuf = torch.zeros(n + 1, dtype=torch.float32, device="cuda")
    cbuf = torch.zeros(n + 1, dtype=torch.uint8, device="cuda")
    y = ybuf[1:].view(pooled.shape)
    c = cbuf[1:].view(pooled.shape)
    assert y.data_ptr() % 16 != 0 and c.data_ptr() % 4 != 0
    amax = scalar(0.0)
    log("stem unaligned outputs qa=%g" % qa)
    esb.esb_conv2d_relu_maxpool(dev(x), 5, 3, scalar(ALPHA_X), dev(w), 5, 3, scalar(ALPHA_W),
                                out_alpha=scalar(qa), out_n=5, out_k_sig=3, stride=(2, 2),
                                pad=(3, 3), y=y, codes=c, want_codes=True, absmax=amax)
    np.testing.assert_array_equal(host(y).view(np.uint32), pooled.view(np.uint32))
    np.testing.assert_array_equal(host(c), codes)
    assert host(ybuf)[0] == 0 and host(cbuf)[0] == 0
    assert host(amax)[0] == np.max(pooled)
