"""The direct 3x3 / pad-1 convolution kernels, stride 1 and 2 (input and output channels in
multiples of 64 on the fp8 MFMA; tiles of 256, 128 or 64 output pixels over the batch,
crossing image boundaries; input channels in chunks of 64; the filter slice per chunk, or
resident for the workgroup; with stride 2 the even padded columns of a patch row first)
against the oracle's convolution
and post-processing: bit-exact int32 sums, fp32 outputs and codes, equal running maximum;
and bit for bit equal to the implicit-GEMM path, which an input one byte off a 16-byte
boundary takes."""
import numpy as np
import pytest

import oracle
from gpuutil import dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
ALPHA_X, ALPHA_W = 0.43, 0.027


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def unaligned(torch, a):
    """A device copy of the uint8 array a whose data starts one byte past a 16-byte boundary."""
    buf = torch.empty(a.size + 16, dtype=torch.uint8, device="cuda")
    v = buf[1:1 + a.size].view(a.shape)
    v.copy_(torch.from_numpy(np.ascontiguousarray(a)))
    assert v.data_ptr() % 16 == 1
    return v


CASES = [
    # N, H, W, C, K, fx, fw, variant
    (2, 56, 56, 64, 64, (5, 3), (5, 3), "plain"),     # the ResNet18 l1 shape, batch 2
    (3, 7, 7, 64, 64, (5, 3), (5, 3), "all"),         # 49-pixel images: a tile spans six of them
    (1, 13, 5, 64, 64, (4, 2), (5, 3), "relu"),       # H != W, ragged last tile, mixed formats
    (2, 9, 62, 64, 64, (5, 3), (4, 2), "residual"),   # widest rows taken (Q + 2 = 64)
    (1, 1, 1, 64, 64, (5, 3), (5, 3), "affine"),      # one pixel
    (4, 17, 23, 64, 64, (6, 3), (4, 1), "all"),       # ESB(6,3) x ESB(4,1)
    # several chunks of input channels and / or tiles of output channels
    (2, 28, 28, 128, 128, (5, 3), (5, 3), "all"),     # the l2 shape, batch 2 (1568 pixels)
    (3, 14, 14, 256, 192, (5, 3), (4, 2), "relu"),    # four chunks, three channel tiles
    (1, 5, 9, 192, 64, (5, 3), (5, 3), "residual"),   # three chunks, ragged
    (2, 7, 7, 512, 128, (5, 3), (5, 3), "plain"),     # eight chunks (the l4 reduction)
    # one chunk: 64-pixel tiles when tiles of 128 give fewer workgroups than CUs; several
    # chunks: 128-pixel tiles down to half a workgroup per CU
    (50, 7, 7, 128, 512, (5, 3), (5, 3), "plain"),    # several chunks, 128-pixel tiles
    (16, 14, 14, 64, 512, (5, 3), (5, 3), "affine"),  # one chunk, eight channel tiles
    (8, 1, 40, 128, 64, (5, 3), (5, 3), "all"),       # several chunks, 64-pixel tiles (one-row
                                                      # images: 128 pixels need 15 patch rows)
    # several chunks and more than 16384 pixels: the resident-filter kernel (eight waves,
    # one workgroup per CU, 64 or 32 output channels per workgroup)
    (24, 28, 28, 128, 128, (5, 3), (5, 3), "all"),    # 64 channels per workgroup, ragged
    (88, 14, 14, 256, 64, (5, 3), (4, 2), "plain"),   # 32 channels per workgroup
]
# stride 2 (output (H - 1) / 2 + 1): N, H, W, C, K, fx, fw, variant.  The direct kernel
# takes 256 or more input channels; the others check the implicit-GEMM path.
CASES_S2 = [
    (2, 14, 14, 256, 512, (5, 3), (4, 2), "plain"),   # l4.0.c1: four chunks, eight channel tiles
    (3, 7, 7, 256, 64, (6, 3), (4, 1), "all"),        # 4 x 4 outputs per image
    (2, 9, 11, 320, 128, (5, 3), (5, 3), "residual"), # five chunks, odd H and W
    (4, 15, 17, 256, 64, (4, 2), (5, 3), "relu"),     # H != W, ragged last tile
    (1, 1, 1, 256, 64, (5, 3), (5, 3), "affine"),     # one input pixel, one output
    (2, 30, 62, 256, 64, (5, 3), (5, 3), "relu"),     # W + 2 = 64: 11 patch rows, implicit GEMM
    (2, 56, 56, 64, 128, (5, 3), (5, 3), "all"),      # the ResNet18 l2.0.c1 shape, batch 2
    (3, 28, 28, 128, 256, (5, 3), (5, 3), "relu"),    # l3.0.c1
    (2, 13, 9, 64, 64, (5, 3), (5, 3), "residual"),   # odd H, W
]


def post_params(seed, y, K, variant):
    r = np.random.default_rng(seed)
    sd = float(np.std(y)) or 1.0
    a = b = res = None
    if variant in ("affine", "all"):
        a = r.uniform(-0.5, 1.5, K).astype(np.float32)
        b = (r.standard_normal(K) * 0.3 * sd).astype(np.float32)
    if variant in ("residual", "all"):
        res = (r.standard_normal(y.shape) * sd).astype(np.float32)
    relu = variant in ("relu", "all")
    return a, b, res, relu, np.float32(0.4 * sd)


@pytest.mark.parametrize("stride,Nb,H,W,C,K,fx,fw,variant",
                         [(1,) + c for c in CASES] + [(2,) + c for c in CASES_S2])
def test_conv3x3_direct(esb, stride, Nb, H, W, C, K, fx, fw, variant):
    torch = torch_cuda()
    x = wl.random_codes(40 + H + C, (Nb, H, W, C), fx[0])
    w = wl.random_codes(41 + W + K, (K, 3, 3, C), fw[0])
    sd = (stride, stride)
    st, acc_o, y_o = oracle.conv2d(x, w, fx[0], fx[1], ALPHA_X, fw[0], fw[1], ALPHA_W,
                                   stride=sd, pad=(1, 1))
    assert st == 0
    log("conv3x3 direct stride %d %s %s" % (stride, (Nb, H, W, C, K, fx, fw), variant))
    if variant == "plain":
        for want_acc in (True, False):
            acc, y = esb.esb_conv2d(dev(x), fx[0], fx[1], scalar(ALPHA_X), dev(w), fw[0], fw[1],
                                    scalar(ALPHA_W), stride=sd, pad=(1, 1), want_acc=want_acc)
            np.testing.assert_array_equal(host(y).view(np.uint32), y_o.view(np.uint32))
            if want_acc:
                np.testing.assert_array_equal(host(acc), acc_o)
        acc_u, y_u = esb.esb_conv2d(unaligned(torch, x), fx[0], fx[1], scalar(ALPHA_X), dev(w),
                                    fw[0], fw[1], scalar(ALPHA_W), stride=sd, pad=(1, 1))
        np.testing.assert_array_equal(host(acc_u), acc_o)
        np.testing.assert_array_equal(host(y_u).view(np.uint32), y_o.view(np.uint32))
        return
    a, b, res, relu, qa = post_params(7, y_o, K, variant)
    z_o, codes_o = oracle.post(y_o.reshape(-1, K), 5, 3, qa, a=a, bias=b,
                               res=None if res is None else res.reshape(-1, K), relu=relu)
    z_o = z_o.reshape(y_o.shape)
    codes_o = codes_o.reshape(y_o.shape)
    outs = []
    for xin, want_acc in ((dev(x), True), (dev(x), False), (unaligned(torch, x), True)):
        amax = scalar(0.0)
        acc, y, codes = esb.esb_conv2d_post(
            xin, fx[0], fx[1], scalar(ALPHA_X), dev(w), fw[0], fw[1], scalar(ALPHA_W),
            scalar(qa), 5, 3, a=None if a is None else dev(a), b=None if b is None else dev(b),
            residual=None if res is None else dev(res), relu=relu, stride=sd, pad=(1, 1),
            want_codes=True, want_acc=want_acc, want_y=True, absmax=amax)
        np.testing.assert_array_equal(host(y).view(np.uint32), z_o.view(np.uint32))
        np.testing.assert_array_equal(host(codes), codes_o)
        assert host(amax)[0] == np.max(np.abs(z_o))
        if want_acc:
            np.testing.assert_array_equal(host(acc), acc_o)
        outs.append(host(y))
    np.testing.assert_array_equal(outs[0].view(np.uint32), outs[2].view(np.uint32))


def random_shapes(count, seed=2109):
    """Seeded shapes in the direct kernels' domain (channels in multiples of 64, stride 1
    or 2), each at most about 1.5e8 multiply-adds so that the oracle finishes quickly."""
    r = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        st = int(r.choice([1, 2]))
        C = 64 * int(r.choice([1, 2, 3, 4, 5, 8]))
        K = 64 * int(r.choice([1, 2, 3]))
        H, W = int(r.integers(1, 41)), int(r.integers(1, 41))
        Nb = int(r.integers(1, 5))
        P, Q = (H - 1) // st + 1, (W - 1) // st + 1
        if Nb * P * Q * K * 9 * C > 150_000_000:
            continue
        out.append((st, Nb, H, W, C, K))
    return out


@pytest.mark.parametrize("st,Nb,H,W,C,K", random_shapes(24))
def test_conv3x3_direct_random_shapes(esb, st, Nb, H, W, C, K):
    """Plain outputs and int32 sums against the oracle on seeded shapes: ragged tiles, tiles
    across images, odd and even chunk counts, both strides (stride 2 below 256 channels and
    shapes the direct kernels do not take run the implicit GEMM: the same results)."""
    x = wl.random_codes(5000 + H * W + C, (Nb, H, W, C), 5)
    w = wl.random_codes(6000 + K + C, (K, 3, 3, C), 5)
    sd = (st, st)
    status, acc_o, y_o = oracle.conv2d(x, w, 5, 3, ALPHA_X, 5, 3, ALPHA_W, stride=sd, pad=(1, 1))
    assert status == 0
    log("conv3x3 random stride %d %s" % (st, (Nb, H, W, C, K)))
    acc, y = esb.esb_conv2d(dev(x), 5, 3, scalar(ALPHA_X), dev(w), 5, 3, scalar(ALPHA_W),
                            stride=sd, pad=(1, 1), want_acc=True)
    np.testing.assert_array_equal(host(acc), acc_o)
    np.testing.assert_array_equal(host(y).view(np.uint32), y_o.view(np.uint32))
