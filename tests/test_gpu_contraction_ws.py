"""GPU contraction with a caller workspace (esb_gemm_ws, esb_conv2d_ws), where
shapes with enough work per operand byte decode both operands once (to packed
E2M1, packed E2M3 or E4M3, whichever holds both formats) ahead of the
contraction: bit-exact int32 accumulators and fp32 outputs within 1e-6
relative against the oracle, like the plain calls."""
import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
YREL = 1e-6


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def workspace(nbytes, fill=0xA5):
    torch = torch_cuda()
    return torch.full((max(nbytes, 1),), fill, dtype=torch.uint8, device="cuda")   # not zeroed


def sampled_rows(M, tile):
    r = sorted(set(list(range(0, min(M, 24))) + list(range(max(0, M - 24), M)) +
                   list(range(tile // 2, M, tile))))
    return np.array(r, dtype=np.int64)


@pytest.mark.parametrize("M,N,K,fa,fb", [
    (2049, 2050, 400, (5, 3), (5, 3)),     # decode-once path, ragged M and N
    (4097, 4100, 208, (4, 2), (4, 2)),     # 256 x 256 tiles, ragged K within a stage
    (1600, 1537, 1152, (5, 3), (4, 2)),    # mixed formats, 18 stages
    (64, 64, 576, (4, 2), (4, 2)),         # too little work: the workspace is not used
    (300, 257, 200, (3, 2), (3, 1)),       # K % 32 != 0: no E2M1 path, int8 table
    (2049, 2050, 416, (4, 2), (4, 2)),     # E2M1 (fp4) path: ESB(4,1) is exactly E2M1
    (2048, 2080, 576, (3, 2), (3, 1)),     # E2M1 path for the 3-bit formats
    (1537, 1600, 1024, (2, 1), (4, 2)),    # E2M1 path, mixed formats
    (4097, 4100, 576, (5, 3), (5, 3)),     # E2M3 (fp6) path (256 x 256 tiles): nine stages, ragged
    (4100, 4097, 1024, (6, 4), (6, 4)),    # E2M3 path, three fraction bits
    (4097, 4100, 640, (5, 3), (3, 2)),     # E2M3 path, mixed formats
    (2049, 2050, 576, (5, 3), (5, 3)),     # too few 256 x 256 tiles for the E2M3 path: E4M3
    (128, 4096, 9216, (3, 2), (3, 1)),     # AlexNet FC at batch 128: reduction split in 8 ranges
    (100, 3000, 4160, (5, 3), (5, 3)),     # split reduction, E4M3 decode in LDS, ragged last range
    (64, 2048, 8192, (3, 2), (3, 1)),      # 64 x 64 tiles, 16 ranges
])
def test_gemm_ws_sampled(esb, M, N, K, fa, fb):
    (bA, ksA), (bB, ksB) = fa, fb
    A = wl.random_codes(21, (M, K), 8)
    B = wl.random_codes(22, (N, K), 8)
    need = esb.esb_gemm_workspace_size(M, N, K, bA, ksA, bB, ksB)
    log("gemm_ws M=%d N=%d K=%d A=%s B=%s ws=%d" % (M, N, K, fa, fb, need))
    ws = workspace(need)
    acc, y = esb.esb_gemm(dev(A), bA, ksA, scalar(0.37), dev(B), bB, ksB, scalar(0.021), workspace=ws)
    rows = sampled_rows(M, 128)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, bA, ksA, 0.37, bB, ksB, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")


def test_gemm_ws_equals_plain_and_reuse(esb):
    """Two calls through one unzeroed workspace, the second smaller, equal the plain call."""
    for (M, N, K, seed) in [(2048, 2048, 1024, 1), (1536, 1664, 512, 2)]:
        A = dev(wl.random_codes(seed, (M, K), 8))
        B = dev(wl.random_codes(seed + 10, (N, K), 8))
        need = esb.esb_gemm_workspace_size(2048, 2048, 1024, 5, 3, 5, 3)
        ws = workspace(need) if seed == 1 else ws
        log("gemm_ws reuse M=%d N=%d K=%d" % (M, N, K))
        acc1, y1 = esb.esb_gemm(A, 5, 3, scalar(0.5), B, 5, 3, scalar(0.25), workspace=ws)
        acc0, y0 = esb.esb_gemm(A, 5, 3, scalar(0.5), B, 5, 3, scalar(0.25))
        np.testing.assert_array_equal(host(acc1), host(acc0))
        np.testing.assert_array_equal(host(y1).view(np.uint32), host(y0).view(np.uint32))


@pytest.mark.parametrize("case", [
    # N, H, W, C, K, R, stride, pad
    (8, 14, 14, 256, 256, 3, 1, 1),        # ResNet18 layer3 3x3 at batch 8
    (4, 15, 13, 128, 320, 3, 2, 1),        # stride 2, odd sizes, ragged N tile
    (2, 7, 7, 512, 512, 3, 1, 1),          # layer4 3x3
    (64, 56, 56, 64, 256, 3, 1, 1),        # 784 tiles of 256 x 256: the E2M3 path for ESB(5,2)
    (64, 7, 7, 512, 512, 3, 1, 1),         # ResNet18 layer4 at batch 64 (100 tiles of 128 x 128
                                           # are under half the CUs: 64 x 64 tiles)
    (64, 14, 14, 256, 512, 3, 2, 1),       # layer4's first conv (stride 2)
    (4, 224, 224, 3, 64, 7, 2, 3),         # image stem, C = 3: byte-gathering kernel
    (3, 33, 31, 24, 40, 1, 1, 0),          # C = 24 (1x1)
    (2, 57, 61, 5, 16, 3, 2, 1),           # C = 5, ragged everything
])
@pytest.mark.parametrize("fmt", [((5, 3), (5, 3)), ((4, 2), (4, 2)), ((3, 2), (3, 1)),
                                 ((4, 1), (4, 1))])
def test_conv_ws_parity(esb, case, fmt):
    Nb, H, W, C, K, R, st, pd = case
    (bX, ksX), (bW, ksW) = fmt
    x = wl.random_codes(31, (Nb, H, W, C), 8)
    w = wl.random_codes(32, (K, R, R, C), 8)
    need = esb.esb_conv2d_workspace_size(x.shape, w.shape, bX, ksX, bW, ksW, stride=(st, st),
                                         pad=(pd, pd))
    log("conv_ws %s fmt=%s ws=%d" % (case, fmt, need))
    ws = workspace(need)
    acc, y = esb.esb_conv2d(dev(x), bX, ksX, scalar(0.5), dev(w), bW, ksW, scalar(0.03),
                            stride=(st, st), pad=(pd, pd), workspace=ws)
    acc, y = host(acc), host(y)
    for img in sorted({0, Nb - 1}):
        s, oacc, oy = oracle.conv2d(np.ascontiguousarray(x[img:img + 1]), w, bX, ksX, 0.5, bW, ksW,
                                    0.03, stride=(st, st), pad=(pd, pd))
        assert s == 0
        np.testing.assert_array_equal(acc[img:img + 1], oacc)
        assert_rel(y[img:img + 1], oy, YREL, "y")


def extreme_codes(b, ks, shape, seed):
    v = oracle.valueset(b, ks)
    top = oracle.encode(float(v[-1]), b, ks)
    small = oracle.encode(float(v[v > 0][0]), b, ks)
    r = np.random.default_rng(seed)
    c = np.where(r.random(shape) < 0.8, top, small).astype(np.uint8)
    neg = r.random(shape) < 0.3
    return np.where(neg, c | (1 << (b - 1)), c).astype(np.uint8)


def test_gemm_ws_product_spread_at_accumulator_bound(esb):
    """ESB(5,2) on the decode-once path: products from 1 to 784 in one reduction and
    K * 784 just below 2^24, where every partial sum is still exact in fp32."""
    M, N, K = 1536, 1536, 21392
    A = extreme_codes(5, 3, (M, K), 3)
    B = extreme_codes(5, 3, (N, K), 4)
    need = esb.esb_gemm_workspace_size(M, N, K, 5, 3, 5, 3)
    assert need > 0
    log("gemm_ws spread M=%d N=%d K=%d" % (M, N, K))
    acc, y = esb.esb_gemm(dev(A), 5, 3, scalar(0.37), dev(B), 5, 3, scalar(0.021),
                          workspace=workspace(need))
    rows = np.array([0, 1, 777, M - 1], dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, 5, 3, 0.37, 5, 3, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")


def test_gemm_ws_e2m1_spread_at_accumulator_bound(esb):
    """ESB(4,1) on the E2M1 path: products m_A*m_B from 1 to 144 in one reduction and
    K * 144 just below 2^24 (every partial sum exact in fp32)."""
    M, N, K = 1536, 1536, 116480
    A = extreme_codes(4, 2, (M, K), 5)
    B = extreme_codes(4, 2, (N, K), 6)
    need = esb.esb_gemm_workspace_size(M, N, K, 4, 2, 4, 2)
    assert need > 0
    log("gemm_ws e2m1 spread M=%d N=%d K=%d" % (M, N, K))
    acc, y = esb.esb_gemm(dev(A), 4, 2, scalar(0.37), dev(B), 4, 2, scalar(0.021),
                          workspace=workspace(need))
    rows = np.array([0, 5, 1000, M - 1], dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, 4, 2, 0.37, 4, 2, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")


def test_gemm_ws_e2m3_spread_at_accumulator_bound(esb):
    """ESB(5,2) on the E2M3 (fp6) path (K % 64 == 0): products m_A*m_B from 1 to 784 in
    one reduction and K * 784 just below 2^24 (every partial sum exact in fp32)."""
    M, N, K = 4096, 4096, 21376
    A = extreme_codes(5, 3, (M, K), 7)
    B = extreme_codes(5, 3, (N, K), 8)
    need = esb.esb_gemm_workspace_size(M, N, K, 5, 3, 5, 3)
    assert need > 0
    log("gemm_ws e2m3 spread M=%d N=%d K=%d" % (M, N, K))
    acc, y = esb.esb_gemm(dev(A), 5, 3, scalar(0.37), dev(B), 5, 3, scalar(0.021),
                          workspace=workspace(need))
    rows = np.array([0, 3, 999, M - 1], dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, 5, 3, 0.37, 5, 3, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")


# The E4M3 (fp8) path at the edge of what the dispatcher admits for it: every product
# m_A * m_B at most 2^12 and K * max|m_A| * max|m_B| below 2^24.  ESB(4,0) (n = 4,
# k_sig = 1, Table 1's 4-bit power-of-two row) reaches the product bound exactly
# (m up to 64, p = 4096); ESB(6,3) (k_sig = 4) gives p = 60 * 60 = 3600.  Codes take the
# largest and the smallest nonzero magnitude at random, with random signs, so every
# 64-long slice of the reduction mixes products 2^12 apart, and K sits just below
# 2^24 / p.
FP8_EDGE = [
    # fmt, K of the GEMM (K % 16 == 0), conv (C, R) with R * R * C just below 2^24 / p
    ((4, 1), 4080, (448, 3)),
    ((6, 4), 4656, (512, 3)),
]


@pytest.mark.parametrize("fmt,K,convRC", FP8_EDGE)
@pytest.mark.parametrize("use_ws", [False, True])
def test_gemm_fp8_path_at_admission_bound(esb, fmt, K, convRC, use_ws):
    b, ks = fmt
    M, N = 640, 576
    MA = oracle.C(b, ks) * 2 ** (ks - 1)
    assert K * MA * MA < 2 ** 24 <= (K + 16) * MA * MA   # the largest K % 16 == 0 admitted
    A = extreme_codes(b, ks, (M, K), 11)
    B = extreme_codes(b, ks, (N, K), 12)
    ws = None
    if use_ws:
        need = esb.esb_gemm_workspace_size(M, N, K, b, ks, b, ks)
        assert need > 0
        ws = workspace(need)
    log("gemm fp8 edge fmt=%s M=%d N=%d K=%d ws=%s" % (fmt, M, N, K, use_ws))
    acc, y = esb.esb_gemm(dev(A), b, ks, scalar(0.37), dev(B), b, ks, scalar(0.021), workspace=ws)
    rows = np.array([0, 1, 129, 300, M - 1], dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, b, ks, 0.37, b, ks, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")


@pytest.mark.parametrize("fmt,K,convRC", FP8_EDGE)
@pytest.mark.parametrize("use_ws", [False, True])
def test_conv_fp8_path_at_admission_bound(esb, fmt, K, convRC, use_ws):
    b, ks = fmt
    C, R = convRC
    Nb, H, W, Kout = 4, 14, 14, 256
    x = extreme_codes(b, ks, (Nb, H, W, C), 13)
    w = extreme_codes(b, ks, (Kout, R, R, C), 14)
    ws = None
    if use_ws:
        need = esb.esb_conv2d_workspace_size(x.shape, w.shape, b, ks, b, ks, stride=(1, 1),
                                             pad=(1, 1))
        assert need > 0
        ws = workspace(need)
    log("conv fp8 edge fmt=%s x=%s w=%s ws=%s" % (fmt, x.shape, w.shape, use_ws))
    acc, y = esb.esb_conv2d(dev(x), b, ks, scalar(0.5), dev(w), b, ks, scalar(0.03), stride=(1, 1),
                            pad=(1, 1), workspace=ws)
    acc, y = host(acc), host(y)
    for img in (0, Nb - 1):
        s, oacc, oy = oracle.conv2d(np.ascontiguousarray(x[img:img + 1]), w, b, ks, 0.5, b, ks, 0.03,
                                    stride=(1, 1), pad=(1, 1))
        assert s == 0
        np.testing.assert_array_equal(acc[img:img + 1], oacc)
        assert_rel(y[img:img + 1], oy, YREL, "y")
