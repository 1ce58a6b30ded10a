"""GPU contraction with the fused post-processing (esb_gemm_post, esb_conv2d_post) vs the
oracle's contraction followed by its post-processing (eq. (16) affine, residual, ReLU,
projection): bit-exact int32 sums, bit-exact post-processed fp32 values and bit-exact
output codes, on every contraction path (k_contract, k_mma with the int8 table or E4M3
decode, the decode-once E4M3 / E2M1 / E2M3 kernels, the split reduction, depthwise)."""
import numpy as np
import pytest

import oracle
from gpuutil import dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu

ALPHA_A, ALPHA_B = 0.37, 0.021


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def workspace(nbytes):
    torch = torch_cuda()
    return torch.full((max(nbytes, 1),), 0xA5, dtype=torch.uint8, device="cuda")


def sampled_rows(M, tile):
    r = sorted(set(list(range(0, min(M, 24))) + list(range(max(0, M - 24), M)) +
                   list(range(tile // 2, M, tile))))
    return np.array(r, dtype=np.int64)


def post_params(seed, yref, channels, variant):
    """(a, b, residual (full output shape), relu, out_alpha) scaled to the outputs' spread."""
    r = np.random.default_rng(seed)
    sd = float(np.std(yref)) or 1.0
    a = b = res = None
    if variant in ("affine", "all"):
        a = r.uniform(-0.5, 1.5, channels).astype(np.float32)
        b = (r.standard_normal(channels) * 0.3 * sd).astype(np.float32)
    if variant in ("residual", "all"):
        res = "make"
    relu = variant in ("relu", "all")
    out_alpha = np.float32(0.4 * sd)
    return a, b, res, relu, out_alpha


GEMM_CASES = [
    # M, N, K, fa, fb, workspace, variant
    (300, 257, 200, (3, 2), (3, 1), False, "all"),      # k_mma, int8 table
    (100, 70, 50, (4, 2), (4, 2), False, "affine"),     # K % 16 != 0: k_contract
    (130, 90, 96, (8, 6), (5, 3), False, "all"),        # split int8: k_contract
    (500, 300, 512, (5, 3), (5, 3), False, "relu"),     # k_mma, E4M3 decode in LDS
    (2049, 2050, 400, (5, 3), (5, 3), True, "all"),     # decode-once E4M3
    (2049, 2050, 416, (4, 2), (4, 2), True, "residual"),  # decode-once E2M1 (fp4)
    (4097, 4100, 576, (5, 3), (5, 3), True, "all"),     # decode-once E2M3 (fp6), 256 x 256 tiles
    (128, 4096, 9216, (3, 2), (3, 1), True, "all"),     # split reduction (k_splitk_sum)
    (100, 3000, 4160, (5, 3), (5, 3), True, "relu"),    # split reduction, ragged last range
    (64, 64, 576, (4, 2), (4, 2), True, "none"),        # codes only, identity post
]


@pytest.mark.parametrize("M,N,K,fa,fb,ws,variant", GEMM_CASES)
@pytest.mark.parametrize("out", [(4, 2), (5, 3)])
def test_gemm_post(esb, M, N, K, fa, fb, ws, variant, out):
    torch = torch_cuda()
    (bA, ksA), (bB, ksB) = fa, fb
    A = wl.random_codes(31, (M, K), 8)
    B = wl.random_codes(32, (N, K), 8)
    rows = sampled_rows(M, 128) if M * N > 400000 else np.arange(M)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, bA, ksA, ALPHA_A, bB, ksB, ALPHA_B)
    assert st == 0
    a, b, res, relu, qa = post_params([M, N, K], oy, N, variant)
    R = None
    if res is not None:
        R = (np.random.default_rng(7).standard_normal((M, N)) * np.std(oy)).astype(np.float32)
    oz, ocodes = oracle.post(oy, out[0], out[1], qa, a=a, bias=b,
                             res=None if R is None else R[rows], relu=relu)
    w = workspace(esb.esb_gemm_workspace_size(M, N, K, bA, ksA, bB, ksB)) if ws else None
    log("gemm_post M=%d N=%d K=%d A=%s B=%s ws=%s variant=%s out=%s" % (M, N, K, fa, fb, ws,
                                                                       variant, out))
    amax = scalar(0.0)
    acc, y, codes = esb.esb_gemm_post(
        dev(A), bA, ksA, scalar(ALPHA_A), dev(B), bB, ksB, scalar(ALPHA_B), scalar(qa), out[0],
        out[1], a=None if a is None else dev(a), b=None if b is None else dev(b),
        residual=None if R is None else dev(R), relu=relu, want_acc=True, want_y=True,
        workspace=w, absmax=amax)
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    np.testing.assert_array_equal(host(y)[rows].view(np.uint32), oz.view(np.uint32))
    np.testing.assert_array_equal(host(codes)[rows], ocodes)
    check_absmax(host(amax)[0], oz, rows.size == M)


def check_absmax(got, oz, complete):
    """max |z| over the call: equal to the oracle's when every row was computed by the oracle,
    else at least the sampled rows' maximum."""
    want = np.float32(np.max(np.abs(oz))) if oz.size else np.float32(0)
    if complete:
        assert got == want, (got, want)
    else:
        assert got >= want


def test_gemm_post_codes_only_and_in_place_residual(esb):
    """Only codes requested; then y doubling as the residual (read before written)."""
    M, N, K = 700, 520, 384
    A = wl.random_codes(41, (M, K), 8)
    B = wl.random_codes(42, (N, K), 8)
    st, oacc, oy = oracle.gemm(A, B, 5, 3, ALPHA_A, 5, 3, ALPHA_B)
    qa = np.float32(0.3 * np.std(oy))
    _, oc = oracle.post(oy, 4, 2, qa, relu=True)
    acc, y, codes = esb.esb_gemm_post(dev(A), 5, 3, scalar(ALPHA_A), dev(B), 5, 3, scalar(ALPHA_B),
                                      scalar(qa), 4, 2, relu=True)
    assert acc is None and y is None
    np.testing.assert_array_equal(host(codes), oc)
    R = (np.random.default_rng(3).standard_normal((M, N)) * np.std(oy)).astype(np.float32)
    yd = dev(R.copy())
    oz, oc = oracle.post(oy, 5, 3, qa, res=R, relu=True)
    _, y, codes = esb.esb_gemm_post(dev(A), 5, 3, scalar(ALPHA_A), dev(B), 5, 3, scalar(ALPHA_B),
                                    scalar(qa), 5, 3, residual=yd, y=yd, relu=True)
    np.testing.assert_array_equal(host(y).view(np.uint32), oz.view(np.uint32))
    np.testing.assert_array_equal(host(codes), oc)


def test_gemm_post_invalid_output_scale(esb):
    """An output scale that is not a positive finite number gives +0 codes (as esb_project)."""
    M, N, K = 64, 64, 64
    A = wl.random_codes(51, (M, K), 8)
    B = wl.random_codes(52, (N, K), 8)
    for qa in (0.0, -1.0, np.inf, np.nan):
        _, _, codes = esb.esb_gemm_post(dev(A), 4, 2, scalar(0.5), dev(B), 4, 2, scalar(0.5),
                                        scalar(qa), 4, 2)
        assert (host(codes) == oracle.encode(0.0, 4, 2)).all()


CONV_CASES = [
    # N, H, W, C, K, R, S, stride, pad, groups, fx, fw, workspace, variant
    (4, 28, 28, 64, 64, 3, 3, 1, 1, 1, (5, 3), (5, 3), True, "all"),    # decode-once, conv
    (4, 28, 28, 64, 64, 3, 3, 1, 1, 1, (4, 2), (4, 2), True, "all"),    # decode-once E2M1 conv
    (2, 30, 30, 64, 96, 3, 3, 2, 1, 1, (5, 3), (5, 3), False, "all"),   # k_mma conv, stride 2
    (2, 14, 14, 32, 48, 1, 1, 1, 0, 1, (3, 2), (3, 1), False, "residual"),  # 1x1, int8 table
    (2, 17, 19, 24, 40, 3, 3, 1, 1, 2, (4, 2), (4, 2), False, "affine"),    # grouped: k_contract
    (2, 20, 20, 32, 32, 3, 3, 1, 1, 32, (5, 3), (5, 3), False, "all"),  # depthwise, 4 channels
    (1, 11, 13, 7, 7, 3, 3, 2, 1, 7, (4, 2), (4, 2), False, "all"),     # depthwise, scalar path
    (2, 64, 64, 3, 64, 7, 7, 2, 3, 1, (5, 3), (5, 3), True, "all"),     # C = 3 stem, workspace
    (16, 7, 7, 512, 512, 3, 3, 1, 1, 1, (5, 3), (5, 3), True, "all"),   # long reduction, few tiles
]


@pytest.mark.parametrize("Nb,H,W,C,K,R,S,stride,pad,groups,fx,fw,ws,variant", CONV_CASES)
def test_conv2d_post(esb, Nb, H, W, C, K, R, S, stride, pad, groups, fx, fw, ws, variant):
    (bX, ksX), (bW, ksW) = fx, fw
    x = wl.random_codes(61, (Nb, H, W, C), 8)
    w = wl.random_codes(62, (K, R, S, C // groups), 8)
    st, oacc, oy = oracle.conv2d(x, w, bX, ksX, ALPHA_A, bW, ksW, ALPHA_B, stride=(stride, stride),
                                 pad=(pad, pad), groups=groups)
    assert st == 0
    a, b, res, relu, qa = post_params([Nb, C, K], oy, K, variant)
    R_ = None
    if res is not None:
        R_ = (np.random.default_rng(8).standard_normal(oy.shape) * np.std(oy)).astype(np.float32)
    flat = oy.reshape(-1, K)
    oz, oc = oracle.post(flat, 5, 3, qa, a=a, bias=b,
                         res=None if R_ is None else R_.reshape(-1, K), relu=relu)
    d = dict(stride=(stride, stride), pad=(pad, pad), groups=groups)
    wsz = 0
    if ws:
        from paper_2109_03513_amd.esb import ConvDesc, lib
        import ctypes
        P_, Q_ = oy.shape[1], oy.shape[2]
        cd = ConvDesc(Nb, H, W, C, K, R, S, stride, stride, pad, pad, groups)
        wsz = lib().esb_conv2d_workspace_size(ctypes.byref(cd), bX, ksX, bW, ksW)
    log("conv_post %s groups=%d ws=%d variant=%s" % ((Nb, H, W, C, K, R, S, stride, pad), groups,
                                                     wsz, variant))
    amax = scalar(0.0)
    acc, y, codes = esb.esb_conv2d_post(
        dev(x), bX, ksX, scalar(ALPHA_A), dev(w), bW, ksW, scalar(ALPHA_B), scalar(qa), 5, 3,
        a=None if a is None else dev(a), b=None if b is None else dev(b),
        residual=None if R_ is None else dev(R_), relu=relu, want_acc=True, want_y=True,
        workspace=workspace(wsz) if ws else None, absmax=amax, **d)
    np.testing.assert_array_equal(host(acc), oacc)
    np.testing.assert_array_equal(host(y).reshape(-1, K).view(np.uint32), oz.view(np.uint32))
    np.testing.assert_array_equal(host(codes).reshape(-1, K), oc)
    check_absmax(host(amax)[0], oz, True)


def test_absmax_only_and_accumulation(esb):
    """Only the maximum requested; a second call raises the same scalar further."""
    M, N, K = 300, 200, 128
    A = wl.random_codes(71, (M, K), 8)
    B = wl.random_codes(72, (N, K), 8)
    st, _, oy = oracle.gemm(A, B, 5, 3, ALPHA_A, 5, 3, ALPHA_B)
    oz, _ = oracle.post(oy, 5, 3, 1.0, relu=True)
    amax = scalar(0.0)
    acc, y, codes = esb.esb_gemm_post(dev(A), 5, 3, scalar(ALPHA_A), dev(B), 5, 3, scalar(ALPHA_B),
                                      None, 5, 3, relu=True, want_codes=False, absmax=amax)
    assert acc is None and y is None and codes is None
    assert host(amax)[0] == np.float32(np.max(np.abs(oz)))
    big = np.float32(np.max(np.abs(oz)) * 4)
    amax2 = scalar(big)
    esb.esb_gemm_post(dev(A), 5, 3, scalar(ALPHA_A), dev(B), 5, 3, scalar(ALPHA_B), None, 5, 3,
                      relu=True, want_codes=False, absmax=amax2)
    assert host(amax2)[0] == big
