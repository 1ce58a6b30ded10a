"""Pins of the oracle's contraction (GEMM and convolution over ESB codes):
an fp64 dot product on decoded values, integer arithmetic on an independently
built decode table, im2col equivalence, the output scaling and the contract."""
import numpy as np
import pytest

import oracle
from paper_2109_03513_amd import workloads

from test_oracle_valueset import minifloat_values


def int_table(b, ks):
    """m = q * 2^k per code from the minifloat construction (not from eq. (14) code)."""
    k = ks - 1
    ebits = b - k - 1
    emax = (1 << ebits) - 1
    t = np.zeros(256, dtype=np.int64)
    for c in range(256):
        cc = c & ((1 << b) - 1)
        s, e, f = (cc >> (b - 1)) & 1, (cc >> k) & emax, cc & ((1 << k) - 1)
        # minifloat with bias 1 where the all-ones exponent field plays the subnormal role
        m = f if e == emax else ((1 << k) + f) << e
        t[c] = -m if s else m
    assert set(np.abs(t[: 1 << b]) / 2.0 ** k) == set(minifloat_values(b, ks))
    return t


def dec_table(b, ks):
    return np.array([oracle.decode(c, b, ks) for c in range(256)])


GEMM_CASES = [((7, 5, 33), (4, 2), (4, 2)), ((64, 64, 576), (4, 2), (4, 2)),
              ((19, 37, 130), (3, 2), (3, 1)), ((16, 8, 64), (5, 3), (5, 3)),
              ((5, 9, 40), (5, 2), (8, 7)), ((3, 4, 17), (8, 5), (6, 3))]


@pytest.mark.parametrize("shape,fa,fb", GEMM_CASES)
@pytest.mark.parametrize("layout", [0, 1])
def test_gemm_matches_integer_and_fp64_dot(shape, fa, fb, layout):
    M, N, K = shape
    (bA, ksA), (bB, ksB) = fa, fb
    A = workloads.random_codes(1, (M, K), bA)
    Bnk = workloads.random_codes(2, (N, K), bB)
    B = Bnk if layout == 0 else np.ascontiguousarray(Bnk.T)
    aA, aB = np.float32(0.37), np.float32(0.021)
    st, acc, y = oracle.gemm(A, B, bA, ksA, aA, bB, ksB, aB, b_layout=layout)
    assert st == 0
    ref = int_table(bA, ksA)[A] @ int_table(bB, ksB)[Bnk].T
    np.testing.assert_array_equal(acc, ref)
    dot = dec_table(bA, ksA)[A] @ dec_table(bB, ksB)[Bnk].T       # fp64, exact for these sizes
    np.testing.assert_array_equal(dot, acc * 2.0 ** -((ksA - 1) + (ksB - 1)))
    s = np.float32(np.ldexp(np.float32(aA * aB), -((ksA - 1) + (ksB - 1))))
    np.testing.assert_array_equal(y, s * acc.astype(np.float32))


def test_gemm_contract_errors():
    A = np.zeros((2, 4), np.uint8)
    # ESB(6, k=1): N = 15, max |m| = 3 * 2^14 > 32767 -> unsupported
    assert oracle.gemm(A, A, 6, 2, 1.0, 6, 2, 1.0)[0] == oracle.ESO_E_UNSUPPORTED
    # ESB(8, k=4): max |m| = 1984; K * 1984^2 > 2^31 - 1 for K = 600
    A = np.zeros((1, 600), np.uint8)
    assert oracle.gemm(A, A, 8, 5, 1.0, 8, 5, 1.0)[0] == oracle.ESO_E_OVERFLOW
    A = np.zeros((1, 545), np.uint8)
    assert oracle.gemm(A, A, 8, 5, 1.0, 8, 5, 1.0)[0] == 0


def im2col(x, R, S, stride, pad):
    Nb, H, W, C = x.shape
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    cols = np.zeros((Nb, P, Q, R, S, C), dtype=np.int64)
    for r in range(R):
        for s in range(S):
            for p in range(P):
                ih = p * stride[0] - pad[0] + r
                if ih < 0 or ih >= H:
                    continue
                for q in range(Q):
                    iw = q * stride[1] - pad[1] + s
                    if 0 <= iw < W:
                        cols[:, p, q, r, s, :] = x[:, ih, iw, :]
    return cols.reshape(Nb * P * Q, R * S * C), (Nb, P, Q)


CONV_CASES = [
    (1, 9, 11, 8, 16, 3, (1, 1), (1, 1), 1),
    (2, 8, 8, 3, 5, 7, (2, 2), (3, 3), 1),
    (1, 7, 6, 16, 16, 3, (2, 1), (1, 0), 1),
    (2, 6, 6, 12, 12, 3, (1, 1), (1, 1), 12),   # depthwise
    (1, 5, 5, 8, 4, 1, (2, 2), (0, 0), 2),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_equals_im2col_gemm(case):
    Nb, H, W, C, Kout, R, stride, pad, groups = case
    bX, ksX, bW, ksW = 5, 3, 4, 2
    x = workloads.random_codes(3, (Nb, H, W, C), bX)
    w = workloads.random_codes(4, (Kout, R, R, C // groups), bW)
    st, acc, y = oracle.conv2d(x, w, bX, ksX, 0.5, bW, ksW, 0.25, stride=stride, pad=pad, groups=groups)
    assert st == 0
    tX, tW = int_table(bX, ksX), int_table(bW, ksW)
    Cg, Kg = C // groups, Kout // groups
    out = np.zeros(acc.shape, dtype=np.int64)
    for g in range(groups):
        cols, (n_, P, Q) = im2col(tX[x[..., g * Cg:(g + 1) * Cg]], R, R, stride, pad)
        wg = tW[w[g * Kg:(g + 1) * Kg]].reshape(Kg, -1)
        out[..., g * Kg:(g + 1) * Kg] = (cols @ wg.T).reshape(n_, P, Q, Kg)
    np.testing.assert_array_equal(acc, out)
    s = np.float32(np.ldexp(np.float32(np.float32(0.5) * np.float32(0.25)), -(2 + 1)))
    np.testing.assert_array_equal(y, s * acc.astype(np.float32))


def test_conv_zero_padding_is_value_zero():
    """Padding contributes value 0, not the decoded value of code 0x00 (which is 1.0)."""
    x = np.zeros((1, 1, 1, 1), np.uint8)       # code 0 = +1.0 in ESB(4, k=1)
    w = np.zeros((1, 3, 3, 1), np.uint8)
    st, acc, _ = oracle.conv2d(x, w, 4, 2, 1.0, 4, 2, 1.0, pad=(1, 1))
    assert st == 0 and acc.shape == (1, 1, 1, 1)
    assert acc[0, 0, 0, 0] == 2 * 2             # only the centre tap: m = 2 each
