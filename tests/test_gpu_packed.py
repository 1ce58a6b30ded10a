"""Packed 4-bit code storage (esb_pack) and the GEMM that reads it in place
(esb_gemm_packed), against the oracle: bit-exact int32 accumulators, fp32 outputs
within 1e-6 relative, and bit-identical to esb_gemm on the same codes.

The packed layout is pinned independently of the contraction: every nibble,
read through the OCP E2M1 value table (tests/golden/ocp_fp4_e2m1.txt), equals the
oracle's value of the code it stores, at the position the header documents."""
import os

import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, dev, host, log, scalar, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
YREL = 1e-6
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def e2m1_table():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "ocp_fp4_e2m1.txt"))
            if l.strip() and not l.startswith("#")]
    return np.array([float(t) for t in rows[0]])


def workspace(nbytes):
    torch = torch_cuda()
    return torch.full((max(nbytes, 1),), 0x5A, dtype=torch.uint8, device="cuda")   # not zeroed


@pytest.mark.parametrize("fmt", [(4, 2), (3, 1), (3, 2), (2, 1)])
def test_pack_layout_is_e2m1(esb, fmt):
    n, ks = fmt
    rows, K = 37, 96
    codes = wl.random_codes(41, (rows, K), n)
    log("pack layout fmt=%s" % (fmt,))
    packed = host(esb.esb_pack(dev(codes), n, ks))
    assert packed.shape == (rows, K // 2)
    mag = e2m1_table()
    tab = np.array([oracle.decode(c, n, ks) for c in range(1 << n)])
    vals = tab[codes]
    for r in (0, 17, rows - 1):
        for g in range(K // 32):
            blk = packed[r, 16 * g:16 * g + 16]
            for w in range(4):
                for i in range(4):
                    byte = int(blk[4 * w + i])
                    for half, c in ((byte & 15, 8 * w + i), (byte >> 4, 8 * w + 4 + i)):
                        v = mag[half & 7] * (-1.0 if half & 8 else 1.0)
                        q = float(vals[r, 32 * g + c])
                        assert v == q or (v == 0.0 and q == 0.0), (fmt, r, g, w, i, half, q)


@pytest.mark.parametrize("M,N,K,fa,fb", [
    (128, 4096, 9216, (3, 2), (3, 1)),     # AlexNet FC at batch 128: the reduction split over
                                           # the waves of one workgroup per 64 x 32 tile
    (100, 4001, 4160, (4, 2), (3, 1)),     # same kernel: ragged M and N (N % 4 != 0: unaligned
                                           # rows), a partial last 128-byte line (32 bytes)
    (200, 2600, 8256, (3, 2), (4, 2)),     # same kernel: four M tiles, the last of 8 rows
    (301, 1000, 2048, (4, 2), (4, 2)),     # ragged M, N; ESB(4,1) both
    (4097, 2050, 512, (2, 1), (3, 2)),     # many tiles: no split
    (64, 3000, 8192, (3, 2), (4, 2)),      # 64 x 64 tiles, split over workgroups
])
def test_gemm_packed_vs_oracle(esb, M, N, K, fa, fb):
    (bA, ksA), (bB, ksB) = fa, fb
    A = wl.random_codes(43, (M, K), bA)
    B = wl.random_codes(44, (N, K), bB)
    need = esb.esb_gemm_packed_workspace_size(M, N, K, bA, ksA, bB, ksB)
    log("gemm_packed M=%d N=%d K=%d A=%s B=%s ws=%d" % (M, N, K, fa, fb, need))
    Bp = esb.esb_pack(dev(B), bB, ksB)
    acc, y = esb.esb_gemm_packed(dev(A), bA, ksA, scalar(0.37), Bp, bB, ksB, scalar(0.021),
                                 workspace(need))
    rows = np.array(sorted(set([0, 1, M // 2, M - 2, M - 1])), dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, bA, ksA, 0.37, bB, ksB, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")
    acc0, y0 = esb.esb_gemm(dev(A), bA, ksA, scalar(0.37), dev(B), bB, ksB, scalar(0.021))
    np.testing.assert_array_equal(host(acc), host(acc0))
    np.testing.assert_array_equal(host(y).view(np.uint32), host(y0).view(np.uint32))


def test_gemm_packed_reused_workspace(esb):
    """One unzeroed workspace, two calls with different split plans."""
    ws = workspace(esb.esb_gemm_packed_workspace_size(128, 4096, 9216, 3, 2, 3, 1))
    for (M, N, K, seed) in [(128, 4096, 9216, 1), (96, 2048, 4096, 2)]:
        A = wl.random_codes(seed, (M, K), 3)
        B = wl.random_codes(seed + 5, (N, K), 3)
        log("gemm_packed reuse M=%d N=%d K=%d" % (M, N, K))
        acc, _ = esb.esb_gemm_packed(dev(A), 3, 2, scalar(1.0), esb.esb_pack(dev(B), 3, 1), 3, 1,
                                     scalar(1.0), ws)
        acc0, _ = esb.esb_gemm(dev(A), 3, 2, scalar(1.0), dev(B), 3, 1, scalar(1.0))
        np.testing.assert_array_equal(host(acc), host(acc0))


def extreme_codes(b, ks, shape, seed):
    """Mostly the largest magnitude, else the smallest nonzero one, 30 % negative."""
    v = oracle.valueset(b, ks)
    top = oracle.encode(float(v[-1]), b, ks)
    small = oracle.encode(float(v[v > 0][0]), b, ks)
    r = np.random.default_rng(seed)
    c = np.where(r.random(shape) < 0.8, top, small).astype(np.uint8)
    neg = r.random(shape) < 0.3
    return np.where(neg, c | (1 << (b - 1)), c).astype(np.uint8)


def test_gemm_packed_wave_split_at_accumulator_bound(esb):
    """The wave-split kernel with ESB(4,1) both: products m_A*m_B from 1 to 144 in one
    reduction and K * 144 just below 2^24, where every per-wave partial and the total are
    still exact in fp32; ragged M; accumulators only, then outputs only."""
    M, N, K = 100, 2048, 116480
    A = extreme_codes(4, 2, (M, K), 21)
    B = extreme_codes(4, 2, (N, K), 22)
    top = oracle.encode(6.0, 4, 2)
    A[0, :] = top          # output (0, 0) = K * 144 = 16773120, the largest sum below 2^24
    B[0, :] = top
    need = esb.esb_gemm_packed_workspace_size(M, N, K, 4, 2, 4, 2)
    log("gemm_packed bound M=%d N=%d K=%d ws=%d" % (M, N, K, need))
    assert need < M * K   # A packed only: no partial sums in memory
    Bp = esb.esb_pack(dev(B), 4, 2)
    acc, _ = esb.esb_gemm_packed(dev(A), 4, 2, scalar(0.37), Bp, 4, 2, scalar(0.021),
                                 workspace(need), want_y=False)
    _, y = esb.esb_gemm_packed(dev(A), 4, 2, scalar(0.37), Bp, 4, 2, scalar(0.021),
                               workspace(need), want_acc=False)
    rows = np.array([0, 31, 32, 63, 64, M - 1], dtype=np.int64)
    st, oacc, oy = oracle.gemm(np.ascontiguousarray(A[rows]), B, 4, 2, 0.37, 4, 2, 0.021)
    assert st == 0
    np.testing.assert_array_equal(host(acc)[rows], oacc)
    assert_rel(host(y)[rows], oy, YREL, "y")
    assert oacc[0, 0] == K * 144
