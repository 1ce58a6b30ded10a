"""The C ABI loads and exports every symbol include/esb.h declares; host-only
calls and argument validation work without a GPU (no device work is enqueued
by any call in this file)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from conftest import ALL_BK, ROOT

LIB = os.path.join(ROOT, "paper_2109_03513_amd", "libesb.so")
HEADER = os.path.join(ROOT, "include", "esb.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LIB):
        from paper_2109_03513_amd import build
        build.build()
    from paper_2109_03513_amd import esb
    return esb.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(esb_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 10, names
    for n in names:
        assert hasattr(L, n), n


def test_version_and_strerror(L):
    assert L.esb_version() >= 100
    for s in (0, -1, -3, -4, -5, -6, 12345):
        assert isinstance(L.esb_strerror(s), bytes)


@pytest.mark.parametrize("b,ks", ALL_BK)
def test_valueset_matches_oracle(b, ks):
    from paper_2109_03513_amd import esb
    np.testing.assert_array_equal(esb.esb_valueset(b, ks), oracle.full_valueset(b, ks).astype(np.float32))


def test_valueset_errors(L):
    out = np.zeros(4, np.float32)
    cnt = ctypes.c_int()
    p = out.ctypes.data_as(ctypes.c_void_p)
    assert L.esb_valueset(4, 2, p, 4, ctypes.byref(cnt)) == -1          # cap too small
    assert L.esb_valueset(9, 2, p, 1000, ctypes.byref(cnt)) == -1
    assert L.esb_valueset(4, 4, p, 1000, ctypes.byref(cnt)) == -1
    assert L.esb_valueset(4, 2, None, 1000, ctypes.byref(cnt)) == -1


def test_argument_validation_without_launch(L):
    fake = ctypes.c_void_p(0x1000)     # never dereferenced: every call below fails validation
    assert L.esb_project(fake, -1, fake, 4, 2, fake, None) == -1
    assert L.esb_project(fake, 10, fake, 4, 0, fake, None) == -1
    assert L.esb_project(None, 10, fake, 4, 2, fake, None) == -1
    assert L.esb_project(fake, 10, None, 4, 2, fake, None) == -1
    assert L.esb_dequantize(fake, 10, fake, 1, 1, fake, None) == -1
    # DDA: grid too large, workspace missing / too small
    assert L.esb_dda_align(fake, 100, 8, 7, fake, 65, fake, None, fake, 1 << 30, None) == -1
    assert L.esb_dda_align(fake, 100, 4, 2, fake, 64, fake, None, None, 0, None) == -6
    need = L.esb_dda_workspace_size(100, 4, 2, 64)
    assert need > 0
    assert L.esb_dda_align(fake, 100, 4, 2, fake, 64, fake, None, fake, need - 1, None) == -6
    assert L.esb_dda_workspace_size(100, 4, 2, 0) == 0
    assert L.esb_dda_workspace_size(100, 8, 7, 65) == 0
    # glue: windows made only of padding, bad sizes, missing pointers
    mp = L.esb_maxpool2d
    assert mp(fake, 1, 8, 8, 4, 3, 3, 2, 3, fake, None) == -1          # pad >= window
    assert mp(fake, 1, 8, 8, 4, 3, 3, 0, 1, fake, None) == -1          # stride 0
    assert mp(fake, 1, 2, 2, 4, 5, 5, 1, 1, fake, None) == -1          # window beyond padded input
    assert mp(None, 1, 8, 8, 4, 3, 3, 2, 1, fake, None) == -1
    assert mp(None, 0, 8, 8, 4, 3, 3, 2, 1, None, None) == 0           # empty batch: nothing to do
    assert L.esb_avgpool_global(fake, 2, 0, 4, fake, None, None) == -1
    assert L.esb_avgpool_global(None, 2, 49, 4, fake, None, None) == -1
    assert L.esb_absmax(fake, 10, None, None) == -1
    assert L.esb_absmax(None, 10, fake, None) == -1
    assert L.esb_absmax(None, 0, fake, None) == 0
    # DDA plans: sizes, too small or unaligned plan buffers, missing arguments
    assert L.esb_dda_plan_size(5, 3, 64) > 64 * 15 * 4
    assert L.esb_dda_plan_size(5, 3, 0) == 0 and L.esb_dda_plan_size(9, 3, 64) == 0
    assert L.esb_dda_plan_size(8, 7, 65) == 0                            # 65 * 127 > 8192
    psz = L.esb_dda_plan_size(5, 3, 64)
    assert L.esb_dda_plan(5, 3, fake, 64, fake, psz - 1, None) == -6
    assert L.esb_dda_plan(5, 3, fake, 64, ctypes.c_void_p(0x1008), psz, None) == -6
    assert L.esb_dda_plan(5, 3, None, 64, fake, psz, None) == -1
    pl = L.esb_dda_align_planned
    wsz = L.esb_dda_workspace_size(100, 5, 3, 64)
    assert pl(fake, 100, 5, 3, fake, 64, fake, fake, None, fake, wsz - 1, None) == -6
    assert pl(fake, 100, 5, 3, None, 64, fake, fake, None, fake, wsz, None) == -1
    assert pl(fake, 100, 5, 3, fake, 64, None, fake, None, fake, wsz, None) == -1
    assert pl(fake, 100, 5, 3, ctypes.c_void_p(0x1004), 64, fake, fake, None, fake, wsz, None) == -1
    # DDA with the static scratch: the same checks, and inputs beyond the scratch refused
    na = L.esb_dda_align_noalloc
    assert na(fake, 100, 8, 7, fake, 65, fake, None, None) == -1
    assert na(fake, 100, 4, 2, None, 64, fake, None, None) == -1
    assert na(None, 100, 4, 2, fake, 64, fake, None, None) == -1
    big = 1 << 33
    assert L.esb_dda_workspace_size(big, 4, 2, 64) > (4 << 20)
    assert na(fake, big, 4, 2, fake, 64, fake, None, None) == -7
    assert L.esb_strerror(-7) != L.esb_strerror(-99)
    # GEMM contract: unsupported magnitudes, overflow, bad pitches, no output
    g = L.esb_gemm
    assert g(4, 4, 8, fake, 8, 6, 2, fake, fake, 8, 6, 2, fake, 0, fake, None, 4, None) == -4
    assert g(4, 4, 600, fake, 600, 8, 5, fake, fake, 600, 8, 5, fake, 0, fake, None, 4, None) == -3
    assert g(4, 4, 8, fake, 7, 4, 2, fake, fake, 8, 4, 2, fake, 0, fake, None, 4, None) == -1
    assert g(4, 4, 8, fake, 8, 4, 2, fake, fake, 8, 4, 2, fake, 0, None, None, 4, None) == -1
    assert g(4, 4, 8, fake, 8, 4, 2, fake, fake, 8, 4, 2, fake, 2, fake, None, 4, None) == -1
    assert g(4, 4, 8, fake, 8, 4, 2, None, fake, 8, 4, 2, fake, 0, None, fake, 4, None) == -1
    from paper_2109_03513_amd.esb import ConvDesc
    d = ConvDesc(1, 8, 8, 6, 4, 3, 3, 1, 1, 1, 1, 4)       # groups does not divide C
    assert L.esb_conv2d(ctypes.byref(d), fake, 4, 2, fake, fake, 4, 2, fake, fake, None, None) == -1
    d = ConvDesc(1, 2, 2, 4, 4, 5, 5, 1, 1, 0, 0, 1)       # window larger than padded input
    assert L.esb_conv2d(ctypes.byref(d), fake, 4, 2, fake, fake, 4, 2, fake, fake, None, None) == -1
    d = ConvDesc(1, 8, 8, 600, 4, 1, 1, 1, 1, 0, 0, 1)
    assert L.esb_conv2d(ctypes.byref(d), fake, 8, 5, fake, fake, 8, 5, fake, fake, None, None) == -3


def test_contract_matches_oracle():
    """Status codes of the contraction contract agree with the oracle's."""
    from paper_2109_03513_amd import esb
    fake = ctypes.c_void_p(0x1000)
    for (bA, ksA), (bB, ksB), K in [((6, 2), (4, 2), 8), ((8, 5), (8, 5), 545), ((8, 5), (8, 5), 546),
                                    ((5, 1), (3, 1), 4)]:
        A = np.zeros((1, K), np.uint8)
        ost = oracle.gemm(A, A, bA, ksA, 1.0, bB, ksB, 1.0)[0]
        gst = esb.lib().esb_gemm(0, 0, K, fake, K, bA, ksA, fake, fake, K, bB, ksB, fake, 0, fake,
                                 None, 0, None)
        assert gst == ost, (bA, ksA, bB, ksB, K, gst, ost)


def test_contraction_workspace_sizes_and_errors(L):
    """Workspace sizes of the decode-once path: nonzero exactly for pairs of formats the E4M3
    or the E2M1 path takes, at least both operands' decoded bytes; a too small workspace is
    refused before any launch (ESB_E_WORKSPACE)."""
    from paper_2109_03513_amd import esb
    fake = ctypes.c_void_p(0x1000)
    M, N, K = 300, 200, 576
    need = L.esb_gemm_workspace_size(M, N, K, 5, 3, 5, 3)
    assert need >= M * K + N * K
    assert L.esb_gemm_workspace_size(M, N, K, 3, 2, 3, 1) >= M * K // 2 + N * K // 2   # E2M1 path
    assert L.esb_gemm_workspace_size(M, N, 48, 3, 2, 3, 1) == 0      # K % 32: int8 table path only
    assert L.esb_gemm_workspace_size(M, N, K, 8, 5, 8, 5) == 0       # outside the E4M3 window
    assert L.esb_gemm_workspace_size(M, N, K, 9, 2, 5, 3) == 0       # invalid format
    g = L.esb_gemm_ws
    assert g(M, N, K, fake, K, 5, 3, fake, fake, K, 5, 3, fake, 0, fake, None, N, fake, need - 1,
             None) == -6
    assert g(M, N, K, fake, K - 1, 5, 3, fake, fake, K, 5, 3, fake, 0, fake, None, N, fake, need,
             None) == -1
    d = esb.ConvDesc(64, 14, 14, 256, 256, 3, 3, 1, 1, 1, 1, 1)
    cneed = L.esb_conv2d_workspace_size(ctypes.byref(d), 5, 3, 5, 3)
    assert cneed >= 64 * 14 * 14 * 256 + 256 * 9 * 256
    assert L.esb_conv2d_ws(ctypes.byref(d), fake, 5, 3, fake, fake, 5, 3, fake, fake, None, fake,
                           cneed - 1, None) == -6
    dw = esb.ConvDesc(32, 56, 56, 144, 144, 3, 3, 1, 1, 1, 1, 144)  # depthwise: no workspace
    assert L.esb_conv2d_workspace_size(ctypes.byref(dw), 5, 3, 5, 3) == 0
    assert esb.esb_conv2d_workspace_size((64, 14, 14, 256), (256, 3, 3, 256), 5, 3, 5, 3,
                                         pad=(1, 1)) == cneed


def test_packed_sizes_and_errors(L):
    """Packed 4-bit storage: sizes for formats inside OCP E2M1 only, refusals before any
    launch (formats outside E2M1, K % 32, too small workspace, bad pitch)."""
    fake = ctypes.c_void_p(0x1000)
    assert L.esb_pack_size(10, 64, 4, 2) == 10 * 32          # ESB(4,1) = E2M1
    assert L.esb_pack_size(7, 9216, 3, 1) == 7 * 4608         # ESB(3,0)
    assert L.esb_pack_size(10, 48, 4, 2) == 0                 # K % 32 != 0
    assert L.esb_pack_size(10, 64, 5, 3) == 0                 # ESB(5,2): two fraction bits
    assert L.esb_pack_size(10, 64, 4, 3) == 0                 # ESB(4,2)
    assert L.esb_pack(fake, 10, 64, 64, 5, 3, fake, None) == -4     # ESB_E_UNSUPPORTED
    assert L.esb_pack(fake, 10, 64, 63, 4, 2, fake, None) == -1     # ld < K
    assert L.esb_pack(fake, 10, 48, 48, 4, 2, fake, None) == -4     # K % 32
    M, N, K = 128, 4096, 9216
    need = L.esb_gemm_packed_workspace_size(M, N, K, 3, 2, 3, 1)
    assert need >= M * K // 2
    assert L.esb_gemm_packed_workspace_size(M, N, K, 5, 3, 3, 1) == 0
    gp = L.esb_gemm_packed
    assert gp(M, N, K, fake, K, 3, 2, fake, fake, 3, 1, fake, fake, None, N, fake, need - 1,
              None) == -6
    assert gp(M, N, K, fake, K, 3, 2, fake, fake, 3, 1, fake, fake, None, N, None, need,
              None) == -6
    assert gp(M, N, K, fake, K, 5, 3, fake, fake, 3, 1, fake, fake, None, N, fake, need,
              None) == -4
    assert gp(M, N, K, fake, K - 1, 3, 2, fake, fake, 3, 1, fake, fake, None, N, fake, need,
              None) == -1


def test_dn_and_dda_normal_refusals(L):
    """Normalization and the analytic aligner refuse bad arguments before any launch."""
    fake = ctypes.c_void_p(0x1000)
    need = L.esb_dn_workspace_size(1 << 20)
    assert need >= 8
    assert L.esb_dn_workspace_size(-1) == 0
    assert L.esb_dn_stats(fake, -1, fake, fake, need, None) == -1
    assert L.esb_dn_stats(fake, 10, None, fake, need, None) == -1
    assert L.esb_dn_stats(None, 10, fake, fake, need, None) == -1
    assert L.esb_dn_stats(fake, 1 << 20, fake, fake, need - 1, None) == -6
    assert L.esb_dn_stats(fake, 1 << 20, fake, None, need, None) == -6
    assert L.esb_project_dn(fake, 10, fake, fake, 9, 2, fake, None) == -1   # n > 8
    assert L.esb_project_dn(fake, 10, None, fake, 4, 2, fake, None) == -1
    assert L.esb_project_dn(fake, -1, fake, fake, 4, 2, fake, None) == -1
    assert L.esb_dda_normal(4, 2, fake, 0, fake, None, None, None) == -1
    assert L.esb_dda_normal(4, 4, fake, 10, fake, None, None, None) == -1          # k_sig >= n
    assert L.esb_dda_normal(4, 2, None, 10, fake, None, None, None) == -1
    assert L.esb_dda_normal(4, 2, fake, 10, None, fake, None, None) == -1
    assert L.esb_dda_normal(4, 2, fake, 10, fake, None, fake, None) == -1   # D_out required


def test_post_refusals(L):
    """The fused post-processing refuses bad arguments before any launch."""
    from paper_2109_03513_amd.esb import PostDesc
    fake = ctypes.c_void_p(0x1000)
    M = N = K = 64
    gp = L.esb_gemm_post

    def call(post, acc=fake, y=fake, alphaA=fake):
        return gp(M, N, K, fake, K, 4, 2, alphaA, fake, K, 4, 2, fake, 0, acc, y, N,
                  None if post is None else ctypes.byref(post), None, 0, None)

    assert call(PostDesc(None, None, None, 0, 0x1000, 4, 2, 0x1000, None), alphaA=None) == -1
    assert call(PostDesc(None, None, None, 0, None, 4, 2, 0x1000, None)) == -1      # codes, no alpha
    assert call(PostDesc(None, None, None, 0, 0x1000, 4, 4, 0x1000, None)) == -1    # bad format
    assert call(PostDesc(None, None, None, 0, 0x1000, 9, 2, 0x1000, None)) == -1
    assert call(PostDesc(None, None, None, 1, None, 0, 0, None, None), acc=None, y=None) == -1
    assert call(None, acc=None, y=None) == -1


def test_batch_refusals(L):
    """Batched DDA and projection validate every job before any launch."""
    from paper_2109_03513_amd.esb import DdaJob, ProjectJob
    jobs = (DdaJob * 2)(DdaJob(0x1000, 100, 4, 2, 0x1000, 64, 0x1000, None, None),
                        DdaJob(0x1000, 5000, 5, 3, 0x1000, 17, 0x1000, 0x1000, 0x1000))
    need = L.esb_dda_batch_workspace_size(2, jobs)
    single = L.esb_dda_workspace_size(100, 4, 2, 64) + L.esb_dda_workspace_size(5000, 5, 3, 17)
    assert need >= single > 0
    assert L.esb_dda_align_batch(2, jobs, ctypes.c_void_p(0x1000), need - 1, None) == -6
    assert L.esb_dda_align_batch(2, jobs, None, need, None) == -6
    bad = (DdaJob * 2)(jobs[0], DdaJob(0x1000, 5000, 5, 5, 0x1000, 17, 0x1000, None, None))
    assert L.esb_dda_batch_workspace_size(2, bad) == 0
    assert L.esb_dda_align_batch(2, bad, ctypes.c_void_p(0x1000), need, None) == -1
    assert L.esb_dda_align_batch(0, None, None, 0, None) == 0
    assert L.esb_dda_align_batch(-1, jobs, None, 0, None) == -1
    pj = (ProjectJob * 2)(ProjectJob(0x1000, 10, 0x1000, 4, 2, 0x1000),
                          ProjectJob(0x1000, 10, None, 4, 2, 0x1000))
    assert L.esb_project_batch(2, pj, None) == -1
    assert L.esb_project_batch(0, None, None) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without libesb.so the binding raises instead of computing anything elsewhere."""
    from paper_2109_03513_amd import esb
    monkeypatch.setattr(esb, "_lib", None)
    monkeypatch.setattr(esb, "LIB_PATH", str(tmp_path / "libesb.so"))
    with pytest.raises(RuntimeError, match="not built"):
        esb.lib()
