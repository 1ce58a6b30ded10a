"""Thin ctypes binding of libesb (include/esb.h), same entry-point names.

Argument marshalling only: every step of the hot path runs in the HIP kernels
of libesb.so.  PyTorch provides device memory and streams.  If libesb.so is
missing the import of any entry point raises; there is no fallback.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libesb.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "esb.h")

ESB_OK = 0
ESB_E_INVALID = -1
ESB_E_OVERFLOW = -3
ESB_E_UNSUPPORTED = -4
ESB_E_HIP = -5
ESB_E_WORKSPACE = -6
ESB_E_SCRATCH = -7
ESB_DDA_NOALLOC_SCRATCH = 4 << 20
ESB_B_NK = 0
ESB_B_KN = 1

_lib = None


class EsbError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = lib().esb_strerror(status).decode()
        if status == ESB_E_HIP:
            msg += " (hipError %d)" % lib().esb_last_hip_error()
        super().__init__("%s: %s (%d)" % (fn, msg, status))


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("N", "H", "W", "C", "K", "R", "S", "stride_h", "stride_w", "pad_h", "pad_w",
                 "groups")]


class DdaJob(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("len", ctypes.c_int64), ("n", ctypes.c_int),
                ("k_sig", ctypes.c_int), ("grid", ctypes.c_void_p), ("G", ctypes.c_int),
                ("alpha_out", ctypes.c_void_p), ("D_out", ctypes.c_void_p),
                ("grid_scale", ctypes.c_void_p)]


class ProjectJob(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("len", ctypes.c_int64), ("alpha", ctypes.c_void_p),
                ("n", ctypes.c_int), ("k_sig", ctypes.c_int), ("codes", ctypes.c_void_p)]


class PostDesc(ctypes.Structure):
    _fields_ = [("a", ctypes.c_void_p), ("b", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("relu", ctypes.c_int), ("alpha", ctypes.c_void_p), ("n", ctypes.c_int),
                ("k_sig", ctypes.c_int), ("codes", ctypes.c_void_p), ("absmax_out", ctypes.c_void_p)]


def lib():
    """Load libesb.so (after torch, so that both share one HIP runtime)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libesb.so not built: run paper_2109_03513_amd.build.build()")
        try:
            import torch  # noqa: F401  (loads torch's HIP runtime first)
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
        sig = {
            "esb_version": (i32, []),
            "esb_strerror": (ctypes.c_char_p, [i32]),
            "esb_last_hip_error": (i32, []),
            "esb_valueset": (i32, [i32, i32, P, i32, P]),
            "esb_project": (i32, [P, i64, P, i32, i32, P, P]),
            "esb_dequantize": (i32, [P, i64, P, i32, i32, P, P]),
            "esb_dda_workspace_size": (sz, [i64, i32, i32, i32]),
            "esb_dda_align": (i32, [P, i64, i32, i32, P, i32, P, P, P, sz, P]),
            "esb_dda_align_noalloc": (i32, [P, i64, i32, i32, P, i32, P, P, P]),
            "esb_dda_plan_size": (sz, [i32, i32, i32]),
            "esb_dda_plan": (i32, [i32, i32, P, i32, P, sz, P]),
            "esb_dda_align_planned": (i32, [P, i64, i32, i32, P, i32, P, P, P, P, sz, P]),
            "esb_quantize_planned": (i32, [P, i64, i32, i32, P, i32, P, P, P, P, P, sz, P]),
            "esb_gemm": (i32, [i32, i32, i32, P, i64, i32, i32, P, P, i64, i32, i32, P, i32, P, P,
                               i64, P]),
            "esb_conv2d": (i32, [ctypes.POINTER(ConvDesc), P, i32, i32, P, P, i32, i32, P, P, P,
                                 P]),
            "esb_gemm_workspace_size": (sz, [i32, i32, i32, i32, i32, i32, i32]),
            "esb_gemm_ws": (i32, [i32, i32, i32, P, i64, i32, i32, P, P, i64, i32, i32, P, i32, P,
                                  P, i64, P, sz, P]),
            "esb_conv2d_workspace_size": (sz, [ctypes.POINTER(ConvDesc), i32, i32, i32, i32]),
            "esb_conv2d_ws": (i32, [ctypes.POINTER(ConvDesc), P, i32, i32, P, P, i32, i32, P, P, P,
                                    P, sz, P]),
            "esb_pack_size": (sz, [i32, i32, i32, i32]),
            "esb_pack": (i32, [P, i32, i32, i64, i32, i32, P, P]),
            "esb_gemm_packed_workspace_size": (sz, [i32, i32, i32, i32, i32, i32, i32]),
            "esb_gemm_post": (i32, [i32, i32, i32, P, i64, i32, i32, P, P, i64, i32, i32, P, i32,
                                    P, P, i64, ctypes.POINTER(PostDesc), P, sz, P]),
            "esb_conv2d_post": (i32, [ctypes.POINTER(ConvDesc), P, i32, i32, P, P, i32, i32, P, P,
                                      P, ctypes.POINTER(PostDesc), P, sz, P]),
            "esb_dda_batch_workspace_size": (sz, [i32, ctypes.POINTER(DdaJob)]),
            "esb_dda_align_batch": (i32, [i32, ctypes.POINTER(DdaJob), P, sz, P]),
            "esb_project_batch": (i32, [i32, ctypes.POINTER(ProjectJob), P]),
            "esb_maxpool2d": (i32, [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P]),
            "esb_conv2d_relu_maxpool_workspace_size": (sz, [ctypes.POINTER(ConvDesc), i32, i32, i32,
                                                             i32, i32, i32, i32]),
            "esb_conv2d_relu_maxpool": (i32, [ctypes.POINTER(ConvDesc), P, i32, i32, P, P, i32, i32,
                                              P, ctypes.POINTER(PostDesc), i32, i32, i32, P, P, sz,
                                              P]),
            "esb_avgpool_global": (i32, [P, i32, i32, i32, P, P, P]),
            "esb_absmax": (i32, [P, i64, P, P]),
            "esb_dn_workspace_size": (sz, [i64]),
            "esb_dn_stats": (i32, [P, i64, P, P, sz, P]),
            "esb_project_dn": (i32, [P, i64, P, P, i32, i32, P, P]),
            "esb_dda_normal": (i32, [i32, i32, P, i32, P, P, P, P]),
            "esb_gemm_packed": (i32, [i32, i32, i32, P, i64, i32, i32, P, P, i32, i32, P, P, P, i64,
                                      P, sz, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(fn, status):
    if status != ESB_OK:
        raise EsbError(fn, status)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream if isinstance(stream, int) else stream.cuda_stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev_tensor(t, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s" % (name, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def esb_version():
    return lib().esb_version()


def esb_valueset(n, k_sig):
    """Sorted 2^n - 1 unscaled values of Q_e (host call)."""
    out = np.zeros(256, dtype=np.float32)
    cnt = ctypes.c_int(0)
    _check("esb_valueset", lib().esb_valueset(n, k_sig, out.ctypes.data_as(ctypes.c_void_p), 256,
                                              ctypes.byref(cnt)))
    return out[:cnt.value].copy()


def esb_project(x, alpha, n, k_sig, codes=None, stream=None):
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(alpha, torch.float32, "alpha")
    if codes is None:
        codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _dev_tensor(codes, torch.uint8, "codes")
    if codes.numel() != x.numel():
        raise ValueError("codes must have as many elements as x")
    _check("esb_project", lib().esb_project(_ptr(x), x.numel(), _ptr(alpha), n, k_sig, _ptr(codes),
                                            _stream(stream)))
    return codes


def esb_dequantize(codes, alpha, n, k_sig, out=None, stream=None):
    import torch
    _dev_tensor(codes, torch.uint8, "codes")
    _dev_tensor(alpha, torch.float32, "alpha")
    if out is None:
        out = torch.empty(codes.shape, dtype=torch.float32, device=codes.device)
    _dev_tensor(out, torch.float32, "out")
    _check("esb_dequantize", lib().esb_dequantize(_ptr(codes), codes.numel(), _ptr(alpha), n, k_sig,
                                                  _ptr(out), _stream(stream)))
    return out


def esb_dda_workspace_size(length, n, k_sig, G):
    return int(lib().esb_dda_workspace_size(length, n, k_sig, G))


def esb_dda_align(x, n, k_sig, grid, alpha_out=None, D_out=None, workspace=None, stream=None,
                  want_D=True):
    """Returns (alpha_out[1] fp32 tensor, D_out[G] fp64 tensor or None)."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(grid, torch.float32, "grid")
    G = grid.numel()
    dev = x.device
    if alpha_out is None:
        alpha_out = torch.empty(1, dtype=torch.float32, device=dev)
    if D_out is None and want_D:
        D_out = torch.empty(G, dtype=torch.float64, device=dev)
    need = esb_dda_workspace_size(x.numel(), n, k_sig, G)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("esb_dda_align", lib().esb_dda_align(_ptr(x), x.numel(), n, k_sig, _ptr(grid), G,
                                                _ptr(alpha_out), _ptr(D_out), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(),
                                                _stream(stream)))
    return alpha_out, D_out


def esb_dda_align_noalloc(x, n, k_sig, grid, alpha_out, D_out=None, stream=None):
    """esb_dda_align with the library's static scratch (no workspace); alpha_out (and D_out,
    if given) are preallocated device tensors, so that the call allocates nothing."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(grid, torch.float32, "grid")
    _dev_tensor(alpha_out, torch.float32, "alpha_out")
    if D_out is not None:
        _dev_tensor(D_out, torch.float64, "D_out")
    _check("esb_dda_align_noalloc", lib().esb_dda_align_noalloc(
        _ptr(x), x.numel(), n, k_sig, _ptr(grid), grid.numel(), _ptr(alpha_out), _ptr(D_out),
        _stream(stream)))
    return alpha_out, D_out


def esb_dda_plan(n, k_sig, factors, plan=None, stream=None):
    """The grid-only set-up of the DDA for candidates factors[j] (device fp32), built on the
    device; returns the plan (a uint8 device tensor)."""
    import torch
    _dev_tensor(factors, torch.float32, "factors")
    G = factors.numel()
    need = int(lib().esb_dda_plan_size(n, k_sig, G))
    if need == 0:
        raise EsbError("esb_dda_plan_size", ESB_E_INVALID)
    if plan is None:
        plan = torch.empty(need, dtype=torch.uint8, device=factors.device)
    _check("esb_dda_plan", lib().esb_dda_plan(n, k_sig, _ptr(factors), G, _ptr(plan),
                                              plan.numel(), _stream(stream)))
    return plan


def esb_dda_align_planned(x, n, k_sig, plan, G, scale, alpha_out=None, D_out=None, workspace=None,
                          stream=None, want_D=True):
    """DDA over the candidates 2^E factors[j] of a plan, E the binary exponent of |scale|
    (device scalar).  Returns (alpha_out, D_out)."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(scale, torch.float32, "scale")
    dev = x.device
    if alpha_out is None:
        alpha_out = torch.empty(1, dtype=torch.float32, device=dev)
    if D_out is None and want_D:
        D_out = torch.empty(G, dtype=torch.float64, device=dev)
    if workspace is None:
        need = esb_dda_workspace_size(x.numel(), n, k_sig, G)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("esb_dda_align_planned", lib().esb_dda_align_planned(
        _ptr(x), x.numel(), n, k_sig, _ptr(plan), G, _ptr(scale), _ptr(alpha_out), _ptr(D_out),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))
    return alpha_out, D_out


def esb_quantize_planned(x, n, k_sig, plan, G, scale, alpha_out=None, D_out=None, codes=None,
                         workspace=None, stream=None, want_D=True):
    """The planned DDA's alpha (and D), then the codes of x under it, in one call.
    Returns (alpha_out, D_out, codes)."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(scale, torch.float32, "scale")
    dev = x.device
    if alpha_out is None:
        alpha_out = torch.empty(1, dtype=torch.float32, device=dev)
    if D_out is None and want_D:
        D_out = torch.empty(G, dtype=torch.float64, device=dev)
    if codes is None:
        codes = torch.empty(x.shape, dtype=torch.uint8, device=dev)
    if workspace is None:
        need = esb_dda_workspace_size(x.numel(), n, k_sig, G)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("esb_quantize_planned", lib().esb_quantize_planned(
        _ptr(x), x.numel(), n, k_sig, _ptr(plan), G, _ptr(scale), _ptr(alpha_out), _ptr(D_out),
        _ptr(codes), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(stream)))
    return alpha_out, D_out, codes


def esb_gemm_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig):
    return int(lib().esb_gemm_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig))


def esb_conv2d_workspace_size(x_shape, w_shape, nX, kX_sig, nW, kW_sig, stride=(1, 1), pad=(0, 0),
                              groups=1):
    Nb, H, W, C = x_shape
    K, R, S, _ = w_shape
    d = ConvDesc(Nb, H, W, C, K, R, S, stride[0], stride[1], pad[0], pad[1], groups)
    return int(lib().esb_conv2d_workspace_size(ctypes.byref(d), nX, kX_sig, nW, kW_sig))


def _ws(workspace):
    """(pointer, bytes) of an optional workspace tensor."""
    if workspace is None:
        return None, 0
    return _ptr(workspace), workspace.numel() * workspace.element_size()


def esb_gemm(A, nA, kA_sig, alphaA, B, nB, kB_sig, alphaB, b_layout=ESB_B_NK, acc=None, y=None,
             want_acc=True, want_y=True, stream=None, workspace=None):
    """A: M x K codes; B: N x K (ESB_B_NK) or K x N (ESB_B_KN) codes.  Returns (acc, y).
    With a workspace tensor (esb_gemm_workspace_size bytes) the call goes to esb_gemm_ws."""
    import torch
    _dev_tensor(A, torch.uint8, "A")
    _dev_tensor(B, torch.uint8, "B")
    M, K = A.shape
    N = B.shape[0] if b_layout == ESB_B_NK else B.shape[1]
    dev = A.device
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=dev)
    if y is None and want_y:
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
    lda = A.stride(0) if M else K
    ldb = B.stride(0) if B.shape[0] else 0
    if workspace is None:
        _check("esb_gemm", lib().esb_gemm(M, N, K, _ptr(A), lda, nA, kA_sig, _ptr(alphaA), _ptr(B),
                                          ldb, nB, kB_sig, _ptr(alphaB), b_layout, _ptr(acc), _ptr(y),
                                          N, _stream(stream)))
    else:
        wp, wb = _ws(workspace)
        _check("esb_gemm_ws", lib().esb_gemm_ws(M, N, K, _ptr(A), lda, nA, kA_sig, _ptr(alphaA),
                                                _ptr(B), ldb, nB, kB_sig, _ptr(alphaB), b_layout,
                                                _ptr(acc), _ptr(y), N, wp, wb, _stream(stream)))
    return acc, y


def _addr(t):
    return None if t is None else t.data_ptr()


def post_desc(alpha, n, k_sig, codes=None, a=None, b=None, residual=None, relu=False, absmax=None):
    """esb_post of device tensors: per-channel a, b, a residual in the output layout, relu, the
    output codes (uint8, output layout) under the device scalar alpha in ESB(n, k_sig), and a
    device fp32 scalar raised to max|z|."""
    return PostDesc(_addr(a), _addr(b), _addr(residual), int(bool(relu)), _addr(alpha), n, k_sig,
                    _addr(codes), _addr(absmax))


def esb_gemm_post(A, nA, kA_sig, alphaA, B, nB, kB_sig, alphaB, out_alpha, out_n, out_k_sig,
                  a=None, b=None, residual=None, relu=False, b_layout=ESB_B_NK, codes=None,
                  want_codes=True, acc=None, want_acc=False, y=None, want_y=False, workspace=None,
                  stream=None, absmax=None):
    """Contraction with the fused post-processing; returns (acc, y, codes), M x N each."""
    import torch
    _dev_tensor(A, torch.uint8, "A")
    _dev_tensor(B, torch.uint8, "B")
    M, K = A.shape
    N = B.shape[0] if b_layout == ESB_B_NK else B.shape[1]
    dev = A.device
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=dev)
    if y is None and want_y:
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
    if codes is None and want_codes:
        codes = torch.empty((M, N), dtype=torch.uint8, device=dev)
    d = post_desc(out_alpha, out_n, out_k_sig, codes, a, b, residual, relu, absmax)
    lda = A.stride(0) if M else K
    ldb = B.stride(0) if B.shape[0] else 0
    wp, wb = _ws(workspace)
    _check("esb_gemm_post", lib().esb_gemm_post(M, N, K, _ptr(A), lda, nA, kA_sig, _ptr(alphaA),
                                                _ptr(B), ldb, nB, kB_sig, _ptr(alphaB), b_layout,
                                                _ptr(acc), _ptr(y), N, ctypes.byref(d), wp, wb,
                                                _stream(stream)))
    return acc, y, codes


def esb_conv2d_post(x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, out_alpha, out_n, out_k_sig,
                    a=None, b=None, residual=None, relu=False, stride=(1, 1), pad=(0, 0),
                    groups=1, codes=None, want_codes=True, acc=None, want_acc=False, y=None,
                    want_y=False, workspace=None, stream=None, absmax=None):
    """Convolution with the fused post-processing; returns (acc, y, codes), NHWC each."""
    import torch
    _dev_tensor(x, torch.uint8, "x")
    _dev_tensor(w, torch.uint8, "w")
    Nb, H, W, C = x.shape
    K, R, S, _ = w.shape
    P, Q = conv_out_hw(H, W, R, S, stride, pad)
    dev = x.device
    if acc is None and want_acc:
        acc = torch.empty((Nb, P, Q, K), dtype=torch.int32, device=dev)
    if y is None and want_y:
        y = torch.empty((Nb, P, Q, K), dtype=torch.float32, device=dev)
    if codes is None and want_codes:
        codes = torch.empty((Nb, P, Q, K), dtype=torch.uint8, device=dev)
    pd = post_desc(out_alpha, out_n, out_k_sig, codes, a, b, residual, relu, absmax)
    d = ConvDesc(Nb, H, W, C, K, R, S, stride[0], stride[1], pad[0], pad[1], groups)
    wp, wb = _ws(workspace)
    _check("esb_conv2d_post", lib().esb_conv2d_post(ctypes.byref(d), _ptr(x), nX, kX_sig,
                                                    _ptr(alphaX), _ptr(w), nW, kW_sig,
                                                    _ptr(alphaW), _ptr(acc), _ptr(y),
                                                    ctypes.byref(pd), wp, wb, _stream(stream)))
    return acc, y, codes


def esb_conv2d_relu_maxpool(x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, out_alpha=None,
                            out_n=5, out_k_sig=3, a=None, b=None, stride=(2, 2), pad=(3, 3),
                            pool=(3, 2, 1), y=None, want_y=True, codes=None, want_codes=False,
                            absmax=None, workspace=None, stream=None):
    """Convolution, post-processing with a ReLU and max pooling (pool = (window, stride, pad));
    returns (y, codes), each [N, PP, QQ, K] or None."""
    import torch
    _dev_tensor(x, torch.uint8, "x")
    _dev_tensor(w, torch.uint8, "w")
    Nb, H, W, C = x.shape
    K, R, S, _ = w.shape
    P, Q = conv_out_hw(H, W, R, S, stride, pad)
    PP, QQ = conv_out_hw(P, Q, pool[0], pool[0], (pool[1], pool[1]), (pool[2], pool[2]))
    dev = x.device
    if y is None and want_y:
        y = torch.empty((Nb, PP, QQ, K), dtype=torch.float32, device=dev)
    if codes is None and want_codes:
        codes = torch.empty((Nb, PP, QQ, K), dtype=torch.uint8, device=dev)
    pd = post_desc(out_alpha, out_n, out_k_sig, codes, a, b, None, True, absmax)
    d = ConvDesc(Nb, H, W, C, K, R, S, stride[0], stride[1], pad[0], pad[1], 1)
    wp, wb = _ws(workspace)
    _check("esb_conv2d_relu_maxpool", lib().esb_conv2d_relu_maxpool(
        ctypes.byref(d), _ptr(x), nX, kX_sig, _ptr(alphaX), _ptr(w), nW, kW_sig, _ptr(alphaW),
        ctypes.byref(pd), pool[0], pool[1], pool[2], _ptr(y), wp, wb, _stream(stream)))
    return y, codes


def esb_conv2d_relu_maxpool_workspace_size(x_shape, w_shape, nX, kX_sig, nW, kW_sig,
                                           stride=(2, 2), pad=(3, 3), pool=(3, 2, 1)):
    Nb, H, W, C = x_shape
    K, R, S, _ = w_shape
    d = ConvDesc(Nb, H, W, C, K, R, S, stride[0], stride[1], pad[0], pad[1], 1)
    return int(lib().esb_conv2d_relu_maxpool_workspace_size(ctypes.byref(d), nX, kX_sig, nW,
                                                             kW_sig, pool[0], pool[1], pool[2]))


def dda_jobs(specs):
    """ctypes array of esb_dda_job from (x, n, k_sig, grid, alpha_out, D_out[, grid_scale])
    tuples; with grid_scale (a device scalar) candidate j is fl32(grid_scale * grid[j])."""
    arr = (DdaJob * len(specs))()
    for i, spec in enumerate(specs):
        x, n, k_sig, grid, alpha_out, D_out = spec[:6]
        gs = spec[6] if len(spec) > 6 else None
        arr[i] = DdaJob(_addr(x), x.numel(), n, k_sig, _addr(grid), grid.numel(), _addr(alpha_out),
                        _addr(D_out), _addr(gs))
    return arr


def esb_dda_batch_workspace_size(jobs):
    return int(lib().esb_dda_batch_workspace_size(len(jobs), jobs))


def esb_dda_align_batch(jobs, workspace, stream=None):
    """DDA of every job (a dda_jobs() array) in one launch of each kernel."""
    wp, wb = _ws(workspace)
    _check("esb_dda_align_batch", lib().esb_dda_align_batch(len(jobs), jobs, wp, wb,
                                                            _stream(stream)))


def project_jobs(specs):
    """ctypes array of esb_project_job from (x, alpha, n, k_sig, codes) tuples."""
    arr = (ProjectJob * len(specs))()
    for i, (x, alpha, n, k_sig, codes) in enumerate(specs):
        arr[i] = ProjectJob(_addr(x), x.numel(), _addr(alpha), n, k_sig, _addr(codes))
    return arr


def esb_project_batch(jobs, stream=None):
    """Projection of every job (a project_jobs() array) in one launch."""
    _check("esb_project_batch", lib().esb_project_batch(len(jobs), jobs, _stream(stream)))


def esb_maxpool2d(x, window, stride, pad, out=None, stream=None):
    """NHWC fp32 max pool (padding never selected); returns out [N, P, Q, C]."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    N, H, W, C = x.shape
    P, Q = conv_out_hw(H, W, window, window, (stride, stride), (pad, pad))
    if out is None:
        out = torch.empty((N, P, Q, C), dtype=torch.float32, device=x.device)
    _dev_tensor(out, torch.float32, "out")
    _check("esb_maxpool2d", lib().esb_maxpool2d(_ptr(x), N, H, W, C, window, window, stride, pad,
                                                _ptr(out), _stream(stream)))
    return out


def esb_avgpool_global(x, out=None, absmax=None, stream=None):
    """x [N, H, W, C] (or [N, HW, C]) fp32 -> out [N, C]: fp64 sums in position order / HW."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    N, C = x.shape[0], x.shape[-1]
    HW = x.numel() // max(N * C, 1) if N * C else 1
    if out is None:
        out = torch.empty((N, C), dtype=torch.float32, device=x.device)
    _dev_tensor(out, torch.float32, "out")
    _check("esb_avgpool_global", lib().esb_avgpool_global(_ptr(x), N, HW, C, _ptr(out),
                                                          _ptr(absmax), _stream(stream)))
    return out


def esb_absmax(x, absmax, stream=None):
    """Raise the device fp32 scalar `absmax` to max |x| (the caller sets its start value)."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    _dev_tensor(absmax, torch.float32, "absmax")
    _check("esb_absmax", lib().esb_absmax(_ptr(x), x.numel(), _ptr(absmax), _stream(stream)))
    return absmax


def esb_pack_size(rows, K, n, k_sig):
    return int(lib().esb_pack_size(rows, K, n, k_sig))


def esb_pack(codes, n, k_sig, packed=None, stream=None):
    """codes: rows x K (K % 32 == 0, format inside OCP E2M1) -> rows x K/2 packed bytes."""
    import torch
    _dev_tensor(codes, torch.uint8, "codes")
    rows, K = codes.shape
    if packed is None:
        packed = torch.empty((rows, K // 2), dtype=torch.uint8, device=codes.device)
    ld = codes.stride(0) if rows else K
    _check("esb_pack", lib().esb_pack(_ptr(codes), rows, K, ld, n, k_sig, _ptr(packed),
                                      _stream(stream)))
    return packed


def esb_gemm_packed_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig):
    return int(lib().esb_gemm_packed_workspace_size(M, N, K, nA, kA_sig, nB, kB_sig))


def esb_gemm_packed(A, nA, kA_sig, alphaA, B_packed, nB, kB_sig, alphaB, workspace, acc=None,
                    y=None, want_acc=True, want_y=True, stream=None):
    """A: M x K codes; B_packed: N x K/2 bytes from esb_pack.  Returns (acc, y)."""
    import torch
    _dev_tensor(A, torch.uint8, "A")
    _dev_tensor(B_packed, torch.uint8, "B_packed")
    M, K = A.shape
    N = B_packed.shape[0]
    dev = A.device
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=dev)
    if y is None and want_y:
        y = torch.empty((M, N), dtype=torch.float32, device=dev)
    lda = A.stride(0) if M else K
    wp, wb = _ws(workspace)
    _check("esb_gemm_packed", lib().esb_gemm_packed(M, N, K, _ptr(A), lda, nA, kA_sig, _ptr(alphaA),
                                                    _ptr(B_packed), nB, kB_sig, _ptr(alphaB),
                                                    _ptr(acc), _ptr(y), N, wp, wb, _stream(stream)))
    return acc, y


def esb_dn_stats(x, stats=None, workspace=None, stream=None):
    """Device fp32 [mean, std] of x (population standard deviation)."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    n = x.numel()
    if stats is None:
        stats = torch.empty(2, dtype=torch.float32, device=x.device)
    if workspace is None:
        workspace = torch.empty(int(lib().esb_dn_workspace_size(n)), dtype=torch.uint8,
                                device=x.device)
    wp, wb = _ws(workspace)
    _check("esb_dn_stats", lib().esb_dn_stats(_ptr(x), n, _ptr(stats), wp, wb, _stream(stream)))
    return stats


def esb_project_dn(x, stats, alpha, n, k_sig, codes=None, stream=None):
    """Codes of fl32(fl32(x - mean) / fl32(std + 1e-7)) under alpha; stats = [mean, std]."""
    import torch
    _dev_tensor(x, torch.float32, "x")
    if codes is None:
        codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _check("esb_project_dn", lib().esb_project_dn(_ptr(x), x.numel(), _ptr(stats), _ptr(alpha), n,
                                                  k_sig, _ptr(codes), _stream(stream)))
    return codes


def esb_dda_normal(n, k_sig, grid, alpha_out=None, D_out=None, dD_out=None, stream=None):
    """Analytic one-sided D_j for N(0,1) over the candidates grid (device fp32); dD_out
    (optional device fp64 tensor of grid's size) receives dD/dalpha."""
    import torch
    G = grid.numel()
    if alpha_out is None:
        alpha_out = torch.empty(1, dtype=torch.float32, device=grid.device)
    if D_out is None:
        D_out = torch.empty(G, dtype=torch.float64, device=grid.device)
    _check("esb_dda_normal", lib().esb_dda_normal(n, k_sig, _ptr(grid), G, _ptr(alpha_out),
                                                  _ptr(D_out), _ptr(dD_out), _stream(stream)))
    return alpha_out, D_out


def conv_out_hw(H, W, R, S, stride, pad):
    return (H + 2 * pad[0] - R) // stride[0] + 1, (W + 2 * pad[1] - S) // stride[1] + 1


def esb_conv2d(x, nX, kX_sig, alphaX, w, nW, kW_sig, alphaW, stride=(1, 1), pad=(0, 0), groups=1,
               acc=None, y=None, want_acc=True, want_y=True, stream=None, workspace=None):
    """x: [N, H, W, C] codes (NHWC); w: [K, R, S, C/groups] codes (KRSC).  Returns (acc, y) NHWC.
    With a workspace tensor (esb_conv2d_workspace_size bytes) the call goes to esb_conv2d_ws."""
    import torch
    _dev_tensor(x, torch.uint8, "x")
    _dev_tensor(w, torch.uint8, "w")
    Nb, H, W, C = x.shape
    K, R, S, _ = w.shape
    P, Q = conv_out_hw(H, W, R, S, stride, pad)
    dev = x.device
    if acc is None and want_acc:
        acc = torch.empty((Nb, P, Q, K), dtype=torch.int32, device=dev)
    if y is None and want_y:
        y = torch.empty((Nb, P, Q, K), dtype=torch.float32, device=dev)
    d = ConvDesc(Nb, H, W, C, K, R, S, stride[0], stride[1], pad[0], pad[1], groups)
    if workspace is None:
        _check("esb_conv2d", lib().esb_conv2d(ctypes.byref(d), _ptr(x), nX, kX_sig, _ptr(alphaX),
                                              _ptr(w), nW, kW_sig, _ptr(alphaW), _ptr(acc), _ptr(y),
                                              _stream(stream)))
    else:
        wp, wb = _ws(workspace)
        _check("esb_conv2d_ws", lib().esb_conv2d_ws(ctypes.byref(d), _ptr(x), nX, kX_sig,
                                                    _ptr(alphaX), _ptr(w), nW, kW_sig, _ptr(alphaW),
                                                    _ptr(acc), _ptr(y), wp, wb, _stream(stream)))
    return acc, y
