"""CPU oracle for the ESB hot path (Gong et al., IEEE TPDS 2021).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the GPU product path (``paper_2109_03513_amd``); it is a ctypes
wrapper around ``esb_oracle.c``, a plain C implementation written from the
paper (value set eq. (4)-(5), projection eq. (6)-(8), DDA eq. (9)/(13), float
format eq. (14), multiplication eq. (15), convolution stage of Sec. 4.2).

Readings of the paper that the oracle fixes (and that the GPU path must match):
``k_sig`` = significant bits = paper k + 1; v = fl32(x/alpha) by IEEE division;
ties go to the larger magnitude; NaN or an invalid alpha gives +0; zero is
encoded with sign bit 0; code bits above b-1 are ignored.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "esb_oracle.c")
_LIB = os.path.join(_HERE, "libesb_oracle.so")
_lib = None

ESO_OK = 0
ESO_E_INVALID = -1
ESO_E_OVERFLOW = -3
ESO_E_UNSUPPORTED = -4


def build():
    """Compile the oracle with gcc (scalar C, no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=gnu11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
           "-fPIC", "-shared", _SRC, "-o", _LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f32, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_double
        sig = {
            "eso_num_threads": (i32, []),
            "eso_N": (i32, [i32, i32]),
            "eso_C": (f64, [i32, i32]),
            "eso_valueset": (i32, [i32, i32, P, i32]),
            "eso_decode": (f64, [i32, i32, i32]),
            "eso_encode": (i32, [f64, i32, i32]),
            "eso_project_value": (f64, [f32, f32, i32, i32]),
            "eso_project_bruteforce": (f64, [f32, f32, i32, i32]),
            "eso_project": (i32, [P, i64, f32, i32, i32, P]),
            "eso_project_bf": (i32, [P, i64, f32, i32, i32, P]),
            "eso_dequantize": (i32, [P, i64, f32, i32, i32, P]),
            "eso_dda": (i32, [P, i64, i32, i32, P, i32, P]),
            "eso_dda_normal": (f64, [f64, i32, i32]),
            "eso_dda_normal_deriv": (f64, [f64, i32, i32]),
            "eso_post": (i32, [P, i64, i64, i64, P, P, P, i32, f32, i32, i32, P, P]),
            "eso_dn_stats": (i32, [P, i64, P, P]),
            "eso_project_dn": (i32, [P, i64, f32, f32, f32, i32, i32, P]),
            "eso_gemm": (i32, [i32, i32, i32, P, i64, i32, i32, f32, P, i64, i32, i32, f32, i32,
                               P, P, i64]),
            "eso_conv2d": (i32, [i32] * 12 + [P, i32, i32, f32, P, i32, i32, f32, P, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _u8(a):
    return np.ascontiguousarray(a, dtype=np.uint8)


def num_threads():
    return lib().eso_num_threads()


def N(b, k_sig):
    return lib().eso_N(b, k_sig)


def C(b, k_sig):
    return lib().eso_C(b, k_sig)


def valueset(b, k_sig):
    """Non-negative unscaled values of Q_e, ascending (eq. (4)-(5))."""
    out = np.zeros(256, dtype=np.float64)
    n = lib().eso_valueset(b, k_sig, _p(out), 256)
    if n < 0:
        raise ValueError("invalid (b, k_sig)")
    return out[:n].copy()


def full_valueset(b, k_sig):
    v = valueset(b, k_sig)
    return np.concatenate([-v[:0:-1], v])


def decode(code, b, k_sig):
    return lib().eso_decode(int(code), b, k_sig)


def encode(q, b, k_sig):
    return lib().eso_encode(float(q), b, k_sig)


def project_value(x, alpha, b, k_sig):
    return lib().eso_project_value(float(x), float(alpha), b, k_sig)


def project_bruteforce_value(x, alpha, b, k_sig):
    return lib().eso_project_bruteforce(float(x), float(alpha), b, k_sig)


def project(x, alpha, b, k_sig):
    x = _f32(x)
    out = np.empty(x.shape, dtype=np.uint8)
    st = lib().eso_project(_p(x), x.size, np.float32(alpha), b, k_sig, _p(out))
    if st:
        raise ValueError("eso_project: %d" % st)
    return out


def project_bruteforce(x, alpha, b, k_sig):
    x = _f32(x)
    out = np.empty(x.shape, dtype=np.uint8)
    st = lib().eso_project_bf(_p(x), x.size, np.float32(alpha), b, k_sig, _p(out))
    if st:
        raise ValueError("eso_project_bf: %d" % st)
    return out


def dequantize(codes, alpha, b, k_sig):
    codes = _u8(codes)
    out = np.empty(codes.shape, dtype=np.float32)
    st = lib().eso_dequantize(_p(codes), codes.size, np.float32(alpha), b, k_sig, _p(out))
    if st:
        raise ValueError("eso_dequantize: %d" % st)
    return out


def dda(x, b, k_sig, grid):
    """Empirical DDA: returns (j_star, D[G]) (eq. (9), (13))."""
    x = _f32(x)
    grid = _f32(grid)
    D = np.zeros(grid.size, dtype=np.float64)
    j = lib().eso_dda(_p(x), x.size, b, k_sig, _p(grid), grid.size, _p(D))
    if j < 0:
        raise ValueError("eso_dda: %d" % j)
    return j, D


def dda_normal(alpha, b, k_sig):
    """Analytic one-sided D(alpha, b, k) for p = N(0, 1) (eq. (9))."""
    return lib().eso_dda_normal(float(alpha), b, k_sig)


def dda_normal_deriv(alpha, b, k_sig):
    """dD/dalpha of dda_normal (Sec. 3.4, "Resolving extremum")."""
    return lib().eso_dda_normal_deriv(float(alpha), b, k_sig)


def dn_stats(x):
    """(mean, population std) of x in long double (the DN equation), as floats."""
    x = _f32(x)
    m = ctypes.c_double()
    sd = ctypes.c_double()
    st = lib().eso_dn_stats(_p(x), x.size, ctypes.byref(m), ctypes.byref(sd))
    assert st == 0
    return m.value, sd.value


def project_dn(x, mean, std, alpha, b, k_sig):
    """Codes of fl32(fl32(x - mean) / fl32(std + 1e-7)) under alpha (binary32 mean, std)."""
    x = _f32(x)
    out = np.empty(x.shape, dtype=np.uint8)
    st = lib().eso_project_dn(_p(x), x.size, float(np.float32(mean)), float(np.float32(std)),
                              float(np.float32(alpha)), b, k_sig, _p(out))
    assert st == 0
    return out


def post(y, b, k_sig, alpha, a=None, bias=None, res=None, relu=False):
    """Fused post-processing of a 2-D output y (channels = columns): returns (z, codes)."""
    y = _f32(y)
    assert y.ndim == 2
    rows, cols = y.shape
    av = None if a is None else _f32(a)
    bv = None if bias is None else _f32(bias)
    rv = None if res is None else _f32(res)
    z = np.empty_like(y)
    codes = np.empty(y.shape, dtype=np.uint8)
    st = lib().eso_post(_p(y), rows, cols, cols, None if av is None else _p(av),
                        None if bv is None else _p(bv), None if rv is None else _p(rv),
                        int(bool(relu)), float(np.float32(alpha)), b, k_sig, _p(z), _p(codes))
    if st:
        raise ValueError("eso_post: %d" % st)
    return z, codes


def gemm(A, B, bA, ksA, alphaA, bB, ksB, alphaB, b_layout=0, want_acc=True, want_y=True):
    """A: M x K codes; B: N x K (layout 0) or K x N (layout 1).  Returns (status, acc, y)."""
    A = _u8(A)
    B = _u8(B)
    M, K = A.shape
    Nn = B.shape[0] if b_layout == 0 else B.shape[1]
    acc = np.zeros((M, Nn), dtype=np.int32) if want_acc else None
    y = np.zeros((M, Nn), dtype=np.float32) if want_y else None
    st = lib().eso_gemm(M, Nn, K, _p(A), A.shape[1], bA, ksA, np.float32(alphaA),
                        _p(B), B.shape[1], bB, ksB, np.float32(alphaB), b_layout,
                        _p(acc), _p(y), Nn)
    return st, acc, y


def conv2d(x, w, bX, ksX, alphaX, bW, ksW, alphaW, stride=(1, 1), pad=(0, 0), groups=1,
           want_acc=True, want_y=True):
    """x: [N, H, W, C] codes; w: [K, R, S, C/groups] codes.  Returns (status, acc, y), NHWC."""
    x = _u8(x)
    w = _u8(w)
    Nb, H, W, C = x.shape
    Kout, R, S, Cg = w.shape
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    acc = np.zeros((Nb, P, Q, Kout), dtype=np.int32) if want_acc else None
    y = np.zeros((Nb, P, Q, Kout), dtype=np.float32) if want_y else None
    st = lib().eso_conv2d(Nb, H, W, C, Kout, R, S, stride[0], stride[1], pad[0], pad[1], groups,
                          _p(x), bX, ksX, np.float32(alphaX), _p(w), bW, ksW, np.float32(alphaW),
                          _p(acc), _p(y))
    return st, acc, y
