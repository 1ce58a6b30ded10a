"""Helpers shared by the GPU parity tests (marshalling only)."""
import sys

import numpy as np


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


def dev(a):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def scalar(v):
    torch = torch_cuda()
    return torch.tensor([v], dtype=torch.float32, device="cuda")


def host(t):
    torch = torch_cuda()
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_rel(a, b, rel, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    fin = ~(both_nan | same_inf)
    assert np.array_equal(np.isnan(a), np.isnan(b)), what
    err = np.abs(a[fin] - b[fin]) / np.maximum(np.abs(b[fin]), 1e-300)
    assert err.size == 0 or err.max() <= rel, "%s: max rel err %g > %g" % (what, err.max(), rel)
