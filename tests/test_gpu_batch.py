"""Batched DDA and projection (esb_dda_align_batch, esb_project_batch): every job's
result equals its single call bit for bit (alpha, D, codes) and the oracle (alpha exact
where the argmin is decided, D within 1e-9 relative as in the single-call tests, codes
bit-exact), for mixed formats, grids and lengths (empty, ragged, unaligned, many blocks
with group sums), and for more jobs than one launch takes."""
import numpy as np
import pytest

import oracle
from gpuutil import assert_rel, dev, host, log, torch_cuda
from paper_2109_03513_amd import workloads as wl

pytestmark = pytest.mark.gpu
REL = 1e-9


@pytest.fixture(scope="module")
def esb():
    from paper_2109_03513_amd import esb as e
    e.lib()
    return e


def job_specs(seed, count):
    r = np.random.default_rng(seed)
    fmts = [(4, 2), (3, 1), (5, 3), (8, 5), (2, 1), (6, 3), (7, 4), (4, 3)]
    lens = [0, 1, 3, 4097, 36864, 200704, (1 << 21) + 5, 77777, 16384, 9]
    out = []
    for i in range(count):
        b, ks = fmts[i % len(fmts)]
        n = lens[i % len(lens)]
        x = (r.standard_normal(n) * r.uniform(0.01, 3.0)).astype(np.float32)
        if i % 3 == 1:
            x = np.maximum(x, 0)
        G = [64, 17, 1, 100, 64, 33][i % 6]
        G = min(G, 8192 // ((1 << (b - 1)) - 1))   # at most 8192 thresholds per job
        s = float(np.std(x)) if n > 1 else 1.0
        grid = (s * np.linspace(0.02, 3.0, G)).astype(np.float32)
        if G > 3:
            r.shuffle(grid)              # the grid need not be sorted
        out.append((b, ks, x, grid))
    return out


def run_batch(esb, specs, offset=False):
    torch = torch_cuda()
    keep, rows = [], []
    for (b, ks, x, grid) in specs:
        xd = dev(np.concatenate([[np.float32(0)], x])) [1:] if offset else dev(x)
        gd = dev(grid)
        a = torch.empty(1, dtype=torch.float32, device="cuda")
        D = torch.empty(grid.size, dtype=torch.float64, device="cuda")
        keep.append((xd, gd, a, D))
        rows.append((xd, b, ks, gd, a, D))
    jobs = esb.dda_jobs(rows)
    ws = torch.full((max(esb.esb_dda_batch_workspace_size(jobs), 1),), 0x5A, dtype=torch.uint8,
                    device="cuda")
    esb.esb_dda_align_batch(jobs, ws)
    return [(host(a)[0], host(D)) for (_, _, a, D) in keep]


@pytest.mark.parametrize("count,offset", [(2, False), (6, True), (11, False)])
def test_dda_batch(esb, count, offset):
    specs = job_specs(count, count)
    log("dda batch count=%d offset=%s lens=%s" % (count, offset, [s[2].size for s in specs]))
    got = run_batch(esb, specs, offset)
    for (b, ks, x, grid), (a, D) in zip(specs, got):
        a1, D1 = esb.esb_dda_align(dev(x), b, ks, dev(grid))
        np.testing.assert_array_equal(D.view(np.uint64), host(D1).view(np.uint64))
        assert a == host(a1)[0]
        j, Do = oracle.dda(x, b, ks, grid)
        assert_rel(D, Do, REL, "D b=%d k_sig=%d len=%d" % (b, ks, x.size))
        Ds = np.sort(Do[~np.isnan(Do)])
        if Ds.size > 1 and np.isfinite(Ds[0]) and Ds[0] > 0 and (Ds[1] - Ds[0]) / Ds[0] > 1e-7:
            assert a == grid[j]


def test_dda_batch_conv_step_tensors(esb):
    """The weights and the input of the ResNet18 3x3 layer in one batch."""
    c = wl.resnet_conv3x3(0)
    specs = [(c["nW"], c["ksW"], c["w"].ravel(), c["gridW"]),
             (c["nX"], c["ksX"], c["x"].ravel(), c["gridX"])]
    got = run_batch(esb, specs)
    for (b, ks, x, grid), (a, D) in zip(specs, got):
        j, Do = oracle.dda(x, b, ks, grid)
        assert_rel(D, Do, REL, "conv step")
        assert a == grid[j]


@pytest.mark.parametrize("count", [3, 10])
def test_project_batch(esb, count):
    torch = torch_cuda()
    r = np.random.default_rng(count)
    fmts = [(4, 2), (3, 1), (5, 3), (8, 6), (2, 1)]
    lens = [0, 5, 4096, 200704, 1001, 36864 + 3]
    rows, keep = [], []
    for i in range(count):
        b, ks = fmts[i % len(fmts)]
        x = (r.standard_normal(lens[i % len(lens)]) * 2).astype(np.float32)
        alpha = float(r.uniform(0.05, 1.0))
        if i % 4 == 3:                    # unaligned base pointer
            xd = dev(np.concatenate([[np.float32(1)], x]))[1:]
        else:
            xd = dev(x)
        ad = torch.tensor([alpha], dtype=torch.float32, device="cuda")
        cd = torch.empty(x.size + 1, dtype=torch.uint8, device="cuda")[1:] if i % 5 == 2 else \
            torch.empty(x.size, dtype=torch.uint8, device="cuda")
        rows.append((xd, ad, b, ks, cd))
        keep.append((x, alpha, b, ks, cd))
    log("project batch count=%d" % count)
    esb.esb_project_batch(esb.project_jobs(rows))
    for (x, alpha, b, ks, cd) in keep:
        np.testing.assert_array_equal(host(cd), oracle.project(x, alpha, b, ks))


def test_dda_batch_grid_scale(esb):
    """Candidates given as factors times a device scalar equal the explicit grid
    fl32(s * c_j), bit for bit, against the oracle."""
    torch = torch_cuda()
    r = np.random.default_rng(5)
    x = np.maximum(r.standard_normal(50001), 0).astype(np.float32) * np.float32(3.7)
    c = ((np.arange(64) + 1) / (64 * 6.0)).astype(np.float32)
    s = np.float32(np.max(np.abs(x)))
    grid = (s * c).astype(np.float32)
    xd = dev(x)
    a = torch.empty(1, dtype=torch.float32, device="cuda")
    D = torch.empty(64, dtype=torch.float64, device="cuda")
    cd, sd = dev(c), dev(np.array([s], dtype=np.float32))   # alive until the call has run
    jobs = esb.dda_jobs([(xd, 5, 3, cd, a, D, sd)])
    ws = torch.empty(esb.esb_dda_batch_workspace_size(jobs), dtype=torch.uint8, device="cuda")
    esb.esb_dda_align_batch(jobs, ws)
    j, Do = oracle.dda(x, 5, 3, grid)
    assert_rel(host(D), Do, REL, "scaled grid")
    assert host(a)[0] == grid[j]


def test_dda_batch_mixed_grid_scales(esb):
    """Jobs with and without a device grid scale in one batch; a scale that makes every
    candidate invalid (0, NaN) gives NaN objectives and alpha = the first candidate's value,
    like a grid of such candidates in a single call."""
    torch = torch_cuda()
    r = np.random.default_rng(8)
    xs = [(r.standard_normal(n) * 0.7).astype(np.float32) for n in (30000, 7001, 123457, 64)]
    c = ((np.arange(32) + 1) / 32.0).astype(np.float32)
    scales = [np.float32(np.max(np.abs(xs[0]))), None, np.float32(0.0), np.float32(np.nan)]
    keep, rows = [], []
    for x, sc in zip(xs, scales):
        xd = dev(x)
        cd = dev(c if sc is not None else (c * np.float32(2.5)).astype(np.float32))
        sd = None if sc is None else dev(np.array([sc], dtype=np.float32))
        a = torch.empty(1, dtype=torch.float32, device="cuda")
        D = torch.empty(32, dtype=torch.float64, device="cuda")
        keep.append((xd, cd, sd, a, D))
        rows.append((xd, 4, 2, cd, a, D, sd))
    jobs = esb.dda_jobs(rows)
    ws = torch.empty(esb.esb_dda_batch_workspace_size(jobs), dtype=torch.uint8, device="cuda")
    esb.esb_dda_align_batch(jobs, ws)
    for (x, sc), (_, _, _, a, D) in zip(zip(xs, scales), keep):
        grid = (c if sc is not None else (c * np.float32(2.5))).astype(np.float32)
        if sc is not None:
            grid = (np.float32(sc) * grid).astype(np.float32)
        j, Do = oracle.dda(x, 4, 2, grid)
        assert_rel(host(D), Do, REL, "mixed scales")
        # alpha is the chosen candidate's value: grid[0] (0 or NaN) when every one is invalid
        np.testing.assert_array_equal(host(a)[:1], grid[j:j + 1])
