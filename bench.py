"""Benchmark of the ESB hot path on one MI355X.

One step = the whole hot path over one batch of the ResNet18-shaped 3x3
convolution workload (64->64 channels, 56x56, stride 1, pad 1, batch 1,
ESB n=4 / k_sig=2 for weights and activations):
    DDA scale search (64 candidates) on the weights and on the activations,
    projection of both to ESB codes, implicit-GEMM convolution over the codes
    to scaled fp32 outputs.
Inputs are synthetic, seeded and resident in HBM before timing starts.

Prints ONE JSON line.  `value` is the convolution's integer operations
(2*M*N*K) per second over the whole step, in TOPS.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
INT8_PEAK_TOPS = 5000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="approximate CPU time budget of the oracle baseline")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run only a plain device copy of known size (for counter calibration)")
    return p.parse_args()


def copy_calibration():
    import torch
    n = 256 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the hot path is measured on one MI355X "
              "(multi-GPU sharding is not part of this build); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if args.copy_calibration:
        copy_calibration()
        return

    from paper_2109_03513_amd import esb, workloads

    torch.cuda.set_device(0)
    c = workloads.resnet_conv3x3(0)
    n, ks = c["nW"], c["ksW"]
    w = torch.from_numpy(c["w"]).cuda()
    x = torch.from_numpy(c["x"]).cuda()
    gw = torch.from_numpy(c["gridW"]).cuda()
    gx = torch.from_numpy(c["gridX"]).cuda()
    Nb, H, W, C = x.shape
    K, R, S, _ = w.shape
    P, Q = esb.conv_out_hw(H, W, R, S, c["stride"], c["pad"])
    M, Ncol, Kred = Nb * P * Q, K, R * S * C
    ops = 2.0 * M * Ncol * Kred

    stream = torch.cuda.Stream()      # default priority
    sh = stream.cuda_stream
    dev = "cuda"
    aw = torch.empty(1, dtype=torch.float32, device=dev)
    ax = torch.empty(1, dtype=torch.float32, device=dev)
    Dw = torch.empty(64, dtype=torch.float64, device=dev)
    Dx = torch.empty(64, dtype=torch.float64, device=dev)
    wsw = torch.empty(esb.esb_dda_workspace_size(w.numel(), n, ks, 64), dtype=torch.uint8, device=dev)
    wsx = torch.empty(esb.esb_dda_workspace_size(x.numel(), n, ks, 64), dtype=torch.uint8, device=dev)
    cw = torch.empty(w.shape, dtype=torch.uint8, device=dev)
    cx = torch.empty(x.shape, dtype=torch.uint8, device=dev)
    y = torch.empty((Nb, P, Q, K), dtype=torch.float32, device=dev)

    stages = ["dda_w", "dda_x", "project_w", "project_x", "conv2d"]

    def run_stage(i):
        if i == 0:
            esb.esb_dda_align(w, n, ks, gw, alpha_out=aw, D_out=Dw, workspace=wsw, stream=sh)
        elif i == 1:
            esb.esb_dda_align(x, n, ks, gx, alpha_out=ax, D_out=Dx, workspace=wsx, stream=sh)
        elif i == 2:
            esb.esb_project(w, aw, n, ks, codes=cw, stream=sh)
        elif i == 3:
            esb.esb_project(x, ax, n, ks, codes=cx, stream=sh)
        else:
            esb.esb_conv2d(cx, n, ks, ax, cw, n, ks, aw, stride=c["stride"], pad=c["pad"], y=y,
                           want_acc=False, stream=sh)

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            for i in range(5):
                run_stage(i)
        stream.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(args.steps):
            ev[s][0].record(stream)
            for i in range(5):
                run_stage(i)
                ev[s][i + 1].record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    stage_ms = [sum(ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(args.steps)) / args.steps
                for i in range(5)]
    step_ms = sum(ev[s][0].elapsed_time(ev[s][5]) for s in range(args.steps)) / args.steps
    ms_per_step = max(step_ms, 1e3 * wall / args.steps)
    value = ops / (ms_per_step * 1e-3) / 1e12

    # roofline of the dominant stage
    nel_w, nel_x = w.numel(), x.numel()
    traffic_alg = {
        "dda_w": ("hbm", 4.0 * nel_w), "dda_x": ("hbm", 4.0 * nel_x),
        "project_w": ("hbm", 5.0 * nel_w), "project_x": ("hbm", 5.0 * nel_x),
        # conv: codes of x and w read once, fp32 y written once
        "conv2d": ("hbm", 1.0 * nel_x + 1.0 * nel_w + 4.0 * M * Ncol),
    }
    dom = int(np.argmax(stage_ms))
    name = stages[dom]
    bound, nbytes = traffic_alg[name]
    achieved = nbytes / (stage_ms[dom] * 1e-3) / 1e9
    roof = {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": None,
            "algorithmic_bytes": nbytes}
    conv_ms = stage_ms[4]
    extra = {
        "stages_ms": {k: round(v, 5) for k, v in zip(stages, stage_ms)},
        "conv_int_tops": round(ops / (conv_ms * 1e-3) / 1e12, 3),
        "conv_frac_int8_peak": round(ops / (conv_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 6),
        "project_x_gbps": round(5.0 * nel_x / (stage_ms[3] * 1e-3) / 1e9, 2),
        "dda_x_gbps": round(4.0 * nel_x / (stage_ms[1] * 1e-3) / 1e9, 2),
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(c, ops, args.cpu_seconds)

    rec = {
        "metric": "ESB GEMM/conv int TOPS (% of int8 MFMA peak) + projection GB/s (% HBM)",
        "value": round(value, 4), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": c["name"] + "_esb4k2_dda64",
                   "note": "DDA(w)+DDA(x)+project(w)+project(x)+conv2d per step"},
        "roofline": roof, "cpu_baseline": cpu, "detail": extra,
    }
    print(json.dumps(rec), flush=True)


def cpu_baseline(c, ops, budget_s):
    """The oracle, as it stands, on the host cores: whole steps of the same workload."""
    import numpy as np
    import oracle
    n, ks = c["nW"], c["ksW"]
    t0 = time.perf_counter()
    steps = 0
    while True:
        jw, _ = oracle.dda(c["w"], n, ks, c["gridW"])
        jx, _ = oracle.dda(c["x"], n, ks, c["gridX"])
        cw = oracle.project(c["w"], c["gridW"][jw], n, ks)
        cx = oracle.project(c["x"], c["gridX"][jx], n, ks)
        oracle.conv2d(cx, cw, n, ks, c["gridX"][jx], n, ks, c["gridW"][jw], stride=c["stride"],
                      pad=c["pad"], want_acc=False)
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 1000:
            break
    per = el / steps
    return {"value": round(ops / per / 1e12, 6), "unit": "TOPS", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": "%d whole steps of the same workload (%.3f s/step)" % (steps, per)}


if __name__ == "__main__":
    main()
