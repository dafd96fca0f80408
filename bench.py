"""Benchmark of the FCM crossbar path on one MI355X.

One step = one pass of the whole path over one batch: rebuild every array's
G' from the layer weights (w_max reduction + fp64 build), unroll the input
patches through the DAC, and evaluate DAC -> V.G' -> ADC -> accumulate for
every row tile and array.  The workload is the 3x3 64->64 convolution on a
batch of 32 56 x 56 inputs mapped onto 64 x 64 crossbars (6-bit DAC, 8-bit
ADC, 1 kOhm driver and sense, 2.5 Ohm wire segments).

Prints one JSON line.  Kernel durations come from HIP events that the
library records around each of its launches on the launch stream.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix
FP64_PEAK_TFLOPS = 78.6         # MI355X fp64 (vector and matrix)
HBM_PEAK_GBS = 8000.0


def build_flops(M, N):
    """Algorithmic fp64 flops of one array's G' (row sweep, per row: one SPD
    solve of order N with N + M right-hand sides, one SPD inversion of order N;
    Cholesky counts), plus the final solve with M right-hand sides."""
    per_row = N ** 3 / 3 + 2 * N ** 2 * (N + M) + N ** 3
    return M * per_row + N ** 3 / 3 + 2 * N ** 2 * M


def cpu_baseline(work):
    """The oracle on the full workload (map every array, evaluate all images)."""
    import numpy as np
    from oracle import fcm as ofcm, mapping as omap
    from paper_1809_00072_amd import workloads as wl
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        threads = 1
    t0 = time.perf_counter()
    lay = omap.map_layer(work["W"], work["xbar"])
    t1 = time.perf_counter()
    Y = ofcm.conv_layer(work["X"], lay, work["xbar"], work["periph"], work["conv"])
    t2 = time.perf_counter()
    assert np.isfinite(Y).all()
    macs = wl.alg_macs(work)
    return {"value": macs / (t2 - t0), "unit": "MAC/s", "cores": threads, "kind": "oracle",
            "sample": "full workload once: G' of all %d arrays by sparse nodal LU (%.2f s) + "
                      "evaluation of all %d images (%.2f s), fp64 numpy/scipy"
                      % (lay["R"] * lay["C"] * lay["A"], t1 - t0, work["conv"]["n"], t2 - t1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the crossbar path is built and measured on a "
              "single MI355X; --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1809_00072_amd import rxnn, workloads as wl

    rxnn.load()
    assert torch.cuda.is_available(), "bench.py needs the HIP device"
    work = wl.conv3x3_64_56()
    cv, xb, pp = work["conv"], work["xbar"], work["periph"]
    dev = torch.device("cuda:0")
    Wd = torch.from_numpy(work["W"]).to(dev)
    Xd = torch.from_numpy(work["X"]).to(dev)
    ho, wo = rxnn.conv_out_hw(cv)
    Yd = torch.empty((cv["n"], cv["c_out"], ho, wo), dtype=torch.float32, device=dev)
    L = rxnn.map_layer(Wd, xb)
    stream = torch.cuda.current_stream()
    macs = wl.alg_macs(work)
    n_arrays = L.R * L.C * L.A

    def step():
        rxnn.remap_layer(L, Wd, stream)
        rxnn.conv_layer(L, pp, cv, Xd, Yd, stream)

    def evaluate():
        rxnn.conv_layer(L, pp, cv, Xd, Yd, stream)

    print("[bench] warmup %d" % args.warmup, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K whole steps, kernel events recorded by the library
    rxnn.profile_reset()
    rxnn.profile_enable(True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    rxnn.profile_enable(False)
    step_ms = ev0.elapsed_time(ev1) / args.steps
    kern = {}
    for name in ("wmax", "gprime_build", "dac_im2col", "xbar_vmm", "fill", "finish"):
        tot, cnt = rxnn.profile_read(name)
        if cnt:
            kern[name] = {"avg_us": 1e3 * tot / cnt, "launches": cnt}
    print("[bench] timed %d steps: %.3f ms/step" % (args.steps, step_ms), file=sys.stderr,
          flush=True)

    # evaluation only (G' kept): the paper's phase 2
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        evaluate()
    ev1.record(stream)
    torch.cuda.synchronize()
    eval_ms = ev0.elapsed_time(ev1) / args.steps

    vmm_us = kern["xbar_vmm"]["avg_us"]
    build_us = kern["gprime_build"]["avg_us"]
    if vmm_us >= build_us:
        ach = 2.0 * macs / (vmm_us * 1e-6) / 1e12
        roof = {"kernel": "xbar_vmm", "bound": "mfma", "achieved": ach,
                "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": ach / FP32_MFMA_PEAK_TFLOPS, "traffic": None}
    else:
        ach = n_arrays * build_flops(L.M, L.N) / (build_us * 1e-6) / 1e12
        roof = {"kernel": "gprime_build", "bound": "alu", "achieved": ach,
                "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": ach / FP64_PEAK_TFLOPS, "traffic": None}
    vmm_tf = 2.0 * macs / (vmm_us * 1e-6) / 1e12

    out = {
        "metric": "non-ideal crossbar MACs/sec per layer",
        "value": macs / (step_ms * 1e-3),
        "unit": "MAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 evaluation (MFMA), f64 G' build",
        "data": "synthetic",
        "config": {
            "workload": "conv3x3 s1 p1 64->64, 56x56, batch 32, 64x64 crossbars, "
                        "6-bit DAC / 8-bit ADC, 1k/1k/2.5 ohm; step = G' rebuild + evaluation",
            "alg_macs_per_step": macs,
            "arrays": n_arrays,
        },
        "roofline": roof,
        "eval_only": {"ms": eval_ms, "value": macs / (eval_ms * 1e-3), "unit": "MAC/s",
                      "xbar_vmm_tflops": vmm_tf,
                      "xbar_vmm_frac_fp32_mfma": vmm_tf / FP32_MFMA_PEAK_TFLOPS},
        "kernels": kern,
        "wall_s_timed": wall,
    }
    if not args.no_cpu_baseline:
        print("[bench] oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(work)
    L.free()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
