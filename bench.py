"""Benchmark of the FCM crossbar path on one MI355X.

One step = one pass of the whole path over one batch: rebuild every array's
G' from the layer weights (w_max reduction + fp64 build), unroll the input
patches through the DAC, and evaluate DAC -> V.G' -> ADC -> accumulate for
every row tile and array.  The workload is the 3x3 64->64 convolution on a
batch of 32 56 x 56 inputs mapped onto 64 x 64 crossbars (6-bit DAC, 8-bit
ADC, 1 kOhm driver and sense, 2.5 Ohm wire segments).

Prints one JSON line.  Kernel durations come from HIP events that the
library records around each of its launches on the launch stream.

--workload selects one of the other workloads instead (each prints its own
line; the default is the convolution above):
  fc256      FC 256 -> 128, batch 16, 64 x 64 crossbars (launch bound);
  resnet18   the 21 layers of a ResNet-18 shaped stack, 128 x 128 crossbars,
             wire 1 Ohm, batch 64, each layer on its own seeded input; a step
             evaluates every layer (G' mapped once);
  vgg16fc    the VGG-16 shaped FC head 25088 -> 4096 -> 4096 -> 1000, batch
             256, 8-bit weights in four 2-bit slices; a step evaluates the
             three layers;
  resnet50   the 54 layers of a ResNet-50 shaped stack, batch 128, crossbar
             side --crossbar (32 / 64 / 128 / 256), wire --wire; a step
             perturbs every layer's weights, rebuilds G' and evaluates it
             (reported: the whole step and the evaluation alone).

--retrain adds, for the convolution, a leg timed after the others: one
model-in-the-loop re-training step = G' rebuild + crossbar forward pass +
floating-point backward pass (dX and dW through the ideal weights), with the
backward GEMMs' fp32 roofline.
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
# HBM bytes per launch of k_xbar_vmm on the convolution workload, from the
# FETCH_SIZE / WRITE_SIZE counters of this kernel version, each scaled by what
# the counter reads for a plain 2 GiB copy (fetch x 2.000, write x 1.000);
# the summary and its commands are in the repository's profiles folder
VMM_TRAFFIC_BYTES = 2.0 * 15384 * 1024 + 40314 * 1024
FP64_PEAK_TFLOPS = 78.6         # MI355X fp64 (vector and matrix)
HBM_PEAK_GBS = 8000.0


def nd_ports(i0, j0, h, w, T):
    return h + (h if j0 + w < T else 0) + (w if i0 > 0 else 0) + w


def build_flops(M, N):
    """Algorithmic fp64 flops of one array's G' by nested dissection: the
    symmetric elimination of every merge's shared nodes (c of them, with E
    external ports: c^3/3 + c^2 E + c E^2) on the T x T grid the tile is
    embedded in, plus the drivers' step (eliminate the T row-input nodes and
    form the N x M transfer block)."""
    T = 16
    while T < max(M, N):
        T *= 2
    flops = 0.0
    h = w = 1
    vert = True
    while h < T or w < T:
        nh, nw = (2 * h, w) if vert else (h, 2 * w)
        c = w if vert else h
        for bi in range(T // nh):
            for bj in range(T // nw):
                E = nd_ports(bi * nh, bj * nw, nh, nw, T)
                flops += c ** 3 / 3 + c * c * E + c * E * E
        h, w, vert = nh, nw, not vert
    flops += T ** 3 / 3 + T * T * (M + T) + 2.0 * N * M * T
    return flops


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
    out = {"value": macs / (t2 - t0), "unit": "MAC/s", "cores": threads, "kind": "oracle",
           "sample": "full workload once: G' of all %d arrays by sparse nodal LU (%.2f s) + "
                     "evaluation of all %d images (%.2f s), fp64 numpy/scipy"
                     % (lay["R"] * lay["C"] * lay["A"], t1 - t0, work["conv"]["n"], t2 - t1)}
    # the same on one core (BLAS limited to one thread)
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            lay = omap.map_layer(work["W"], work["xbar"])
            ofcm.conv_layer(work["X"], lay, work["xbar"], work["periph"], work["conv"])
            t2 = time.perf_counter()
        out["one_core"] = {"value": macs / (t2 - t0), "unit": "MAC/s", "seconds": t2 - t0}
    except ImportError:
        pass
    return out


KERNEL_NAMES = ("wmax", "nd_block", "nd_merge", "nd_final", "gprime_sweep", "dac", "ktab",
                "fill", "xbar_vmm", "finish", "bw_gemm", "bw_aux", "gload")


def read_kernels(rxnn, steps):
    kern = {}
    for name in KERNEL_NAMES:
        tot, cnt = rxnn.profile_read(name)
        if cnt:
            kern[name] = {"avg_us": 1e3 * tot / cnt, "launches": cnt,
                          "us_per_step": 1e3 * tot / steps}
    return kern


# A saturating device characteristic (normalised conductance at 17 levels).
DEVICE_LUT = [(k / 16.0) ** 0.6 for k in range(17)]


def device_options(xb, args, seed=5000):
    """Per-device variation (generated, sigma = --variation) and the
    non-linear characteristic (--lut) on a crossbar parameter dict."""
    xb = dict(xb)
    if args.variation > 0.0:
        xb["variation_sigma"] = args.variation
        xb["variation_seed"] = seed
    if args.lut:
        xb["g_lut"] = DEVICE_LUT
    return xb


# The load-dependent divider DAC: full-scale branch 200 ohm, pull-down 2 kOhm.
DIVIDER_G_ON, DIVIDER_G_PD = 5e-3, 5e-4


def device_note(args):
    note = ""
    if getattr(args, "divider", False):
        note += "; load-dependent divider DAC (g_on 5 mS, g_pd 0.5 mS, no driver resistance)"
    if args.variation > 0.0:
        note += "; per-device variation sigma %g" % args.variation
    if args.lut:
        note += "; non-linear device table"
    return note


def copy_probe(torch, dev):
    """A plain elementwise copy of known size, for scaling HBM byte counters.
    The 2 GiB source is written first and then a 1 GiB buffer, so that
    little of the source is left in the 256 MB last-level cache."""
    n = 512 << 20
    a = torch.rand(n, device=dev)
    flush = torch.empty(256 << 20, device=dev)
    flush.fill_(1.0)
    b = torch.empty_like(a)
    torch.mul(a, 1.0, out=b)
    torch.cuda.synchronize()
    print("[bench] copy probe: %d bytes read, %d bytes written" % (4 * n, 4 * n),
          file=sys.stderr, flush=True)


def bench_fc256(args):
    """FC 256 -> 128, batch 16 (launch bound; absolute time only)."""
    import torch
    from paper_1809_00072_amd import rxnn, workloads as wl
    rxnn.load()
    w = wl.fc_256x128()
    dev = torch.device("cuda:0")
    Wd = torch.from_numpy(w["W"]).to(dev)
    Xd = torch.from_numpy(w["X"]).to(dev)
    L = rxnn.map_layer(Wd, w["xbar"])
    Y = rxnn.crossbar_vmm(L, w["periph"], Xd)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        rxnn.crossbar_vmm(L, w["periph"], Xd, Y, stream)
    torch.cuda.synchronize()
    rxnn.profile_reset()
    rxnn.profile_enable(2)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        rxnn.crossbar_vmm(L, w["periph"], Xd, Y, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    rxnn.profile_enable(False)
    ms = ev0.elapsed_time(ev1) / args.steps
    macs = wl.alg_macs(w)
    kern = read_kernels(rxnn, args.steps)
    vmm_us = kern["xbar_vmm"]["avg_us"]
    ach = 2.0 * macs / (vmm_us * 1e-6) / 1e12
    out = {"metric": "non-ideal crossbar MACs/sec per layer", "value": macs / (ms * 1e-3),
           "unit": "MAC/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": "fc256->128, batch 16, 64x64 crossbars, 4-bit DAC / 8-bit ADC; "
                                  "step = evaluation (launch bound)", "alg_macs_per_step": macs},
           "roofline": {"kernel": "k_xbar_vmm", "bound": "mfma", "achieved": ach,
                        "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": ach / FP32_MFMA_PEAK_TFLOPS, "traffic": None,
                        "note": "16 arrays of 64 x 64: launch and latency bound"},
           "kernels": kern}
    L.free()
    print(json.dumps(out), flush=True)


def bench_stack(args):
    """Every layer of a stacked workload, standalone on its seeded input."""
    import numpy as np
    import torch
    from paper_1809_00072_amd import rxnn, workloads as wl
    rxnn.load()
    assert torch.cuda.is_available(), "bench.py needs the HIP device"
    dev = torch.device("cuda:0")
    cfg = args.workload
    n_layers = {"resnet18": len(wl.resnet18_layers()), "vgg16fc": len(wl.vgg16_fc_layers()),
                "resnet50": len(wl.resnet50_layers())}[cfg]
    rebuild = cfg == "resnet50"
    layers = []
    print("[bench] %s: generating %d layers" % (cfg, n_layers), file=sys.stderr, flush=True)
    for l in range(n_layers):
        w = wl.stack_layer(cfg, l, crossbar=args.crossbar if rebuild else None,
                           wire=args.wire if rebuild else None)
        if rebuild:
            w["xbar"] = device_options(w["xbar"], args, seed=5000 + l)
        Wd = torch.from_numpy(w["W"]).to(dev)
        Xd = torch.from_numpy(w["X"]).to(dev)
        L = rxnn.map_layer(Wd, w["xbar"])
        if w["kind"] == "conv":
            Y = rxnn.conv_layer(L, w["periph"], w["conv"], Xd)
        else:
            Y = rxnn.crossbar_vmm(L, w["periph"], Xd)
        ent = {"w": w, "L": L, "X": Xd, "Y": Y, "W": Wd, "Wt": []}
        if rebuild:
            # model-in-the-loop update of every step: W + 1e-3 sigma eps_t
            sigma = float(np.sqrt(2.0 / w["W"].shape[0]))
            for t in range(args.warmup + args.steps):
                g = torch.Generator(device=dev).manual_seed(3000 + t)
                eps = torch.randn(Wd.shape, generator=g, device=dev)
                ent["Wt"].append(Wd + 1e-3 * sigma * eps)
        del w["X"]
        layers.append(ent)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def evaluate(e):
        w = e["w"]
        if w["kind"] == "conv":
            rxnn.conv_layer(e["L"], w["periph"], w["conv"], e["X"], e["Y"], stream)
        else:
            rxnn.crossbar_vmm(e["L"], w["periph"], e["X"], e["Y"], stream)

    # The layers' G' rebuilds are independent: they are spread over a few
    # streams (default priority) so that the small layers' builds overlap,
    # and every evaluation waits for its layer's rebuild.
    build_streams = [torch.cuda.Stream(device=dev) for _ in range(8)] if rebuild else []

    def step(t):
        if rebuild:
            done = []
            for i, e in enumerate(layers):
                bs = build_streams[i % len(build_streams)]
                bs.wait_stream(stream)
                rxnn.remap_layer(e["L"], e["Wt"][t], bs)
                ev = torch.cuda.Event()
                ev.record(bs)
                done.append(ev)
            for e, ev in zip(layers, done):
                stream.wait_event(ev)
                evaluate(e)
        else:
            for e in layers:
                evaluate(e)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    # timed steps: only the evaluation kernel carries timing events (an event
    # pair around every launch would leave the GPU idle between kernels)
    rxnn.profile_reset()
    rxnn.profile_enable(2)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for t in range(args.steps):
        step(args.warmup + t)
    ev1.record(stream)
    torch.cuda.synchronize()
    rxnn.profile_enable(False)
    step_ms = ev0.elapsed_time(ev1) / args.steps
    # per-kernel breakdown: the same steps again (same weights), every launch timed
    if rebuild or args.breakdown:
        rxnn.profile_reset()
        rxnn.profile_enable(1)
        for t in range(args.steps):
            step(args.warmup + t)
        torch.cuda.synchronize()
        rxnn.profile_enable(False)
    kern = read_kernels(rxnn, args.steps)
    # evaluation alone (G' kept); the evaluation kernel's roofline is taken
    # here, where no rebuild of another layer shares the GPU with it
    rxnn.profile_reset()
    rxnn.profile_enable(2)
    ev0.record(stream)
    for _ in range(args.steps):
        for e in layers:
            evaluate(e)
    ev1.record(stream)
    torch.cuda.synchronize()
    rxnn.profile_enable(False)
    eval_ms = ev0.elapsed_time(ev1) / args.steps
    kern_eval = read_kernels(rxnn, args.steps)
    # model generation (the paper's phase 1): one G' build of every array of
    # every layer, on one stream (the mapped-once stacks time it here; for the
    # rebuilt stack it is part of every step)
    gen = None
    if not rebuild:
        torch.cuda.synchronize()
        ev0.record(stream)
        for e in layers:
            rxnn.remap_layer(e["L"], e["W"], stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        gen = generation_info(ev0.elapsed_time(ev1),
                              int(sum(e["L"].R * e["L"].C * e["L"].A for e in layers)),
                              layers[0]["L"].M, layers[0]["L"].N)
    macs = wl.stack_alg_macs(cfg)
    vmm_us = kern_eval["xbar_vmm"]["us_per_step"]
    ach = 2.0 * macs / (vmm_us * 1e-6) / 1e12
    desc = {"resnet18": "ResNet-18 shaped stack (21 layers), batch 64, 128x128 crossbars, "
                        "wire 1 ohm, 8-bit DAC/ADC; step = evaluation of every layer",
            "vgg16fc": "VGG-16 shaped FC head 25088->4096->4096->1000, batch 256, 64x64 "
                       "crossbars, 8-bit weights in 4x2-bit slices, 8-bit DAC/ADC; step = "
                       "evaluation of the three layers",
            "resnet50": "ResNet-50 shaped stack (54 layers), batch 128, %dx%d crossbars, wire "
                        "%g ohm, 8-bit DAC/ADC; step = weight update + G' rebuild + evaluation "
                        "of every layer" % (args.crossbar, args.crossbar, args.wire)
                        + device_note(args)}[cfg]
    value_ms = step_ms
    out = {
        "metric": "non-ideal crossbar MACs/sec per layer",
        "value": macs / (value_ms * 1e-3),
        "unit": "MAC/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": value_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": desc, "alg_macs_per_step": macs,
                   "arrays": int(sum(e["L"].R * e["L"].C * e["L"].A for e in layers))},
        "roofline": {"kernel": "k_xbar_vmm (all layers)", "bound": "mfma", "achieved": ach,
                     "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / FP32_MFMA_PEAK_TFLOPS, "traffic": None},
        "eval_only": {"ms": eval_ms, "value": macs / (eval_ms * 1e-3), "unit": "MAC/s",
                      "kernels": kern_eval},
        "kernels": kern,
    }
    if gen is not None:
        out["generation"] = gen
    for e in layers:
        e["L"].free()
    print(json.dumps(out), flush=True)


# The paper's FCM model generation time for one crossbar (Sec. VIII-A; its
# hardware is not named): context for the G' build, not a target.
PAPER_GEN_S = {16: 0.038, 32: 1.2, 64: 61.0}


def generation_info(ms, arrays, M, N):
    out = {"what": "G' build of every array once (model generation)", "ms": ms,
           "arrays": arrays, "us_per_array": 1e3 * ms / arrays, "crossbar": [M, N]}
    if M == N and M in PAPER_GEN_S:
        out["paper_s_per_crossbar"] = PAPER_GEN_S[M]
    return out


def ideal_fp32_leg(torch, cv, Wd, Xd, vmm_us, eval_ms, steps):
    """Context, not the product path: the same contraction done ideally by the
    vendor libraries in fp32 (no TF32), timed with events on torch's stream.
    A convolution with Q A output channels (the differential pair as one
    layer, MIOpen) and the unrolled-patch GEMM [Bv x P] . [P x Q A]
    (hipBLASLt).  The paper sets the slowdown of its non-ideal inference
    against the ideal framework the same way (Sec. VIII, application-level
    evaluation: 2.5x)."""
    F = torch.nn.functional
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.backends.cudnn.allow_tf32 = False
    q = Wd.shape[1]
    w_pair = torch.cat([Wd.clamp(min=0.0), (-Wd).clamp(min=0.0)], dim=1)   # P x 2Q
    wconv = w_pair.t().contiguous().view(2 * q, cv["c_in"], cv["kh"], cv["kw"])
    cols = F.unfold(Xd, (cv["kh"], cv["kw"]), padding=cv["pad"], stride=cv["stride"])
    cols = cols.transpose(1, 2).reshape(-1, cols.shape[1]).contiguous()       # Bv x P
    out = torch.empty((cols.shape[0], 2 * q), dtype=torch.float32, device=Xd.device)
    flops = 2.0 * cols.shape[0] * cols.shape[1] * 2 * q

    def timed(fn):
        for _ in range(3):
            fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return 1e3 * e0.elapsed_time(e1) / steps

    conv_us = timed(lambda: F.conv2d(Xd, wconv, stride=cv["stride"], padding=cv["pad"]))
    gemm_us = timed(lambda: torch.matmul(cols, w_pair, out=out))
    return {"what": "ideal fp32 layer of the same MACs by the vendor libraries (context)",
            "conv2d_us": conv_us, "conv2d_tflops": flops / conv_us * 1e-6,
            "gemm_us": gemm_us, "gemm_tflops": flops / gemm_us * 1e-6,
            "xbar_vmm_over_gemm": vmm_us / gemm_us,
            "eval_over_conv2d": 1e3 * eval_ms / conv_us}


def retrain_leg(args, torch, rxnn, wl, L, pp, cv, Wd, Xd, Yd, stream):
    """K re-training steps of the convolution: rebuild G' from the weights,
    the crossbar forward pass, and the backward pass (dX, dW) of a seeded
    output gradient.  The weight update itself (W -= lr dW) belongs to the
    caller's optimizer and is not part of the step."""
    dY = torch.from_numpy(wl.normal(3003, tuple(Yd.shape), 1.0)).to(Xd.device)
    dX, dW = torch.empty_like(Xd), torch.empty_like(Wd)

    def step():
        rxnn.remap_layer(L, Wd, stream)
        rxnn.conv_layer(L, pp, cv, Xd, Yd, stream)
        rxnn.conv_backward(L, pp, cv, Wd, Xd, dY, dX=dX, dW=dW, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    rxnn.profile_reset()
    rxnn.profile_enable(1)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    rxnn.profile_enable(False)
    kern = read_kernels(rxnn, args.steps)
    ho, wo = rxnn.conv_out_hw(cv)
    bv = cv["n"] * ho * wo
    gemm_flops = 2 * 2.0 * bv * L.P * L.Q           # dW = cols^T dY and dcols = dY W^T
    g_us = kern["bw_gemm"]["us_per_step"]
    ach = gemm_flops / (g_us * 1e-6) / 1e12
    print("[bench] retrain: %.3f ms/step" % ms, file=sys.stderr, flush=True)
    return {"ms_per_step": ms, "backward_gemm": {
        "us_per_step": g_us, "bound": "mfma", "achieved": ach, "peak": FP32_MFMA_PEAK_TFLOPS,
        "unit": "TFLOP/s", "frac": ach / FP32_MFMA_PEAK_TFLOPS, "flops": gemm_flops},
        "backward_aux_us_per_step": kern.get("bw_aux", {}).get("us_per_step", 0.0),
        "kernels": kern}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 2 GiB copy kernel (counter calibration)")
    ap.add_argument("--workload", default="conv3x3",
                    choices=["conv3x3", "fc256", "resnet18", "vgg16fc", "resnet50"])
    ap.add_argument("--crossbar", type=int, default=256, help="resnet50: crossbar side")
    ap.add_argument("--wire", type=float, default=2.5, help="resnet50: wire resistance (Ohm)")
    ap.add_argument("--variation", type=float, default=0.0,
                    help="conv3x3 / resnet50: generated per-device variation, sigma (e.g. 0.1)")
    ap.add_argument("--lut", action="store_true",
                    help="conv3x3 / resnet50: a non-linear device characteristic table")
    ap.add_argument("--divider", action="store_true",
                    help="conv3x3: the load-dependent divider DAC (layer mapped without "
                         "driver resistance)")
    ap.add_argument("--retrain", action="store_true",
                    help="conv3x3: also time re-training steps (rebuild + forward + backward)")
    ap.add_argument("--breakdown", action="store_true",
                    help="stacks without rebuild: also time every launch in a second pass")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the crossbar path is built and measured on a "
              "single MI355X; --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.workload in ("resnet18", "vgg16fc", "resnet50"):
        return bench_stack(args)
    if args.workload == "fc256":
        return bench_fc256(args)

    import numpy as np
    import torch
    from paper_1809_00072_amd import rxnn, workloads as wl

    rxnn.load()
    assert torch.cuda.is_available(), "bench.py needs the HIP device"
    work = wl.conv3x3_64_56()
    cv, xb, pp = work["conv"], work["xbar"], work["periph"]
    xb = device_options(xb, args)
    if args.divider:
        xb = dict(xb, r_driver=0.0)
        pp = dict(pp, dac_bend=0.0, dac_g_on=DIVIDER_G_ON, dac_g_pd=DIVIDER_G_PD)
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

    # timed region: K whole steps; the library brackets the evaluation kernel
    # with HIP events on the launch stream (level 2: the other launches stay
    # back to back, an event pair around each would idle the GPU between them)
    rxnn.profile_reset()
    rxnn.profile_enable(2)
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
    vmm_timed = read_kernels(rxnn, args.steps)["xbar_vmm"]
    print("[bench] timed %d steps: %.3f ms/step" % (args.steps, step_ms), file=sys.stderr,
          flush=True)
    # per-kernel breakdown: K more identical steps with every launch timed
    rxnn.profile_reset()
    rxnn.profile_enable(1)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    rxnn.profile_enable(False)
    kern = read_kernels(rxnn, args.steps)

    # evaluation only (G' kept): the paper's phase 2
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        evaluate()
    ev1.record(stream)
    torch.cuda.synchronize()
    eval_ms = ev0.elapsed_time(ev1) / args.steps

    # the dominant single kernel is the evaluation kernel (timed in the timed region)
    vmm_us = vmm_timed["avg_us"]
    ach = 2.0 * macs / (vmm_us * 1e-6) / 1e12
    roof = {"kernel": "k_xbar_vmm", "bound": "mfma", "achieved": ach,
            "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": ach / FP32_MFMA_PEAK_TFLOPS, "traffic": VMM_TRAFFIC_BYTES}
    build_us = sum(kern[k]["us_per_step"] for k in ("nd_block", "nd_merge", "nd_final",
                                                     "gprime_sweep") if k in kern)
    b_ach = n_arrays * build_flops(L.M, L.N) / (build_us * 1e-6) / 1e12
    build = {"us_per_step": build_us, "bound": "alu", "achieved": b_ach,
             "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": b_ach / FP64_PEAK_TFLOPS,
             "generation": generation_info(1e-3 * build_us, n_arrays, L.M, L.N)}

    ideal = ideal_fp32_leg(torch, cv, Wd, Xd, vmm_us, eval_ms, args.steps)
    if args.copy_probe:
        copy_probe(torch, dev)
    retrain = retrain_leg(args, torch, rxnn, wl, L, pp, cv, Wd, Xd, Yd, stream) \
        if args.retrain else None

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
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "conv3x3 s1 p1 64->64, 56x56, batch 32, 64x64 crossbars, "
                        "6-bit DAC / 8-bit ADC, 1k/1k/2.5 ohm; step = G' rebuild + evaluation"
                        + device_note(args),
            "alg_macs_per_step": macs,
            "arrays": n_arrays,
        },
        "roofline": roof,
        "build": build,
        "eval_only": {"ms": eval_ms, "value": macs / (eval_ms * 1e-3), "unit": "MAC/s"},
        "ideal_fp32": ideal,
        "kernels": kern,
        "kernels_pass": "a second pass of the same steps with every launch timed",
        "wall_s_timed": wall,
    }
    if retrain is not None:
        out["retrain"] = retrain
    if not args.no_cpu_baseline:
        print("[bench] oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(dict(work, xbar=xb, periph=pp))
    L.free()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
