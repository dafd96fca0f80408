"""Benchmark of the FCM crossbar path on one MI355X.

One step = one pass of the whole path over one batch: rebuild every array's
G' from the step's layer weights (w_max reduction + fp64 build; the model is
regenerated every step, as in model-in-the-loop re-training), and evaluate
DAC -> V.G' -> ADC -> accumulate for every row tile and array of every
layer.  The default workload is the ResNet-50 shaped stack (53 convolutions
and the classifier), batch 128, on 256 x 256 crossbars with 2.5 Ohm wire
segments, 8-bit DAC / ADC, 1 kOhm driver and sense resistances.

Prints one JSON line: `value` is the whole step (map + VMM); `eval_only` the
evaluation alone (VMM only, G' kept), `map_only` the rebuild alone.  The
`roofline` is the evaluation kernel's, summed over the layers of an
evaluation-only pass; `hbm` gives the DAC pass's and the finish kernel's
achieved bandwidth; `cpu_baseline` the oracle on a seeded sample, on the
host's cores, extrapolated to the whole step, and `sample_parity` the GPU's
outputs on that sample under the parity tests' rule.  Kernel durations come
from HIP events that the library records around its launches on the launch
stream.

--workload selects one of the other workloads instead:
  conv3x3    3x3 s1 p1 64 -> 64 convolution on 32 x 64 x 56 x 56, 64 x 64
             crossbars, 6-bit DAC / 8-bit ADC; a step rebuilds G' (18 arrays)
             and evaluates; the oracle runs the whole workload;
  fc256      FC 256 -> 128, batch 16, 64 x 64 crossbars (launch bound);
  resnet18   the 21 layers of a ResNet-18 shaped stack, 128 x 128 crossbars,
             wire 1 Ohm, batch 64, each layer on its own seeded input; a step
             evaluates every layer (G' mapped once);
  vgg16fc    the VGG-16 shaped FC head 25088 -> 4096 -> 4096 -> 1000, batch
             256, 8-bit weights in four 2-bit slices; a step evaluates the
             three layers;
  resnet50   the default, with --crossbar (32 / 64 / 128 / 256) and --wire.

--retrain adds, for the convolution, a leg timed after the others: one
model-in-the-loop re-training step = G' rebuild + crossbar forward pass +
floating-point backward pass (dX and dW through the ideal weights), with the
backward contractions' fp32 roofline.
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
VMM_TRAFFIC_BYTES = 2.0 * 15182.7 * 1024 + 39424 * 1024
# HBM bytes of k_xbar_vmm per evaluation-only pass of a stacked workload
# (summed over its layers), from the same counters and the same calibration
# (fetch x 2.000, write x 1.000 from a plain 2 GiB copy in the same run), keyed
# by (workload, crossbar side, wire); the summary and its commands are in the
# repository's profiles folder.  Absent where they have not been taken.
STACK_VMM_TRAFFIC = {
    # ResNet-50 stack, 256 x 256, 2.5 ohm: 7,188,444 KiB fetched x 2.000 +
    # 5,896,956 KiB written per pass (54 dispatches)
    ("resnet50", 256, 2.5): 2.0 * 7188443.9 * 1024 + 5896956.4 * 1024,
}
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


def host_info():
    """CPU model and the number of cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return model, n


def oracle_workers():
    # the GPU machine gives one GPU's job a share of 16 host cores
    return max(1, min(16, host_info()[1]))


def _one_thread_blas():
    # every worker runs its own share: one BLAS thread each, no oversubscription
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(limits=1)
    except ImportError:
        pass


# Inputs of the oracle's sample, set before the worker pool forks (the workers
# inherit them): key -> dict of numpy arrays and parameters.
_SAMPLE = {}


def _oracle_tile(task):
    """Worker: G' of every array of tile (r, c) of sampled layer `key`
    (generator steps 1-3 of the oracle)."""
    import numpy as np
    from oracle import mapping as omap
    key, r, c = task
    s = _SAMPLE[key]
    xb = s["xbar"]
    t0 = time.perf_counter()
    vf = omap.variation_factors(xb, r, c, s["R"], s["A"], s["M"], s["N"])
    G = omap.array_conductances(omap.tile_weights(s["W"], xb, r, c), xb, s["w_max"], vf)
    gp = np.stack([omap.array_gprime(G[a], xb) for a in range(G.shape[0])])
    return key, r, c, gp, time.perf_counter() - t0


def _oracle_eval(task):
    """Worker: product rows [lo, hi) of the sample of layer `key` through the
    oracle's evaluation (DAC, V.G', ADC, integer accumulation) over its column
    tiles, with the G' the sample holds (built before the workers forked).
    Returns those columns of Y; with `debug` also the per-array currents and
    codes (for the parity check; not timed: moving them between processes
    costs more than computing them)."""
    from oracle import fcm as ofcm
    key, lo, hi, debug = task
    s = _SAMPLE[key]
    lay = dict(s["lay"], gp=s["gp"])
    t0 = time.perf_counter()
    res = ofcm.crossbar_vmm(s["Xs"][lo:hi], lay, s["xbar"], s["periph"], col_tiles=s["cols"],
                            debug=debug)
    dt = time.perf_counter() - t0
    Y, dbg = res if debug else (res, None)
    q0 = min(s["cols"]) * s["N"]
    q1 = min(s["Q"], (max(s["cols"]) + 1) * s["N"])
    return key, Y[:, q0:q1], dbg, dt


def _ready(_):
    return os.getpid()


def _layer_scalars(W, xb):
    from oracle import mapping as omap
    P, Q = W.shape
    M, N = int(xb["rows"]), int(xb["cols"])
    R, C = omap.tile_grid(P, Q, M, N)
    w_max = omap.layer_w_max(W, xb)
    return {"P": P, "Q": Q, "M": M, "N": N, "R": R, "C": C,
            "A": omap.arrays_per_position(xb), "w_max": w_max,
            "s_w_eff": omap.effective_weight_scale(xb, w_max)}


def conv_patch_sample(conv, per_image, seed):
    """Seeded product rows of a convolution: per_image output pixels of the
    first and of the last image, always including each image's first and
    last pixel, interleaved (first image, last image, first, ...).  Returns
    (images, pixels, H_out, W_out)."""
    import numpy as np
    ho = (conv["h"] + 2 * conv["pad"] - conv["kh"]) // conv["stride"] + 1
    wo = (conv["w"] + 2 * conv["pad"] - conv["kw"]) // conv["stride"] + 1
    rng = np.random.default_rng(seed)
    per = []
    for img in sorted({0, conv["n"] - 1}):
        k = min(per_image, ho * wo)
        pix = [0, ho * wo - 1] + [int(v) for v in rng.permutation(ho * wo)]
        pix = list(dict.fromkeys(pix))[:k]
        per.append([(img, p) for p in pix])
    rows = [r for grp in zip(*per) for r in grp] if len(per) > 1 else per[0]
    return (np.array([r[0] for r in rows]), np.array([r[1] for r in rows]), ho, wo)


def sample_rows(work, n_rows, seed):
    """The layer's sampled product rows: (X rows for the oracle [S x P],
    a selector that takes the same rows out of the GPU's output)."""
    import numpy as np
    from oracle import fcm as ofcm
    if work["kind"] == "conv":
        cv = work["conv"]
        img, pix, ho, wo = conv_patch_sample(cv, n_rows // 2, seed)
        imgs = sorted(set(int(i) for i in img))
        patches = ofcm.im2col(work["X"], cv, imgs)
        local = np.searchsorted(imgs, img) * (ho * wo) + pix
        return patches[local], ("conv", img, pix, wo)
    B = work["X"].shape[0]
    rows = np.sort(np.random.default_rng(seed).permutation(B)[:min(n_rows, B)])
    return work["X"][rows], ("fc", rows)


def select_rows(Y, sel):
    """The sampled rows of a GPU output (numpy), as [S x Q]."""
    if sel[0] == "conv":
        _, img, pix, wo = sel
        return Y[img, :, pix // wo, pix % wo]
    return Y[sel[1]]


# Sampled rows per layer whose outputs are compared with the GPU's.
PARITY_ROWS = 128
# Arrays of the oracle's build sample per crossbar side: about 10-20 s on 16
# host cores with the oracle's per-array cost at that side.
SAMPLE_ARRAYS = {16: 4096, 32: 2048, 64: 768, 128: 256, 256: 96}


def oracle_sample(works, total_arrays, total_macs, seed=4242, n_rows=1024):
    """The oracle timed on a seeded sample of a stacked workload, on the host's
    cores, and extrapolated to the whole workload.

    Sample: layers in a seeded order until about SAMPLE_ARRAYS[side] arrays;
    for each, the last column tile (possibly padded) with every row tile's G'
    (one process per tile), and n_rows product rows (FC: batch rows; conv:
    output pixels of the first and last image) evaluated over it (one process
    per block of 128 rows).  Full time = build time per array x arrays + evaluation time
    per MAC x MACs, both measured here, on all workers and on one core."""
    import multiprocessing as mp
    import numpy as np
    M = int(works[0]["xbar"]["rows"])
    target = SAMPLE_ARRAYS.get(M, 256)
    order = np.random.default_rng(seed).permutation(len(works))
    keys, n_arrays = [], 0
    for l in order:
        w = works[int(l)]
        sc = _layer_scalars(w["W"], w["xbar"])
        if keys and n_arrays + sc["R"] * sc["A"] > 1.5 * target:
            continue
        c = sc["C"] - 1
        Xs, sel = sample_rows(w, n_rows, seed + int(l))
        _SAMPLE[int(l)] = {"W": w["W"], "xbar": w["xbar"], "periph": w["periph"], "Xs": Xs,
                           "sel": sel, "cols": [c], **sc, "lay": sc}
        keys.append(int(l))
        n_arrays += sc["R"] * sc["A"]
        if n_arrays >= target:
            break
    tasks = [(k, r, _SAMPLE[k]["cols"][0]) for k in keys for r in range(_SAMPLE[k]["R"])]
    workers = oracle_workers()
    ctx = mp.get_context("fork")
    print("[bench] oracle sample: %d layers, %d arrays, %d workers"
          % (len(keys), n_arrays, workers), file=sys.stderr, flush=True)
    with ctx.Pool(workers, initializer=_one_thread_blas) as pool:
        pool.map(_ready, range(workers))   # the workers are up before the clock starts
        t0 = time.perf_counter()
        built = pool.map(_oracle_tile, tasks, chunksize=1)
        t_build = time.perf_counter() - t0
    for k in keys:
        _SAMPLE[k]["gp"] = {}
    for k, r, c, gp, _ in built:
        _SAMPLE[k]["gp"][(r, c)] = gp
    # the evaluation: row blocks over a second pool, forked after the build so
    # that its workers hold every G'; one untimed pass first (the workers'
    # first allocations), then the timed one
    blocks = [(k, lo, min(lo + 128, _SAMPLE[k]["Xs"].shape[0]), False) for k in keys
              for lo in range(0, _SAMPLE[k]["Xs"].shape[0], 128)]
    with ctx.Pool(workers, initializer=_one_thread_blas) as pool:
        pool.map(_oracle_eval, blocks, chunksize=1)
        t0 = time.perf_counter()
        pool.map(_oracle_eval, blocks, chunksize=1)
        t_eval = time.perf_counter() - t0
        # for the parity check (not timed): the first PARITY_ROWS rows
        evals = pool.map(_oracle_eval, [(k, 0, min(PARITY_ROWS, _SAMPLE[k]["Xs"].shape[0]), True)
                                        for k in keys], chunksize=1)

    def sample_macs(s):
        c = s["cols"][0]
        return s["Xs"].shape[0] * s["P"] * (min(s["Q"], (c + 1) * s["N"]) - c * s["N"]) * s["A"]

    macs_all = sum(sample_macs(_SAMPLE[k]) for k in keys)
    # one core: one tile's build and the whole evaluation sample, here
    try:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(limits=1)
    except ImportError:
        limit = None
    _, _, _, _, t1_tile = _oracle_tile(tasks[0])
    t0 = time.perf_counter()
    for k in keys:
        _oracle_eval((k, 0, _SAMPLE[k]["Xs"].shape[0], False))
    t1_eval = time.perf_counter() - t0
    if limit is not None:
        limit.unregister()
    macs1 = macs_all
    a0 = _SAMPLE[tasks[0][0]]["A"]
    t_full = t_build / n_arrays * total_arrays + t_eval / macs_all * total_macs
    t_one = t1_tile / a0 * total_arrays + t1_eval / macs1 * total_macs
    model, ncores = host_info()
    out = {"value": total_macs / t_full, "unit": "MAC/s", "cores": workers, "kind": "oracle",
           "extrapolated": True,
           "sample": "seeded: %d of %d layers, each its last column tile with every row "
                     "tile's G' (%d arrays of %dx%d: oracle row sweep / nodal LU, fp64) and %d "
                     "product rows evaluated over it (%.3g MACs); full step extrapolated as "
                     "build s/array x %d arrays + evaluation s/MAC x %.4g MACs"
                     % (len(keys), len(works), n_arrays, M, M, n_rows, macs_all,
                        total_arrays, total_macs),
           "seconds": {"sample_build": t_build, "sample_eval": t_eval,
                       "extrapolated_step": t_full,
                       "extrapolated_build": t_build / n_arrays * total_arrays,
                       "extrapolated_eval": t_eval / macs_all * total_macs},
           "host": {"cpu": model, "cores_available": ncores, "workers": workers},
           "one_core": {"value": total_macs / t_one, "unit": "MAC/s", "extrapolated_step_s": t_one,
                        "sample": "one tile's build (%d arrays, %.2f s) and the evaluation "
                                  "sample (%.3g MACs, %.2f s) on one core"
                                  % (a0, t1_tile, macs1, t1_eval)}}
    out["all_over_one_core"] = out["value"] / out["one_core"]["value"]
    results = {k: (Y, dbg) for k, Y, dbg, _ in evals}
    return out, results


def sample_parity(works, layers, results, rxnn, torch, stream):
    """GPU outputs of the sampled rows against the oracle's codes on the base
    weights (the rule of the parity tests: fp32(integer) * scale, the integer
    off the oracle's only by codes whose current sits on a threshold)."""
    import numpy as np
    tests_dir = os.path.join(ROOT, "tests")
    if tests_dir not in sys.path:
        sys.path.insert(0, tests_dir)
    from parity import array_weights, check_outputs_by_codes
    from oracle import mapping as omap, periph as oper
    n_out = n_diff = n_codes = 0
    for k, (Yo, dbg) in results.items():
        s, e = _SAMPLE[k], layers[k]
        rxnn.remap_layer(e["L"], e["W"], stream)
        w = works[k]
        if w["kind"] == "conv":
            rxnn.conv_layer(e["L"], w["periph"], w["conv"], e["X"], e["Y"], stream)
        else:
            rxnn.crossbar_vmm(e["L"], w["periph"], e["X"], e["Y"], stream)
        torch.cuda.synchronize()
        n_par = next(iter(dbg.values()))[0].shape[0]
        Yg = select_rows(e["Y"].cpu().numpy(), s["sel"])[:n_par]
        pp, xb = s["periph"], s["xbar"]
        thr = oper.adc_thresholds(int(pp["adc_bits"]), oper.adc_full_scale(pp, s["M"], xb["g_max"]),
                                  pp["adc_bend"])
        scale = oper.output_scale(pp, s["M"], xb["g_max"], s["s_w_eff"])
        weights = array_weights(s["A"], omap.slicing(xb)[1])
        c = s["cols"][0]
        q0, q1 = c * s["N"], min(s["Q"], (c + 1) * s["N"])
        part = {(r, a): (I[:, :q1 - q0], code[:, :q1 - q0])
                for (r, cc, a), (I, code) in dbg.items() if cc == c}
        nd, nc = check_outputs_by_codes(Yg[:, q0:q1], part, weights, thr, scale)
        n_out += Yg[:, q0:q1].size
        n_diff += nd
        n_codes += nc
    return {"outputs_compared": n_out, "outputs_off_by_threshold_flips": n_diff,
            "codes_behind_them": n_codes, "rule": "fp32(integer) x scale; integer off the "
            "oracle's only by codes within 1e-4 of a threshold, <= 0.1 % of the codes"}


def cpu_baseline_conv(work):
    """The oracle on the whole convolution workload: every array's G' (one
    process per tile) and the evaluation of every image (one process per
    image), on the host's cores; then one tile and one image on one core."""
    import multiprocessing as mp
    import numpy as np
    from paper_1809_00072_amd import workloads as wl
    from oracle import fcm as ofcm
    cv = work["conv"]
    sc = _layer_scalars(work["W"], work["xbar"])
    n = cv["n"]
    ho, wo = ofcm.conv_out_hw(cv)
    for img in range(n):
        _SAMPLE[("img", img)] = {"W": work["W"], "xbar": work["xbar"], "periph": work["periph"],
                                 "Xs": ofcm.im2col(work["X"], cv, [img]),
                                 "cols": list(range(sc["C"])), **sc, "lay": sc}
    _SAMPLE["conv"] = _SAMPLE[("img", 0)]
    tasks = [("conv", r, c) for c in range(sc["C"]) for r in range(sc["R"])]
    workers = oracle_workers()
    ctx = mp.get_context("fork")
    with ctx.Pool(workers, initializer=_one_thread_blas) as pool:
        pool.map(_ready, range(workers))   # the workers are up before the clock starts
        t0 = time.perf_counter()
        built = pool.map(_oracle_tile, tasks, chunksize=1)
        t1 = time.perf_counter()
    gp = {(r, c): g for _, r, c, g, _ in built}
    for img in range(n):
        _SAMPLE[("img", img)]["gp"] = gp
    # the evaluation: one process per image, forked after the build (the
    # workers hold G'); one untimed pass first, then the timed one
    img_tasks = [(("img", i), 0, ho * wo, False) for i in range(n)]
    with ctx.Pool(workers, initializer=_one_thread_blas) as pool:
        pool.map(_oracle_eval, img_tasks[:workers], chunksize=1)
        t1b = time.perf_counter()
        evals = pool.map(_oracle_eval, img_tasks, chunksize=1)
        t2 = time.perf_counter()
    t2 -= t1b - t1
    for _, Y, _, _ in evals:
        assert np.isfinite(Y).all()
    macs = wl.alg_macs(work)
    try:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(limits=1)
    except ImportError:
        limit = None
    _, _, _, _, t_tile = _oracle_tile(tasks[0])
    _, _, _, t_img = _oracle_eval((("img", 0), 0, ho * wo, False))
    if limit is not None:
        limit.unregister()
    t_one = t_tile * len(tasks) + t_img * n
    model, ncores = host_info()
    out = {"value": macs / (t2 - t0), "unit": "MAC/s", "cores": workers, "kind": "oracle",
           "sample": "full workload once: G' of all %d arrays (%.2f s) + evaluation of all %d "
                     "images (%.2f s), fp64 numpy/scipy, one process per tile / image"
                     % (sc["R"] * sc["C"] * sc["A"], t1 - t0, n, t2 - t1),
           "host": {"cpu": model, "cores_available": ncores, "workers": workers},
           "one_core": {"value": macs / t_one, "unit": "MAC/s", "seconds": t_one,
                        "sample": "one tile's build and one image's evaluation on one core, "
                                  "scaled to the whole workload"}}
    out["all_over_one_core"] = out["value"] / out["one_core"]["value"]
    return out


KERNEL_NAMES = ("wmax", "nd_block", "nd_merge", "nd_final", "gprime_sweep", "dac", "ktab",
                "fill", "xbar_vmm", "finish", "bw_dw", "bw_dx", "bw_reduce", "gload")


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


STACK_DESC = {
    "resnet18": "ResNet-18 shaped stack (21 layers), batch 64, 128x128 crossbars, wire 1 ohm, "
                "8-bit DAC/ADC; step = evaluation of every layer (G' mapped once)",
    "vgg16fc": "VGG-16 shaped FC head 25088->4096->4096->1000, batch 256, 64x64 crossbars, "
               "8-bit weights in 4x2-bit slices, 8-bit DAC/ADC; step = evaluation of the three "
               "layers (G' mapped once)",
    "resnet50": "ResNet-50 shaped stack (54 layers), batch 128, %dx%d crossbars, wire %g ohm, "
                "8-bit DAC/ADC; step = G' rebuild of all %d arrays from the step's weights "
                "(%s) + "
                "evaluation of every layer (each step's weights W + 1e-3 sigma eps_t are drawn "
                "before the timed region)",
}


def bench_stack(args):
    """Every layer of a stacked workload, standalone on its seeded input.

    resnet50 (the default workload): a step rebuilds every array's G' from
    that step's weights (model-in-the-loop re-training, G' regenerated every
    step) and evaluates every layer; the line also gives the evaluation alone
    (VMM only) and the rebuild alone (map only)."""
    import numpy as np
    from paper_1809_00072_amd import workloads as wl
    cfg = args.workload
    specs = {"resnet18": wl.resnet18_layers, "vgg16fc": wl.vgg16_fc_layers,
             "resnet50": wl.resnet50_layers}[cfg]()
    rebuild = cfg == "resnet50"
    print("[bench] %s: generating %d layers" % (cfg, len(specs)), file=sys.stderr, flush=True)
    works = []
    for l in range(len(specs)):
        w = wl.stack_layer(cfg, l, crossbar=args.crossbar if rebuild else None,
                           wire=args.wire if rebuild else None)
        if rebuild:
            w["xbar"] = device_options(w["xbar"], args, seed=5000 + l)
        works.append(w)
    macs = wl.stack_alg_macs(cfg)
    total_arrays = 0
    for w in works:
        sc = _layer_scalars(w["W"], w["xbar"])
        total_arrays += sc["R"] * sc["C"] * sc["A"]
    # the oracle's sample runs first, before the GPU is touched (its worker
    # processes fork from this one)
    cpu = results = None
    if not args.no_cpu_baseline:
        cpu, results = oracle_sample(works, total_arrays, macs)
        print("[bench] oracle: %.3g MAC/s extrapolated on %d workers (%.3g on one core)"
              % (cpu["value"], cpu["cores"], cpu["one_core"]["value"]), file=sys.stderr,
              flush=True)

    import torch
    from paper_1809_00072_amd import rxnn
    rxnn.load()
    assert torch.cuda.is_available(), "bench.py needs the HIP device"
    dev = torch.device("cuda:0")
    layers = []
    for l, w in enumerate(works):
        Wd = torch.from_numpy(w["W"]).to(dev)
        Xd = torch.from_numpy(w["X"]).to(dev)
        L = rxnn.map_layer(Wd, w["xbar"])
        if w["kind"] == "conv":
            Y = rxnn.conv_layer(L, w["periph"], w["conv"], Xd)
        else:
            Y = rxnn.crossbar_vmm(L, w["periph"], Xd)
        ent = {"L": L, "X": Xd, "Y": Y, "W": Wd, "Wt": []}
        if rebuild:
            # model-in-the-loop update of every step: W + 1e-3 sigma eps_t
            sigma = float(np.sqrt(2.0 / w["W"].shape[0]))
            for t in range(args.warmup + args.steps):
                g = torch.Generator(device=dev).manual_seed(3000 + t)
                eps = torch.randn(Wd.shape, generator=g, device=dev)
                ent["Wt"].append(Wd + 1e-3 * sigma * eps)
        w["X"] = None
        layers.append(ent)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def evaluate(l):
        e, w = layers[l], works[l]
        if w["kind"] == "conv":
            rxnn.conv_layer(e["L"], w["periph"], w["conv"], e["X"], e["Y"], stream)
        else:
            rxnn.crossbar_vmm(e["L"], w["periph"], e["X"], e["Y"], stream)

    # Per-layer rebuilds (for comparison) are spread over a few streams
    # (default priority) so that the small layers' builds overlap.
    build_streams = [torch.cuda.Stream(device=dev) for _ in range(8)] if rebuild else []
    if rebuild and not args.per_layer_rebuild:
        # the batched rebuild's tables and workspace are set up here, outside
        # the timed region
        rxnn.remap_layers([e["L"] for e in layers], [e["W"] for e in layers], stream)

    def rebuild_per_layer(t):
        done = []
        for i, e in enumerate(layers):
            bs = build_streams[i % len(build_streams)]
            bs.wait_stream(stream)
            rxnn.remap_layer(e["L"], e["Wt"][t], bs)
            ev = torch.cuda.Event()
            ev.record(bs)
            done.append(ev)
        for ev in done:
            stream.wait_event(ev)

    def rebuild_all(t):
        # every layer's G' in one launch sequence (the layers share the
        # crossbar size and resistances)
        if args.per_layer_rebuild:
            rebuild_per_layer(t)
        else:
            rxnn.remap_layers([e["L"] for e in layers], [e["Wt"][t] for e in layers], stream)

    def step(t):
        if rebuild:
            rebuild_all(t)
        for l in range(len(layers)):
            evaluate(l)

    def timed(fn, n, level):
        rxnn.profile_reset()
        rxnn.profile_enable(level)
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(n):
            fn(i)
        ev1.record(stream)
        torch.cuda.synchronize()
        rxnn.profile_enable(0)
        return ev0.elapsed_time(ev1) / n

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    # timed steps: only the evaluation kernel carries timing events (an event
    # pair around every launch would leave the GPU idle between kernels)
    w0 = time.perf_counter()
    step_ms = timed(lambda i: step(args.warmup + i), args.steps, 2)
    wall = time.perf_counter() - w0
    print("[bench] timed %d steps: %.3f ms/step" % (args.steps, step_ms), file=sys.stderr,
          flush=True)
    # per-kernel breakdown: the same steps again, every launch timed
    kern = None
    if rebuild or args.breakdown:
        timed(lambda i: step(args.warmup + i), args.steps, 1)
        kern = read_kernels(rxnn, args.steps)
    # the rebuild alone (map only), on the same streams
    map_ms = map_pl_ms = None
    if rebuild:
        map_ms = timed(lambda i: rebuild_all(args.warmup + i), args.steps, 0)
        # for comparison: one rxnn_remap_layer per layer, spread over 8 streams
        map_pl_ms = timed(lambda i: rebuild_per_layer(args.warmup + i), args.steps, 0)
    # the evaluation alone (VMM only, G' kept): the evaluation kernel's
    # roofline is taken here, where no rebuild shares the GPU with it
    def eval_all(i):
        for l in range(len(layers)):
            evaluate(l)
    eval_ms = timed(eval_all, args.steps, 2)
    kern_eval = read_kernels(rxnn, args.steps)
    # and once more with every launch timed: the DAC pass and the finish
    # kernel's achieved HBM bandwidth (their algorithmic bytes per launch are
    # counted by the library)
    timed(eval_all, args.steps, 1)
    kern_eval_all = read_kernels(rxnn, args.steps)
    hbm = {}
    for name, what in (("dac", "k_dac: DAC of every input into the (padded) V buffer; "
                                "4 B read per input + 4 B written per V element"),
                       ("finish", "k_finish / k_finish_nchw: shared tiles' int32 workspace -> "
                                  "Y; 12 B per output (read, zeroing write, fp32 write)")):
        tot_ms, cnt = rxnn.profile_read(name)
        if cnt:
            gbs = rxnn.profile_bytes(name) / (tot_ms * 1e-3) / 1e9
            hbm[name] = {"what": what, "us_per_step": 1e3 * tot_ms / args.steps,
                         "bytes_per_step": rxnn.profile_bytes(name) / args.steps,
                         "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": gbs / HBM_PEAK_GBS}
    gen = None
    if not rebuild:
        # model generation (the paper's phase 1): one G' build of every array
        # of every layer, on one stream
        def gen_all(i):
            for e in layers:
                rxnn.remap_layer(e["L"], e["W"], stream)
        gen = generation_info(timed(gen_all, 1, 0), total_arrays, layers[0]["L"].M,
                              layers[0]["L"].N)
    if args.copy_probe:
        copy_probe(torch, dev)
    parity = None
    if results is not None:
        try:
            parity = sample_parity(works, layers, results, rxnn, torch, stream)
        except AssertionError as exc:
            parity = {"FAILED": str(exc)}
        print("[bench] sample parity: %s" % parity, file=sys.stderr, flush=True)
    vmm_us = kern_eval["xbar_vmm"]["us_per_step"]
    ach = 2.0 * macs / (vmm_us * 1e-6) / 1e12
    M, N = layers[0]["L"].M, layers[0]["L"].N
    desc = STACK_DESC[cfg]
    if rebuild:
        desc = desc % (M, N, args.wire, total_arrays,
                       "one rxnn_remap_layer per layer on 8 streams" if args.per_layer_rebuild
                       else "one rxnn_remap_layers call") + device_note(args)
    traffic = STACK_VMM_TRAFFIC.get((cfg, M, args.wire if rebuild else None))
    out = {
        "metric": "non-ideal crossbar MACs/sec per layer",
        "value": macs / (step_ms * 1e-3),
        "unit": "MAC/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": step_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": desc, "alg_macs_per_step": macs, "arrays": total_arrays},
        "roofline": {"kernel": "k_xbar_vmm, summed over the layers of an evaluation-only pass",
                     "bound": "mfma", "achieved": ach, "peak": FP32_MFMA_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": ach / FP32_MFMA_PEAK_TFLOPS,
                     "traffic": traffic, "us_per_pass": vmm_us,
                     "flops_per_pass": 2.0 * macs},
        "eval_only": {"what": "VMM only: DAC, V.G', ADC, accumulation of every layer, G' kept",
                      "ms": eval_ms, "value": macs / (eval_ms * 1e-3), "unit": "MAC/s",
                      "kernels": kern_eval},
        "hbm": hbm,
        "wall_s_timed": wall,
    }
    if kern is not None:
        out["kernels"] = kern
    if rebuild:
        b_flops = sum(e["L"].R * e["L"].C * e["L"].A for e in layers) * build_flops(M, N)
        b_ach = b_flops / (map_ms * 1e-3) / 1e12
        out["map_only"] = {"what": "G' rebuild of every array (w_max + fp64 build)"
                                   + (", one rxnn_remap_layer per layer on 8 streams"
                                      if args.per_layer_rebuild else
                                      ", all layers in one rxnn_remap_layers call"),
                           "ms": map_ms, "per_layer_8_streams_ms": map_pl_ms, "fp64_flops": b_flops, "achieved": b_ach,
                           "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
                           "frac": b_ach / FP64_PEAK_TFLOPS,
                           "generation": generation_info(map_ms, total_arrays, M, N)}
    if gen is not None:
        out["generation"] = gen
    if cpu is not None:
        cpu["speedup_gpu_over_oracle"] = out["value"] / cpu["value"]
        out["cpu_baseline"] = cpu
    if parity is not None:
        out["sample_parity"] = parity
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
    # dW = clip(patches)^T dY and dX = dY W^T over the patch columns: 2 Bv P Q
    # multiply-adds each
    leg = {}
    for name in ("bw_dw", "bw_dx"):
        us = kern[name]["us_per_step"]
        ach = 2.0 * bv * L.P * L.Q / (us * 1e-6) / 1e12
        leg[name] = {"us_per_step": us, "bound": "mfma", "achieved": ach,
                     "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / FP32_MFMA_PEAK_TFLOPS, "flops": 2.0 * bv * L.P * L.Q}
    g_us = leg["bw_dw"]["us_per_step"] + leg["bw_dx"]["us_per_step"]
    ach = 4.0 * bv * L.P * L.Q / (g_us * 1e-6) / 1e12
    print("[bench] retrain: %.3f ms/step" % ms, file=sys.stderr, flush=True)
    return {"ms_per_step": ms, "backward": {
        "us_per_step": g_us, "bound": "mfma", "achieved": ach, "peak": FP32_MFMA_PEAK_TFLOPS,
        "unit": "TFLOP/s", "frac": ach / FP32_MFMA_PEAK_TFLOPS, "flops": 4.0 * bv * L.P * L.Q},
        **leg,
        "backward_reduce_us_per_step": kern.get("bw_reduce", {}).get("us_per_step", 0.0),
        "kernels": kern}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 2 GiB copy kernel (counter calibration)")
    ap.add_argument("--workload", default="resnet50",
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
    ap.add_argument("--per-layer-rebuild", action="store_true",
                    help="resnet50: rebuild G' with one rxnn_remap_layer per layer on 8 streams "
                         "instead of one rxnn_remap_layers call")
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

    from paper_1809_00072_amd import workloads as wl

    work = wl.conv3x3_64_56()
    cv, xb, pp = work["conv"], work["xbar"], work["periph"]
    xb = device_options(xb, args)
    if args.divider:
        xb = dict(xb, r_driver=0.0)
        pp = dict(pp, dac_bend=0.0, dac_g_on=DIVIDER_G_ON, dac_g_pd=DIVIDER_G_PD)
    # the oracle first, before the GPU is touched (its worker processes fork
    # from this one)
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline_conv(dict(work, xbar=xb, periph=pp))

    import torch
    from paper_1809_00072_amd import rxnn
    rxnn.load()
    assert torch.cuda.is_available(), "bench.py needs the HIP device"
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
    hbm = {}
    for name in ("dac", "finish"):
        tot_ms, cnt = rxnn.profile_read(name)
        if cnt:
            gbs = rxnn.profile_bytes(name) / (tot_ms * 1e-3) / 1e9
            hbm[name] = {"us_per_step": 1e3 * tot_ms / args.steps,
                         "bytes_per_step": rxnn.profile_bytes(name) / args.steps,
                         "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": gbs / HBM_PEAK_GBS}

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
        "hbm": hbm,
        "ideal_fp32": ideal,
        "kernels": kern,
        "kernels_pass": "a second pass of the same steps with every launch timed",
        "wall_s_timed": wall,
    }
    if retrain is not None:
        out["retrain"] = retrain
    if cpu is not None:
        cpu["speedup_gpu_over_oracle"] = out["value"] / cpu["value"]
        out["cpu_baseline"] = cpu
    L.free()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
