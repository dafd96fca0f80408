"""Seeded synthetic workloads shaped like the layers RxNN evaluates.

This module only draws inputs and states parameters; it holds none of the
crossbar model's arithmetic, so the HIP path and the CPU oracle can both be
fed from it.  Every draw is numpy ``default_rng(seed)`` in fp64, cast to fp32.
The layer shapes stand in for the paper's benchmark networks (Sec. VII): no
dataset content is used.

Parameters that the paper's text does not print (its parameter table is a
figure) are readings: conductance range [5 uS, 50 uS], 1 kOhm driver and sense
resistances, wire resistance per segment as named per workload, DAC/ADC curves
with v_read = 0.2 V (the input level of the sneak-path example, Sec. IV-A),
DAC bend 0.1, ADC bend 0.05.
"""

from __future__ import annotations

import numpy as np

G_MIN, G_MAX = 5e-6, 50e-6
R_DRIVER, R_SENSE = 1000.0, 1000.0
V_READ, DAC_BEND, ADC_BEND = 0.2, 0.1, 0.05


def xbar(rows, cols, wire, weight_bits=0, bits_per_slice=0, w_max=0.0,
         r_driver=R_DRIVER, r_sense=R_SENSE):
    return {"rows": rows, "cols": cols, "g_min": G_MIN, "g_max": G_MAX,
            "r_driver": r_driver, "r_sense": r_sense, "r_row": wire, "r_col": wire,
            "weight_bits": weight_bits, "bits_per_slice": bits_per_slice, "w_max": w_max}


def periph(dac_bits, adc_bits, x_max, v_read=V_READ, dac_bend=DAC_BEND, adc_bend=ADC_BEND):
    return {"dac_bits": dac_bits, "x_max": float(x_max), "v_read": v_read,
            "dac_bend": dac_bend, "adc_bits": adc_bits, "adc_bend": adc_bend}


def normal(seed, shape, sigma):
    return np.random.default_rng(seed).normal(0.0, sigma, size=shape).astype(np.float32)


def uniform(seed, shape):
    return np.random.default_rng(seed).random(size=shape).astype(np.float32)


def abs_normal_clipped(seed, shape, clip=None):
    x = np.abs(np.random.default_rng(seed).normal(0.0, 1.0, size=shape))
    if clip is not None:
        x = np.minimum(x, clip)
    return x.astype(np.float32)


# ---------------------------------------------------------------------------
# FC 256 -> 128, batch 16, 64 x 64 crossbars (4 x 2 tiles)
# ---------------------------------------------------------------------------

def fc_256x128(batch=16):
    P, Q = 256, 128
    return {
        "name": "fc256x128_b%d_x64" % batch,
        "kind": "fc",
        "W": normal(1001, (P, Q), 0.05),
        "X": uniform(2001, (batch, P)),
        "xbar": xbar(64, 64, 2.5),
        "periph": periph(4, 8, 1.0),
    }


# ---------------------------------------------------------------------------
# Conv 3x3 s1 p1, 64 -> 64 channels, 56 x 56, batch 32, 64 x 64 crossbars
# ---------------------------------------------------------------------------

def conv3x3_64_56(batch=32):
    c_in, c_out, hw = 64, 64, 56
    weight = normal(1002, (c_out, c_in, 3, 3), np.sqrt(2.0 / (c_in * 9)))
    return {
        "name": "conv3x3_64to64_56x56_b%d_x64" % batch,
        "kind": "conv",
        "weight": weight,
        "W": np.ascontiguousarray(weight.reshape(c_out, -1).T),
        "X": abs_normal_clipped(2002, (batch, c_in, hw, hw), 4.0),
        "conv": {"n": batch, "c_in": c_in, "h": hw, "w": hw, "c_out": c_out,
                 "kh": 3, "kw": 3, "stride": 1, "pad": 1},
        "xbar": xbar(64, 64, 2.5),
        "periph": periph(6, 8, 4.0),
    }


def alg_macs(work):
    """Algorithmic crossbar MACs of one evaluation: rows x P x Q x arrays,
    counted without tile padding."""
    W = work["W"]
    P, Q = W.shape
    xb = work["xbar"]
    wb, sb = xb.get("weight_bits", 0), xb.get("bits_per_slice", 0)
    n_slices = 1 if wb == 0 else wb // (sb or wb)
    if work["kind"] == "fc":
        rows = work["X"].shape[0]
    else:
        cv = work["conv"]
        ho = (cv["h"] + 2 * cv["pad"] - cv["kh"]) // cv["stride"] + 1
        wo = (cv["w"] + 2 * cv["pad"] - cv["kw"]) // cv["stride"] + 1
        rows = cv["n"] * ho * wo
    return rows * P * Q * 2 * n_slices


# ---------------------------------------------------------------------------
# Layer stacks shaped like ResNet-18 / ResNet-50 (224 x 224 inputs) and the
# VGG-16 fully connected head.  A layer spec is a dict with kind "conv"
# (c_in, c_out, k, stride, pad, h = w of its input) or "fc" (P, Q).
# ---------------------------------------------------------------------------

def _conv(name, c_in, c_out, k, stride, hw):
    return {"name": name, "kind": "conv", "c_in": c_in, "c_out": c_out, "k": k,
            "stride": stride, "pad": k // 2, "hw": hw}


def resnet18_layers():
    """The 20 convolutions and the classifier of ResNet-18 (basic blocks)."""
    L = [_conv("conv1", 3, 64, 7, 2, 224)]
    c_in, hw = 64, 56
    for stage, width in enumerate((64, 128, 256, 512)):
        for block in range(2):
            stride = 2 if (stage > 0 and block == 0) else 1
            pre = "layer%d.%d" % (stage + 1, block)
            L.append(_conv(pre + ".conv1", c_in, width, 3, stride, hw))
            hw_out = hw // stride
            L.append(_conv(pre + ".conv2", width, width, 3, 1, hw_out))
            if stride != 1 or c_in != width:
                L.append(_conv(pre + ".downsample", c_in, width, 1, stride, hw))
            c_in, hw = width, hw_out
    L.append({"name": "fc", "kind": "fc", "P": 512, "Q": 1000})
    return L


def resnet18_blocks():
    """How the layers of ``resnet18_layers`` connect (the digital glue between
    crossbar layers is not part of the crossbar path; this only names it):
    the stem (conv1, ReLU, 3x3 stride-2 max pool), eight basic blocks
    ``(conv1, conv2, downsample or None)`` as layer indices, each computing
    ReLU(conv2(ReLU(conv1(x))) + shortcut(x)), then a global average pool and
    the classifier."""
    layers = resnet18_layers()
    idx = {spec["name"]: l for l, spec in enumerate(layers)}
    blocks = []
    for stage in range(4):
        for block in range(2):
            pre = "layer%d.%d" % (stage + 1, block)
            blocks.append((idx[pre + ".conv1"], idx[pre + ".conv2"], idx.get(pre + ".downsample")))
    return {"stem": idx["conv1"], "blocks": blocks, "fc": idx["fc"]}


def resnet50_layers():
    """The 53 convolutions and the classifier of ResNet-50 (bottleneck blocks,
    stride on the 3x3 convolution)."""
    L = [_conv("conv1", 3, 64, 7, 2, 224)]
    c_in, hw = 64, 56
    for stage, (width, blocks) in enumerate(((64, 3), (128, 4), (256, 6), (512, 3))):
        for block in range(blocks):
            stride = 2 if (stage > 0 and block == 0) else 1
            pre = "layer%d.%d" % (stage + 1, block)
            L.append(_conv(pre + ".conv1", c_in, width, 1, 1, hw))
            L.append(_conv(pre + ".conv2", width, width, 3, stride, hw))
            hw_out = hw // stride
            L.append(_conv(pre + ".conv3", width, 4 * width, 1, 1, hw_out))
            if block == 0:
                L.append(_conv(pre + ".downsample", c_in, 4 * width, 1, stride, hw))
            c_in, hw = 4 * width, hw_out
    L.append({"name": "fc", "kind": "fc", "P": 2048, "Q": 1000})
    return L


def vgg16_fc_layers():
    return [{"name": "fc%d" % (i + 6), "kind": "fc", "P": P, "Q": Q}
            for i, (P, Q) in enumerate(((25088, 4096), (4096, 4096), (4096, 1000)))]


def layer_shape(spec):
    """(P, Q) of a layer's weight matrix."""
    if spec["kind"] == "fc":
        return spec["P"], spec["Q"]
    return spec["c_in"] * spec["k"] * spec["k"], spec["c_out"]


def conv_desc(spec, batch):
    return {"n": batch, "c_in": spec["c_in"], "h": spec["hw"], "w": spec["hw"],
            "c_out": spec["c_out"], "kh": spec["k"], "kw": spec["k"],
            "stride": spec["stride"], "pad": spec["pad"]}


def he_weight(seed, spec):
    """He-initialised weight as the P x Q crossbar matrix (for a convolution
    the rows follow weight.reshape(c_out, -1): k = (ci kh + ky) kw + kx)."""
    P, Q = layer_shape(spec)
    if spec["kind"] == "fc":
        return normal(seed, (P, Q), np.sqrt(2.0 / P))
    k = spec["k"]
    weight = normal(seed, (spec["c_out"], spec["c_in"], k, k), np.sqrt(2.0 / P))
    return np.ascontiguousarray(weight.reshape(spec["c_out"], -1).T)


def layer_input(seed, spec, batch, first):
    """The layer's input: U[0, 1) for the network input, |N(0, 1)| (a ReLU-like
    activation) for every other layer."""
    if spec["kind"] == "fc":
        shape = (batch, spec["P"])
    else:
        shape = (batch, spec["c_in"], spec["hw"], spec["hw"])
    return uniform(seed, shape) if first else abs_normal_clipped(seed, shape)


def stack_layer(config, l, batch=None, crossbar=None, wire=None):
    """Layer l of a stacked workload, standalone: its weight, its input and the
    crossbar / converter parameters.

    config "resnet18": 128 x 128 crossbars, wire 1 Ohm, 8-bit DAC / ADC,
        batch 64, seeds W 1003 + l, X 2003 + l.
    config "vgg16fc": 64 x 64 crossbars, wire 2.5 Ohm, 8-bit magnitude in four
        2-bit slices, 8-bit DAC / ADC, batch 256, W N(0, 0.01^2), X |N(0, 1)|,
        seeds W 1004 + l, X 2004 + l.
    config "resnet50": crossbar side S (32 / 64 / 128 / 256), wire 1 / 2.5 /
        5 Ohm, 8-bit DAC / ADC, batch 128, seeds W 1005 + l, X 2005 + l.
    x_max is the exact maximum of the layer's input.
    """
    if config == "resnet18":
        spec = resnet18_layers()[l]
        batch = 64 if batch is None else batch
        W = he_weight(1003 + l, spec)
        X = layer_input(2003 + l, spec, batch, l == 0)
        xb = xbar(128, 128, 1.0)
    elif config == "vgg16fc":
        spec = vgg16_fc_layers()[l]
        batch = 256 if batch is None else batch
        W = normal(1004 + l, layer_shape(spec), 0.01)
        X = layer_input(2004 + l, spec, batch, False)
        xb = xbar(64, 64, 2.5, weight_bits=8, bits_per_slice=2)
    elif config == "resnet50":
        spec = resnet50_layers()[l]
        batch = 128 if batch is None else batch
        S = 256 if crossbar is None else crossbar
        W = he_weight(1005 + l, spec)
        X = layer_input(2005 + l, spec, batch, l == 0)
        xb = xbar(S, S, 2.5 if wire is None else wire)
    else:
        raise ValueError(config)
    work = {"name": "%s.%s_b%d" % (config, spec["name"], batch), "kind": spec["kind"],
            "spec": spec, "W": W, "X": X, "xbar": xb,
            "periph": periph(8, 8, float(X.max()))}
    if spec["kind"] == "conv":
        work["conv"] = conv_desc(spec, batch)
    return work


def weight_perturbation(seed_step, W, sigma):
    """The model-in-the-loop update of one step: W + 1e-3 sigma eps_t, with
    eps_t ~ N(0, 1) drawn from seed 3000 + t."""
    eps = np.random.default_rng(seed_step).normal(0.0, 1.0, size=W.shape)
    return (W.astype(np.float64) + 1e-3 * sigma * eps).astype(np.float32)


def stack_alg_macs(config, batch=None):
    """Algorithmic crossbar MACs of one pass over every layer of a stack."""
    layers = {"resnet18": resnet18_layers, "vgg16fc": vgg16_fc_layers,
              "resnet50": resnet50_layers}[config]()
    batch = {"resnet18": 64, "vgg16fc": 256, "resnet50": 128}[config] if batch is None else batch
    arrays = 8 if config == "vgg16fc" else 2
    total = 0
    for spec in layers:
        P, Q = layer_shape(spec)
        if spec["kind"] == "fc":
            rows = batch
        else:
            ho = (spec["hw"] + 2 * spec["pad"] - spec["k"]) // spec["stride"] + 1
            rows = batch * ho * ho
        total += rows * P * Q * arrays
    return total
