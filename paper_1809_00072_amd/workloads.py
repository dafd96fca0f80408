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
