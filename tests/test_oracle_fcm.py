"""Pins of the mapping and evaluation oracle (``oracle/mapping.py``,
``oracle/fcm.py``): the ideal limit (Eq. 1: zero parasitics and ideal
converters give exactly W.x), the bit-slice recombination identity, tiling and
padding, quantisation error bounds, and conv-as-GEMM against a direct
convolution."""

import numpy as np
import pytest
import torch

from oracle import fcm, mapping
from oracle import periph as pp


def params(**kw):
    p = dict(rows=16, cols=16, g_min=5e-6, g_max=5e-5, r_driver=1000.0, r_sense=1000.0,
             r_row=2.5, r_col=2.5, weight_bits=0, bits_per_slice=0, w_max=0.0)
    p.update(kw)
    return p


IDEAL = dict(r_driver=0.0, r_sense=0.0, r_row=0.0, r_col=0.0)
PER_IDEAL = dict(dac_bits=0, x_max=1.0, v_read=0.2, dac_bend=0.1, adc_bits=0, adc_bend=0.05)
# The DAC output is an fp32 voltage (one fp32 multiply by fp32(v_read/x_max)),
# so the ideal limit holds to two fp32 roundings per term.
TOL_V32 = 2.0 ** -23 + 1e-12


def test_tiling_and_padding():
    rng = np.random.default_rng(0)
    W = rng.normal(0, 1, (37, 21)).astype(np.float32)
    p = params(rows=16, cols=8)
    R, C = mapping.tile_grid(37, 21, 16, 8)
    assert (R, C) == (3, 3)
    full = np.zeros((R * 16, C * 8), np.float32)
    for r in range(R):
        for c in range(C):
            full[r * 16:(r + 1) * 16, c * 8:(c + 1) * 8] = mapping.tile_weights(W, p, r, c)
    assert np.array_equal(full[:37, :21], W)
    assert not full[37:, :].any() and not full[:, 21:].any()
    # padded devices sit at g_min on both sides
    G = mapping.array_conductances(mapping.tile_weights(W, p, 2, 2), p, 3.0)
    assert np.all(G[:, 37 - 32:, :] == 5e-6) and np.all(G[:, :, 21 - 16:] == 5e-6)


def test_continuous_pair():
    W = np.array([[0.5, -0.25, 0.0]], np.float32)
    G = mapping.array_conductances(W, params(), 1.0)
    assert np.allclose(G[0] - G[1], 4.5e-5 * W.astype(np.float64), rtol=0, atol=1e-20)
    assert np.all(np.minimum(G[0], G[1]) == 5e-6)


def test_slice_recombination():
    """sum_s 4^s (G+_s - G-_s) = dG * q * sign(w) with q the 8-bit magnitude."""
    rng = np.random.default_rng(1)
    W = rng.normal(0, 0.01, (40, 30)).astype(np.float32)
    p = params(weight_bits=8, bits_per_slice=2)
    w_max = float(np.max(np.abs(W)))
    G = mapping.array_conductances(W, p, w_max)
    assert G.shape == (8, 40, 30)
    dG = (5e-5 - 5e-6) / 3
    rec = sum((4 ** s) * (G[2 * s] - G[2 * s + 1]) for s in range(4))
    q = np.minimum(255, np.rint(np.abs(W.astype(np.float64)) * (255 / w_max)))
    np.testing.assert_allclose(rec, dG * q * np.sign(W), rtol=1e-12, atol=1e-18)
    assert np.max(q) == 255
    assert set(np.unique((G - 5e-6) / dG).round(9)) <= {0.0, 1.0, 2.0, 3.0}


def _ideal_layer(W, **kw):
    p = params(**IDEAL, **kw)
    return p, mapping.map_layer(W, p)


def test_ideal_limit_fc():
    """Eq. 1: an array free of parasitics behind ideal converters computes W.x."""
    rng = np.random.default_rng(2)
    P, Q, B = 45, 37, 5
    W = rng.normal(0, 0.05, (P, Q)).astype(np.float32)
    X = rng.uniform(0, 1, (B, P)).astype(np.float32)
    p, layer = _ideal_layer(W)
    Y = fcm.crossbar_vmm(X, layer, p, PER_IDEAL)
    ref = X.astype(np.float64) @ W.astype(np.float64)
    scale = np.abs(X).astype(np.float64) @ np.abs(W).astype(np.float64)
    assert np.max(np.abs(Y - ref) / scale) < TOL_V32


def test_ideal_limit_sliced():
    rng = np.random.default_rng(3)
    P, Q, B = 40, 20, 4
    W = rng.normal(0, 0.01, (P, Q)).astype(np.float32)
    X = np.abs(rng.normal(0, 1, (B, P))).astype(np.float32)
    p, layer = _ideal_layer(W, weight_bits=8, bits_per_slice=2)
    per = dict(PER_IDEAL, x_max=float(X.max()))
    Y = fcm.crossbar_vmm(X, layer, p, per)
    w_max = float(np.max(np.abs(W)))
    Wq = np.sign(W) * np.minimum(255, np.rint(np.abs(W.astype(np.float64)) * (255 / w_max))) * (w_max / 255)
    ref = X.astype(np.float64) @ Wq
    scale = np.abs(X).astype(np.float64) @ np.abs(Wq)
    assert np.max(np.abs(Y - ref) / scale) < TOL_V32


def test_quantised_error_bound():
    """Unbent 8-bit converters on an ideal array: the error is bounded by the
    DAC's half step on every input and the ADC's half step on every conversion."""
    rng = np.random.default_rng(4)
    P, Q, B = 64, 24, 50
    W = rng.normal(0, 0.05, (P, Q)).astype(np.float32)
    X = rng.uniform(0, 1, (B, P)).astype(np.float32)
    p, layer = _ideal_layer(W)
    per = dict(dac_bits=8, x_max=1.0, v_read=0.2, dac_bend=0.0, adc_bits=8, adc_bend=0.0)
    Y = fcm.crossbar_vmm(X, layer, p, per).astype(np.float64)
    ref = X.astype(np.float64) @ W.astype(np.float64)
    M = p["rows"]
    lsb_y = pp.adc_full_scale(per, M, p["g_max"]) / 255 / (0.2 * layer["s_w_eff"])
    n_conv = 2 * layer["R"]
    bound = (np.abs(W).sum(axis=0) * 0.5 / 255 + n_conv * lsb_y * 0.5) * (1 + 1e-6)
    assert np.all(np.abs(Y - ref) <= bound)


def test_integer_accumulation_is_exact():
    """Layer output = fp32(sum of weighted codes) * scale: rebuild it from the
    per-array codes returned in debug mode."""
    rng = np.random.default_rng(5)
    W = rng.normal(0, 0.05, (40, 20)).astype(np.float32)
    X = rng.uniform(0, 1, (3, 40)).astype(np.float32)
    p = params()
    layer = mapping.map_layer(W, p)
    per = dict(dac_bits=4, x_max=1.0, v_read=0.2, dac_bend=0.1, adc_bits=8, adc_bend=0.05)
    Y, dbg = fcm.crossbar_vmm(X, layer, p, per, debug=True)
    acc = np.zeros((3, layer["C"] * 16), np.int64)
    for (r, c, a), (I, code) in dbg.items():
        acc[:, c * 16:(c + 1) * 16] += (1 if a % 2 == 0 else -1) * code
    scale = pp.output_scale(per, 16, 5e-5, layer["s_w_eff"])
    assert np.array_equal(Y, acc[:, :20].astype(np.float32) * scale)


def _direct_conv(x, w, stride, pad):
    """Plain loops over output pixels: y[n,o,oy,ox] = sum x[n,c,iy,ix] w[o,c,ky,kx]."""
    n, ci, h, wd = x.shape
    co, _, kh, kw = w.shape
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    xp = np.zeros((n, ci, h + 2 * pad, wd + 2 * pad))
    xp[:, :, pad:pad + h, pad:pad + wd] = x
    y = np.zeros((n, co, ho, wo))
    for oy in range(ho):
        for ox in range(wo):
            patch = xp[:, :, oy * stride:oy * stride + kh, ox * stride:ox * stride + kw]
            y[:, :, oy, ox] = np.einsum("nckl,ockl->no", patch, w)
    return y


@pytest.mark.parametrize("kh,stride,pad", [(3, 1, 1), (3, 2, 1), (1, 1, 0), (5, 2, 2)])
def test_conv_ideal_limit(kh, stride, pad):
    rng = np.random.default_rng(6)
    conv = dict(n=2, c_in=5, h=9, w=8, c_out=7, kh=kh, kw=kh, stride=stride, pad=pad)
    x = np.abs(rng.normal(0, 1, (2, 5, 9, 8))).astype(np.float32)
    wt = rng.normal(0, 0.2, (7, 5, kh, kh)).astype(np.float32)
    W = wt.reshape(7, -1).T.copy()
    p, layer = _ideal_layer(W)
    per = dict(PER_IDEAL, x_max=float(x.max()))
    y = fcm.conv_layer(x, layer, p, per, conv)
    ref = _direct_conv(x.astype(np.float64), wt.astype(np.float64), stride, pad)
    ref_t = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(wt).double(),
                                       stride=stride, padding=pad).numpy()
    np.testing.assert_allclose(ref, ref_t, rtol=1e-12, atol=1e-12)
    scale = _direct_conv(np.abs(x).astype(np.float64), np.abs(wt).astype(np.float64), stride, pad)
    assert np.max(np.abs(y - ref) / np.maximum(scale, 1e-30)) < TOL_V32


def test_im2col_order():
    conv = dict(n=1, c_in=2, h=3, w=3, c_out=1, kh=2, kw=2, stride=1, pad=0)
    x = np.arange(18, dtype=np.float32).reshape(1, 2, 3, 3)
    cols = fcm.im2col(x, conv)
    assert cols.shape == (4, 8)
    # row 1 is output pixel (0, 1); column k = (c*kh + ky)*kw + kx
    assert cols[1].tolist() == [1, 2, 4, 5, 10, 11, 13, 14]
