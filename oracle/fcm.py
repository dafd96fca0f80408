"""Oracle: the FCM evaluation phase of one layer (Sec. V-A 'Peripheral models',
Eq. 14, Sec. VI).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

For every tile (r, c) and array a of the layer:

1. DAC: the layer inputs of row tile r become row voltages
   (``periph.dac_voltages``); padded rows carry 0 V.  With the load-dependent
   divider DAC the inputs become codes, and every array turns them into its
   own row voltages from its rows' loads, the row sums of its G'
   (``periph.divider_voltages``); the layer must then be mapped without a
   driver resistance.
2. Crossbar: ``I = V_r . G'[r, c, a]`` (Eq. 14), fp64, one matrix product.
3. ADC: ``code = periph.adc_codes(I)``.
4. Digital accumulation across tiles (the tiles are merged back into one layer,
   Sec. V-A; the ADC runs as per-layer post-processing, Sec. VI):
   ``acc[b, q] = sum_r sum_a weight(a) code`` in exact integers, then
   ``Y = fp32(acc) * scale_out`` with one fp32 multiply.  With the ideal ADC the
   currents themselves are accumulated in fp64 and scaled by
   ``1 / (s_v s_w')``.

Convolution is evaluated as a matrix product over unrolled patches (Caffe's
conv-as-GEMM, Sec. VI): patch column ``k = (ci * kh + ky) * kw + kx`` (the
order of ``weight.reshape(c_out, -1)``), patch row
``bv = (n * H_out + oy) * W_out + ox``; padded pixels are 0; output NCHW.

Parity status: pinned by the ideal-limit test (zero parasitics, ideal DAC/ADC,
continuous device give exactly W.x) and by a direct-convolution loop in
``tests/test_oracle_fcm.py``.
"""

from __future__ import annotations

import numpy as np

from . import periph as pp
from .mapping import array_weight


def crossbar_vmm(X, layer, params, periph, rows=None, col_tiles=None, debug=False,
                 row_tiles=None):
    """Evaluate one FC layer.  X is [B, P] fp32; returns Y [len(rows), Q].

    Only the column tiles in ``col_tiles`` (default: all) are computed; other
    output columns are NaN.  ``layer`` comes from ``mapping.map_layer`` and must
    hold G' for every row tile of those column tiles.
    ``row_tiles`` (default: all) restricts the evaluation to inputs that are
    zero outside those row tiles: every other row tile then carries V = 0,
    hence I = 0 and code 0 (the first threshold is positive), and adds
    nothing; this is checked, and their G' is not needed.
    With ``debug`` also returns {(r, c, a): (I fp64, codes)}.
    """
    X = np.asarray(X, dtype=np.float32)
    if rows is not None:
        X = X[np.asarray(rows)]
    B, P = X.shape
    M, N, R, C, A, Q = (layer[k] for k in ("M", "N", "R", "C", "A", "Q"))
    assert P == layer["P"]
    divider = pp.divider_dac(periph)
    V = np.zeros((B, R * M), dtype=np.float64)
    if divider:
        assert float(params["r_driver"]) == 0.0, "the divider DAC replaces the driver resistance"
        V[:, :P] = pp.dac_codes(X, int(periph["dac_bits"]), periph["x_max"])
    else:
        V[:, :P] = pp.dac_voltages(X, periph).astype(np.float64)
    quant = int(periph["adc_bits"]) > 0
    if quant:
        i_fs = pp.adc_full_scale(periph, M, params["g_max"])
        thr = pp.adc_thresholds(int(periph["adc_bits"]), i_fs, periph["adc_bend"])
        scale = pp.output_scale(periph, M, params["g_max"], layer["s_w_eff"])
    else:
        scale = pp.ideal_output_scale(periph, layer["s_w_eff"])
    Y = np.full((B, Q), np.nan, dtype=np.float32 if quant else np.float64)
    dbg = {}
    if row_tiles is not None:
        if quant:
            assert thr[0] > 0.0
        for r in set(range(R)) - set(row_tiles):
            assert not V[:, r * M:(r + 1) * M].any(), "inputs outside row_tiles must be zero"
    for c in (range(C) if col_tiles is None else col_tiles):
        acc = np.zeros((B, N), dtype=np.int64 if quant else np.float64)
        for r in (range(R) if row_tiles is None else sorted(row_tiles)):
            Vr = V[:, r * M:(r + 1) * M]
            for a in range(A):
                Gp = layer["gp"][(r, c)][a]
                if divider:
                    # Vr holds codes; this array's rows see their own loads
                    I = pp.divider_voltages(Vr, Gp.sum(axis=1), periph) @ Gp
                else:
                    I = Vr @ Gp
                w = array_weight(params, a)
                if quant:
                    code = pp.adc_codes(I, thr)
                    acc += w * code
                else:
                    code = None
                    acc += w * I
                if debug:
                    dbg[(r, c, a)] = (I, code)
        q0, q1 = c * N, min(Q, (c + 1) * N)
        if quant:
            Y[:, q0:q1] = acc[:, : q1 - q0].astype(np.float32) * scale
        else:
            Y[:, q0:q1] = acc[:, : q1 - q0] * scale
    return (Y, dbg) if debug else Y


def conv_out_hw(conv):
    ho = (conv["h"] + 2 * conv["pad"] - conv["kh"]) // conv["stride"] + 1
    wo = (conv["w"] + 2 * conv["pad"] - conv["kw"]) // conv["stride"] + 1
    return ho, wo


def im2col(X, conv, images=None):
    """Unroll NCHW input patches into [n * H_out * W_out, c_in * kh * kw]."""
    X = np.asarray(X, dtype=np.float32)
    if images is not None:
        X = X[np.asarray(images)]
    n, ci, h, w = X.shape
    kh, kw, s, p = conv["kh"], conv["kw"], conv["stride"], conv["pad"]
    ho, wo = conv_out_hw(conv)
    xp = np.zeros((n, ci, h + 2 * p, w + 2 * p), dtype=np.float32)
    xp[:, :, p:p + h, p:p + w] = X
    cols = np.empty((n, ho, wo, ci, kh, kw), dtype=np.float32)
    for ky in range(kh):
        for kx in range(kw):
            patch = xp[:, :, ky:ky + s * (ho - 1) + 1:s, kx:kx + s * (wo - 1) + 1:s]
            cols[:, :, :, :, ky, kx] = patch.transpose(0, 2, 3, 1)
    return cols.reshape(n * ho * wo, ci * kh * kw)


def conv_layer(X, layer, params, periph, conv, images=None, col_tiles=None, row_tiles=None,
               debug=False):
    """Evaluate one conv layer mapped from ``W = weight.reshape(c_out, -1).T``.
    Returns NCHW output for the selected images (and with ``debug`` the
    per-array currents and codes of ``crossbar_vmm`` over the patch rows)."""
    cols = im2col(X, conv, images)
    Y = crossbar_vmm(cols, layer, params, periph, col_tiles=col_tiles, row_tiles=row_tiles,
                     debug=debug)
    if debug:
        Y, dbg = Y
    n = cols.shape[0] // int(np.prod(conv_out_hw(conv)))
    ho, wo = conv_out_hw(conv)
    Y = Y.reshape(n, ho, wo, -1).transpose(0, 3, 1, 2)
    return (Y, dbg) if debug else Y
