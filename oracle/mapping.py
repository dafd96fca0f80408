"""Oracle: crossbar model generation, W -> G -> G' (Sec. V-A, Fig. 'mapping').

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Step 1 (tiling).  A P x Q weight matrix needs ceil(P/M) * ceil(Q/N) crossbar
instances.  Tile (r, c) holds ``W[rM:(r+1)M, cN:(c+1)N]`` (0-based).  The
corners are zero-padded; the paper's count of padded rows, "P mod M", is read
as ``(M - P mod M) mod M`` (and likewise for columns).  Padded positions hold
weight 0 and are still physical devices at ``g_min``: they load the network.

Step 2 (W -> G), for a linear device between ``g_min`` and ``g_max``:
* ``w_max`` = max |W| over the layer unless the caller fixes it.
* continuous (``weight_bits == 0``): a differential pair,
  ``G+ = g_min + s_w max(w, 0)``, ``G- = g_min + s_w max(-w, 0)`` with
  ``s_w = (g_max - g_min) / w_max``.
* quantised (``weight_bits > 0``): ``q = min(2^wb - 1, rint(|w| (2^wb - 1) / w_max))``
  (the device precision, Sec. III, is the number of conductance levels).  With
  ``bits_per_slice = s_b > 0`` the magnitude is cut into ``wb / s_b`` slices
  ``d_s = (q >> (s_b s)) & (2^s_b - 1)``, each on its own differential pair:
  the side of the weight's sign gets ``g_min + d_s dG``, the other ``g_min``,
  with ``dG = (g_max - g_min) / (2^s_b - 1)``.  ``bits_per_slice == 0`` means
  one slice of ``weight_bits`` bits.
* Array order at one tile position: ``a = 2 s + side`` (side 0 positive,
  1 negative; slice 0 least significant).  Each array is its own M x N
  crossbar with its own ADCs; the arrays are combined digitally with weight
  ``(+1 | -1) * 2^(s_b s)``.

Device characteristic and variation (optional, ``oracle/variation.py``): with a
table ``g_lut`` the normalised conductance of a level u is ``f(u)`` instead of
u, the level being ``min(max(+-w, 0) / w_max, 1)`` (continuous) or
``d_s / (2^s_b - 1)`` (a slice digit): ``G = g_min + (g_max - g_min) f(u)``.
Every conductance is then multiplied by its device's variation factor: the
caller's ``variation`` array ([C, R, A, M, N]) or, for ``variation_sigma > 0``,
the factors drawn from ``variation_seed``.

Step 3 (G -> G'): ``network.gprime_nodal`` per array, or for arrays above
32 x 32 with positive wire and sense resistances ``network.gprime_rowsweep``
(the same equations, eliminated row by row; the two agree to ~1e-12).

Parity status: tiling and W->G are exact integer/fp64 definitions; pinned by
the recombination identity ``sum_s 2^(s_b s) (G+_s - G-_s) = dG q sign(w)``
and the tile/padding tests in ``tests/test_oracle_fcm.py``.
"""

from __future__ import annotations

import math

import numpy as np

from .network import gprime_nodal, gprime_rowsweep
from .variation import characteristic, device_indices, generated_factors

PARAM_KEYS = ("rows", "cols", "g_min", "g_max", "r_driver", "r_sense", "r_row",
              "r_col", "weight_bits", "bits_per_slice", "w_max", "variation",
              "variation_sigma", "variation_seed", "g_lut")


def tile_grid(P, Q, M, N):
    return math.ceil(P / M), math.ceil(Q / N)


def slicing(params):
    """(n_slices, bits per slice) ; bits per slice is 0 for a continuous device."""
    wb = int(params["weight_bits"])
    if wb == 0:
        return 1, 0
    sb = int(params["bits_per_slice"]) or wb
    if wb % sb:
        raise ValueError("weight_bits must be a multiple of bits_per_slice")
    return wb // sb, sb


def arrays_per_position(params):
    return 2 * slicing(params)[0]


def array_weight(params, a):
    """Digital weight of array ``a`` in the shift-and-add accumulation."""
    s, side = divmod(a, 2)
    _, sb = slicing(params)
    return (-1 if side else 1) * (1 << (sb * s))


def layer_w_max(W, params):
    if params.get("w_max", 0.0) > 0.0:
        return float(params["w_max"])
    return float(np.max(np.abs(np.asarray(W, dtype=np.float32))))


def effective_weight_scale(params, w_max):
    """Conductance difference per unit weight, in siemens: the ideal current
    difference of a differential pair is ``s_w' * w * V``."""
    g_min, g_max = float(params["g_min"]), float(params["g_max"])
    wb = int(params["weight_bits"])
    if wb == 0:
        return (g_max - g_min) / w_max
    _, sb = slicing(params)
    dG = (g_max - g_min) / ((1 << sb) - 1)
    return dG * ((1 << wb) - 1) / w_max


def tile_weights(W, params, r, c):
    """The M x N fragment of tile (r, c), zero-padded (step 1)."""
    W = np.asarray(W, dtype=np.float32)
    P, Q = W.shape
    M, N = int(params["rows"]), int(params["cols"])
    frag = np.zeros((M, N), dtype=np.float32)
    p0, q0 = r * M, c * N
    p1, q1 = min(P, p0 + M), min(Q, q0 + N)
    frag[: p1 - p0, : q1 - q0] = W[p0:p1, q0:q1]
    return frag


def array_conductances(frag, params, w_max, vf=None):
    """Step 2 for one tile fragment: conductances of every array, [A, M, N]
    fp64; ``vf`` ([A, M, N]) the devices' variation factors, or None."""
    g_min, g_max = float(params["g_min"]), float(params["g_max"])
    lut = params.get("g_lut")
    w = frag.astype(np.float64)
    ns, sb = slicing(params)
    A = 2 * ns
    out = np.empty((A,) + frag.shape, dtype=np.float64)
    if sb == 0:
        if lut is None:
            s_w = (g_max - g_min) / w_max
            out[0] = g_min + s_w * np.maximum(w, 0.0)
            out[1] = g_min + s_w * np.maximum(-w, 0.0)
        else:
            for side, mag in ((0, np.maximum(w, 0.0)), (1, np.maximum(-w, 0.0))):
                u = np.minimum(mag / w_max, 1.0)
                out[side] = g_min + (g_max - g_min) * characteristic(u, lut)
    else:
        wb = int(params["weight_bits"])
        qmax = (1 << wb) - 1
        q = np.minimum(float(qmax), np.rint(np.abs(w) * (qmax / w_max))).astype(np.int64)
        levels = (1 << sb) - 1
        dG = (g_max - g_min) / levels
        for s in range(ns):
            d = (q >> (sb * s)) & levels
            if lut is None:
                on = g_min + d.astype(np.float64) * dG
            else:
                on = g_min + (g_max - g_min) * characteristic(d / levels, lut)
            out[2 * s] = np.where(w > 0, on, g_min)
            out[2 * s + 1] = np.where(w < 0, on, g_min)
    if vf is not None:
        out = out * np.asarray(vf, dtype=np.float64)
    return out


def variation_factors(params, r, c, R, A, M, N):
    """[A, M, N] variation factors of tile (r, c), or None."""
    var = params.get("variation")
    if var is not None:
        return np.asarray(var, dtype=np.float64)[c, r]
    sigma = float(params.get("variation_sigma", 0.0) or 0.0)
    if sigma > 0.0:
        d = device_indices((c * R + r) * A, A, M, N)
        return generated_factors(d, int(params.get("variation_seed", 0)), sigma)
    return None


def array_gprime(G, params):
    """Step 3 for one array: the nodal solve, or the row sweep for large
    arrays whose wire and sense resistances are positive."""
    res = (params["r_driver"], params["r_sense"], params["r_row"], params["r_col"])
    sweep_ok = params["r_row"] > 0 and params["r_col"] > 0 and params["r_sense"] > 0
    if sweep_ok and G.shape[0] * G.shape[1] > 32 * 32:
        return gprime_rowsweep(G, *res)
    return gprime_nodal(G, *res)


def map_layer(W, params, col_tiles=None, row_tiles=None):
    """Model generation for one layer (steps 1-3).

    Returns a dict with ``gp[(r, c)]`` = [A, M, N] fp64 G' for each requested
    tile (all tiles by default) and the layer's scalars.
    """
    W = np.asarray(W, dtype=np.float32)
    P, Q = W.shape
    M, N = int(params["rows"]), int(params["cols"])
    R, C = tile_grid(P, Q, M, N)
    w_max = layer_w_max(W, params)
    cols = range(C) if col_tiles is None else col_tiles
    rows = range(R) if row_tiles is None else row_tiles
    gp = {}
    A = arrays_per_position(params)
    for c in cols:
        for r in rows:
            vf = variation_factors(params, r, c, R, A, M, N)
            G = array_conductances(tile_weights(W, params, r, c), params, w_max, vf)
            gp[(r, c)] = np.stack([array_gprime(G[a], params) for a in range(G.shape[0])])
    return {"gp": gp, "P": P, "Q": Q, "M": M, "N": N, "R": R, "C": C,
            "A": arrays_per_position(params), "w_max": w_max,
            "s_w_eff": effective_weight_scale(params, w_max)}
