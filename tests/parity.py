"""Comparison rules between the HIP path and the CPU oracle.

* G' per element: relative error <= GP_RTOL (fp64 build rounded to fp32).
* Pre-ADC currents: relative error <= I_RTOL.  V >= 0 and G' >= 0, so no
  cancellation happens inside a current; fp32 accumulation over M <= 256
  terms (worst case about M 2^-24 = 1.5e-5) stays below this bound.
* ADC codes: identical, except a fraction <= FLIP_FRAC of codes that differ
  by exactly one, and only where the oracle current lies within I_RTOL of the
  threshold separating the two codes (fp32 rounding of a current that sits on
  a threshold).
* Layer outputs: the GPU output equals fp32(integer sum of its own codes) *
  scale exactly, and equals the oracle output exactly wherever no code that
  contributes to it flipped.
"""

from __future__ import annotations

import numpy as np

GP_RTOL = 2e-6
I_RTOL = 1e-4
FLIP_FRAC = 1e-3


def check_gprime(gp_gpu, gp_oracle, rtol=GP_RTOL):
    gp_gpu = np.asarray(gp_gpu, dtype=np.float64)
    err = np.abs(gp_gpu - gp_oracle) / np.abs(gp_oracle)
    assert np.all(np.isfinite(gp_gpu))
    worst = float(err.max())
    assert worst <= rtol, f"G' relative error {worst:.3g} > {rtol}"
    return worst


def check_currents(I_gpu, I_oracle, rtol=I_RTOL):
    I_gpu = np.asarray(I_gpu, dtype=np.float64)
    scale = np.abs(I_oracle)
    err = np.abs(I_gpu - I_oracle)
    floor = 1e-30
    ok = err <= rtol * scale + floor
    worst = float((err / np.maximum(scale, floor)).max()) if err.size else 0.0
    assert ok.all(), f"current relative error {worst:.3g} > {rtol}"
    return worst


def check_codes(codes_gpu, codes_oracle, I_oracle, thresholds, max_frac=FLIP_FRAC,
                rtol=I_RTOL):
    """Returns the boolean mask of flipped codes."""
    codes_gpu = np.asarray(codes_gpu, dtype=np.int64)
    codes_oracle = np.asarray(codes_oracle, dtype=np.int64)
    d = codes_gpu - codes_oracle
    flip = d != 0
    n = int(flip.sum())
    if n:
        assert np.all(np.abs(d[flip]) == 1), "an ADC code differs by more than one"
        k = np.maximum(codes_gpu, codes_oracle)[flip]        # separating threshold t_k
        t = np.asarray(thresholds, dtype=np.float64)[k - 1]
        I = I_oracle[flip]
        assert np.all(np.abs(I - t) <= rtol * np.abs(I)), \
            "a flipped code is not at a threshold"
    frac = n / max(codes_oracle.size, 1)
    assert frac <= max_frac, f"{frac:.3g} of codes flipped"
    return flip


def check_outputs_by_codes(Y_gpu, dbg, weights, thresholds, scale,
                           max_frac=FLIP_FRAC, rtol=I_RTOL):
    """Layer outputs of the production path against the oracle's per-array
    currents and codes (``dbg`` = {(r, a): (I [S, n], code [S, n])} for the
    sampled outputs).

    The GPU output is fp32(acc) * scale with an integer acc, so acc is read
    back exactly.  acc_gpu - acc_oracle must be explained by codes at a
    threshold: its magnitude is at most the summed |weight| of the oracle
    codes whose current lies within rtol of a threshold.  Every nonzero
    difference needs at least one flip, so their count must stay within
    max_frac of the codes behind the sample."""
    Y_gpu = np.asarray(Y_gpu, dtype=np.float32)
    t = np.asarray(thresholds, dtype=np.float64)
    acc_o = 0
    slack = 0
    n_codes = 0
    for (r, a), (I, code) in dbg.items():
        acc_o = acc_o + weights[a] * code.astype(np.int64)
        k = np.clip(np.searchsorted(t, I), 1, len(t) - 1)      # nearest thresholds
        near = np.minimum(np.abs(I - t[k - 1]), np.abs(I - t[k])) <= rtol * np.abs(I)
        slack = slack + abs(int(weights[a])) * near
        n_codes += I.size
    acc_g = np.rint(Y_gpu.astype(np.float64) / float(scale)).astype(np.int64)
    assert np.array_equal((acc_g.astype(np.float32) * np.float32(scale)), Y_gpu), \
        "GPU output is not fp32(integer) * scale"
    d = acc_g - acc_o
    assert np.all(np.abs(d) <= slack), "an output differs by more than its threshold codes allow"
    n_diff = int(np.count_nonzero(d))
    assert n_diff <= max_frac * n_codes, f"{n_diff} differing outputs for {n_codes} codes"
    return n_diff, n_codes


def array_weights(A, slice_bits):
    w = []
    for a in range(A):
        s, side = divmod(a, 2)
        w.append((-1 if side else 1) * (1 << (slice_bits * s)))
    return np.array(w, dtype=np.int64)
