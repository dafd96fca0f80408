"""Comparison rules between the HIP path and the CPU oracle.

* G' per element: relative error <= GP_RTOL (fp64 build rounded to fp32).
* Pre-ADC currents: relative error <= I_RTOL.  V >= 0 and G' >= 0, so no
  cancellation happens inside a current; fp32 accumulation over M <= 64 terms
  stays far below this bound.
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


def array_weights(A, slice_bits):
    w = []
    for a in range(A):
        s, side = divmod(a, 2)
        w.append((-1 if side else 1) * (1 << (slice_bits * s)))
    return np.array(w, dtype=np.int64)
