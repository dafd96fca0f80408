"""Oracle: peripheral (DAC and ADC) models of the evaluation phase.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper models the DAC as a resistive divider whose output depends on the
digital input and on the crossbar's load (Sec. IV-A 'Non-ideal DAC', Sec. V-A
'Peripheral models'), and the ADC as a possibly non-linear current-to-code
converter; both equations sit in a figure that is not available.  The reading
implemented here:

* The load dependence of the DAC output is exact inside G': the driver's
  Thevenin resistance ``r_driver`` is part of the network
  (``network.py``).  With no wire or sense resistance that network gives
  ``V_i = Vin_i / (1 + r_driver sum_j G_ij)``, the divider form.
* The code-dependent part is a static, unipolar transfer curve with a
  quadratic bend: ``c = clamp(rint(fp32(x) * s_in), 0, 2^b - 1)`` where
  ``s_in = fp32((2^b - 1) / x_max)`` and the product is one fp32 multiply
  rounded to nearest-even; ``V = fp32(v_read * phi_beta(c / (2^b - 1)))`` with
  ``phi_beta(u) = u - beta u (1 - u)`` evaluated in fp64.  ``dac_bits == 0`` is
  the ideal DAC ``V = fp32(max(x, 0) * fp32(v_read / x_max))``.
* ADC: ``I_FS = v_read * M * g_max`` (the ideal full-scale current of an
  M-row array), ``L = 2^b - 1`` and thresholds
  ``t_k = fp32(I_FS * phi_gamma((k - 1/2) / L))`` for k = 1..L.  The code is
  ``#{k : I >= t_k}`` -- a tie goes up, saturation at 0 and L is implied --
  decided in fp32: the fp64 current is rounded to fp32 before the comparison,
  the precision the accelerator computes currents in.  ``adc_bits == 0`` is the
  ideal ADC (the current passes through).

* Load-dependent DAC (the divider form of Sec. IV-A and Sec. V-A, selected
  by ``dac_g_pd > 0``): the DAC is a divider between the supply V_DD and
  ground, an input-dependent conductance g(c) to the supply and a fixed
  pull-down g_PD to ground, whose output node drives the row into the load
  G_Load.  Readings: the input-dependent branch is binary weighted,
  ``g(c) = (c / L) g_on``; V_DD is set so that the unloaded DAC reaches v_read
  at full scale, ``V_DD = v_read (g_on + g_PD) / g_on``; and the load of row i
  of an array is that array's row sum of G', ``G_Load,i = sum_j G'_ij``, with
  G' built without a driver resistance (the divider stands in for the
  driver).  Then ``V_i = V_DD g(c_i) / (g(c_i) + g_PD + G_Load,i)`` in fp64,
  per array (each array's rows see their own load).  The code c is the
  quantiser's above; the static bend does not apply.

Parity status: the curve shapes and the constants (v_read, beta, gamma) are
readings, "parity unpinned" against the paper; the functions are pinned to
their textbook special cases (beta = 0 is a uniform DAC, gamma = 0 a uniform
round-half-up quantiser) and to their breakpoints in ``tests/test_oracle_periph.py``.
The divider is pinned against the exact network (a one-row array driven by
the divider's Thevenin equivalent, where the row sum of G' is the exact load)
and its limits in ``tests/test_oracle_divider.py``.
"""

from __future__ import annotations

import numpy as np

PERIPH_KEYS = ("dac_bits", "x_max", "v_read", "dac_bend", "adc_bits", "adc_bend", "dac_g_on",
               "dac_g_pd")


def _phi(u, bend):
    """Quadratic-bend transfer curve on [0, 1]; monotone for 0 <= bend < 1."""
    return u - (bend * u) * (1.0 - u)


def dac_scale_in(dac_bits, x_max):
    return np.float32(((1 << dac_bits) - 1) / float(x_max))


def dac_lut(dac_bits, v_read, dac_bend):
    L = (1 << dac_bits) - 1
    c = np.arange(L + 1, dtype=np.float64)
    return (float(v_read) * _phi(c / L, float(dac_bend))).astype(np.float32)


def dac_codes(X, dac_bits, x_max):
    L = (1 << dac_bits) - 1
    prod = np.asarray(X, dtype=np.float32) * dac_scale_in(dac_bits, x_max)  # fp32 multiply
    return np.clip(np.rint(prod), 0, L).astype(np.int64)


def dac_voltages(X, periph):
    """Row voltages (fp32) produced by the DAC for inputs X."""
    X = np.asarray(X, dtype=np.float32)
    b = int(periph["dac_bits"])
    if b == 0:
        s_v = np.float32(float(periph["v_read"]) / float(periph["x_max"]))
        return np.maximum(X, np.float32(0.0)) * s_v
    lut = dac_lut(b, periph["v_read"], periph["dac_bend"])
    return lut[dac_codes(X, b, periph["x_max"])]


def divider_dac(periph):
    """True when the periph selects the load-dependent divider DAC."""
    return float(periph.get("dac_g_pd", 0.0) or 0.0) > 0.0


def divider_vdd(periph):
    g_on, g_pd = float(periph["dac_g_on"]), float(periph["dac_g_pd"])
    return float(periph["v_read"]) * (g_on + g_pd) / g_on


def divider_voltages(codes, g_load, periph):
    """Row voltages (fp64) of the divider DAC for integer codes [..., M] and
    the rows' loads g_load [M] (siemens)."""
    L = (1 << int(periph["dac_bits"])) - 1
    g = np.asarray(codes, dtype=np.float64) / L * float(periph["dac_g_on"])
    return divider_vdd(periph) * g / (g + float(periph["dac_g_pd"]) +
                                      np.asarray(g_load, dtype=np.float64))


def adc_full_scale(periph, M, g_max):
    return float(periph["v_read"]) * M * float(g_max)


def adc_thresholds(adc_bits, i_fs, adc_bend):
    L = (1 << adc_bits) - 1
    k = np.arange(1, L + 1, dtype=np.float64)
    return (float(i_fs) * _phi((k - 0.5) / L, float(adc_bend))).astype(np.float32)


def adc_codes(I, thresholds):
    """Code = number of thresholds at or below the fp32-rounded current."""
    I32 = np.asarray(I, dtype=np.float64).astype(np.float32)
    return np.searchsorted(thresholds, I32, side="right").astype(np.int64)


def output_scale(periph, M, g_max, s_w_eff):
    """fp32 factor from accumulated ADC codes to layer-output units.

    One code step is ``LSB = I_FS / L`` amperes; one unit of ``w * x`` is
    ``s_v * s_w'`` amperes with ``s_v = v_read / x_max``.
    """
    L = (1 << int(periph["adc_bits"])) - 1
    lsb = adc_full_scale(periph, M, g_max) / L
    s_v = float(periph["v_read"]) / float(periph["x_max"])
    return np.float32(lsb / (s_v * s_w_eff))


def ideal_output_scale(periph, s_w_eff):
    """Factor from accumulated currents (ideal ADC) to layer-output units."""
    s_v = float(periph["v_read"]) / float(periph["x_max"])
    return 1.0 / (s_v * s_w_eff)
