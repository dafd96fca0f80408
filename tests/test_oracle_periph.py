"""Pins of the DAC/ADC oracle (``oracle/periph.py``): textbook special cases
(a uniform DAC, a uniform round-half-up quantiser) and breakpoint behaviour.
The bend constants themselves are a reading (parity unpinned)."""

import numpy as np
import pytest

from oracle import periph as pp


@pytest.mark.parametrize("bits", [1, 4, 6, 8])
def test_dac_lut_uniform_when_unbent(bits):
    L = (1 << bits) - 1
    lut = pp.dac_lut(bits, 0.2, 0.0)
    # an unbent DAC is the uniform one: code c -> v_read * c / L
    want = np.array([np.float32(0.2 * (c / L)) for c in range(L + 1)], dtype=np.float32)
    assert np.array_equal(lut, want)


@pytest.mark.parametrize("bits", [4, 6, 8])
def test_dac_lut_shape(bits):
    L = (1 << bits) - 1
    lut = pp.dac_lut(bits, 0.2, 0.1)
    assert lut[0] == 0.0 and lut[-1] == np.float32(0.2)
    assert np.all(np.diff(lut) > 0)                       # monotone
    lin = pp.dac_lut(bits, 0.2, 0.0)
    assert np.all(lut[1:-1] < lin[1:-1])                  # bends below the line
    # the largest sag is beta/4 of full scale, at mid-code
    assert abs(float(np.max(lin - lut)) - 0.2 * 0.1 / 4) < 0.2 * 0.1 / L


def test_dac_codes_rounding_and_clamp():
    # x_max = 15/16 makes s_in = fp32(15 / x_max) = 16 exactly, so x = (k + 1/2) / 16
    # (exact in fp32) gives products that are exact ties
    bits, x_max = 4, 15.0 / 16.0
    s = pp.dac_scale_in(bits, x_max)
    assert s == np.float32(16.0)
    ties = (np.arange(8) + 0.5) / 16.0
    x32 = ties.astype(np.float32)
    assert np.all(x32 * s == np.arange(8) + 0.5)                  # every product is a tie
    codes = pp.dac_codes(x32, bits, x_max)
    assert codes.tolist() == [0, 2, 2, 4, 4, 6, 6, 8]             # ties go to even
    # off-tie products round to nearest
    off = np.array([0.49, 0.51, 1.49, 1.51, 7.2, 7.8], dtype=np.float64) / 16.0
    assert pp.dac_codes(off.astype(np.float32), bits, x_max).tolist() == [0, 1, 1, 2, 7, 8]
    # unipolar clamp
    assert list(pp.dac_codes(np.array([-1.0, 0.0, 1.0, 7.5], np.float32), bits, 1.0)) == [0, 0, 15, 15]


def test_dac_codes_vs_integer_reference():
    rng = np.random.default_rng(1)
    x = rng.uniform(-0.5, 4.5, 100000).astype(np.float32)
    bits, x_max = 6, 4.0
    L = 63
    codes = pp.dac_codes(x, bits, x_max)
    prod = x.astype(np.float64) * np.float64(np.float32(L / x_max))
    # the fp32 product of two fp32 numbers is the exact product rounded once
    prod32 = prod.astype(np.float32).astype(np.float64)
    fl = np.floor(prod32)
    frac = prod32 - fl
    ref = np.where(frac > 0.5, fl + 1, np.where(frac < 0.5, fl, fl + (fl % 2)))
    ref = np.clip(ref, 0, L)
    assert np.array_equal(codes, ref.astype(np.int64))


def test_ideal_dac():
    per = dict(dac_bits=0, x_max=4.0, v_read=0.2, dac_bend=0.1, adc_bits=8, adc_bend=0.0)
    x = np.array([-1.0, 0.0, 1.0, 4.0, 5.0], np.float32)
    v = pp.dac_voltages(x, per)
    assert np.array_equal(v, np.maximum(x, 0) * np.float32(0.05))


@pytest.mark.parametrize("bits", [4, 8])
def test_adc_uniform_when_unbent(bits):
    L = (1 << bits) - 1
    i_fs = 6.4e-4
    thr = pp.adc_thresholds(bits, i_fs, 0.0)
    rng = np.random.default_rng(2)
    I = rng.uniform(-1e-5, 1.2 * i_fs, 200000)
    I32 = I.astype(np.float32).astype(np.float64)
    codes = pp.adc_codes(I, thr)
    # uniform quantiser with step LSB and half-LSB offset, rounding half up
    ref = np.clip(np.floor(I32 / (i_fs / L) + 0.5), 0, L).astype(np.int64)
    # the fp32 rounding of the thresholds can move codes only for currents
    # within a few ulps of a threshold
    diff = codes != ref
    near = np.min(np.abs(I32[:, None] - thr[None, :].astype(np.float64)), axis=1) <= 4 * np.spacing(np.float32(i_fs))
    assert not np.any(diff & ~near)
    assert diff.mean() < 1e-3


@pytest.mark.parametrize("bend", [0.0, 0.05])
def test_adc_breakpoints(bend):
    bits, i_fs = 8, 6.4e-4
    thr = pp.adc_thresholds(bits, i_fs, bend)
    assert np.all(np.diff(thr) > 0)
    k = np.arange(1, len(thr) + 1)
    assert np.array_equal(pp.adc_codes(thr.astype(np.float64), thr), k)        # a tie goes up
    below = np.nextafter(thr, np.float32(-np.inf)).astype(np.float64)
    assert np.array_equal(pp.adc_codes(below, thr), k - 1)
    assert pp.adc_codes(np.array([0.0, -1.0]), thr).tolist() == [0, 0]
    assert pp.adc_codes(np.array([i_fs, 10 * i_fs]), thr).tolist() == [255, 255]


def test_adc_bend_shape():
    thr0 = pp.adc_thresholds(8, 1.0, 0.0)
    thr1 = pp.adc_thresholds(8, 1.0, 0.05)
    assert np.all(thr1 <= thr0)
    assert abs(float(np.max(thr0 - thr1)) - 0.05 / 4) < 1e-3


def test_output_scale():
    """The output scale turns a code count back into units of w x, fixed by the
    physics of one differential pair: a weight w_max on a one-row array with
    ideal input x_max drives v_read (g_max - g_min) more current into the
    positive array than into the negative one.  With g_min = g_max (1 - k / L)
    that difference is exactly k LSBs of the ADC (I_FS = v_read g_max for
    M = 1), so k codes must read back as w_max x_max."""
    L = 255
    for k, w_max, x_max in ((51, 0.3, 2.0), (17, 1.0, 1.0), (200, 0.05, 4.0)):
        g_max = 5e-5
        g_min = g_max * (1.0 - k / L)
        per = dict(dac_bits=8, x_max=x_max, v_read=0.2, dac_bend=0.0, adc_bits=8, adc_bend=0.0)
        s_w = (g_max - g_min) / w_max                    # conductance per unit weight
        lsb = pp.adc_full_scale(per, 1, g_max) / L
        assert abs(0.2 * (g_max - g_min) / lsb - k) < 1e-9 * k
        y = float(np.float32(k) * pp.output_scale(per, 1, g_max, s_w))
        assert abs(y - w_max * x_max) <= 2e-7 * w_max * x_max
