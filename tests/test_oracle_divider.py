"""Pins of the oracle's load-dependent divider DAC (``oracle/periph.py``,
``oracle/fcm.py``).

The exactness pin: a one-row array has no other rows for current to leave
through, so the row sum of its driver-free G' is exactly the conductance the
DAC sees.  Driving that row with the divider's Thevenin equivalent (source
V_DD g / (g + g_PD) behind 1 / (g + g_PD)) through the independent nodal solver
must then give the divider formula's currents, wires and sense resistor
included.
"""

import numpy as np
import pytest

from oracle import fcm as ofcm
from oracle import mapping as omap
from oracle import network as nw
from oracle import periph as pp

PERIPH = {"dac_bits": 4, "x_max": 1.0, "v_read": 0.2, "dac_bend": 0.0, "adc_bits": 0,
          "adc_bend": 0.0, "dac_g_on": 5e-3, "dac_g_pd": 5e-4}


def thevenin(code, periph):
    L = (1 << periph["dac_bits"]) - 1
    g = code / L * periph["dac_g_on"]
    g_th = g + periph["dac_g_pd"]
    return pp.divider_vdd(periph) * g / g_th, 1.0 / g_th


@pytest.mark.parametrize("N,wire,sense", [(1, 0.0, 0.0), (5, 2.5, 1000.0), (16, 10.0, 500.0)])
def test_one_row_matches_thevenin_network(N, wire, sense):
    rng = np.random.default_rng(N)
    G = rng.uniform(5e-6, 50e-6, size=(1, N))
    Gp = nw.gprime_nodal(G, 0.0, sense, wire, wire)        # no driver resistance
    for code in range(16):
        V = pp.divider_voltages(np.array([code]), Gp.sum(axis=1), PERIPH)
        I_div = V[0] * Gp[0]
        v_th, r_th = thevenin(code, PERIPH)
        I_net = v_th * nw.gprime_nodal(G, r_th, sense, wire, wire)[0]
        np.testing.assert_allclose(I_div, I_net, rtol=1e-11, atol=1e-22)


def test_unloaded_full_scale_and_zero():
    L = 15
    V = pp.divider_voltages(np.array([0, L]), np.zeros(2), PERIPH)
    assert V[0] == 0.0
    assert abs(V[1] - PERIPH["v_read"]) < 1e-15
    # any load draws the output below the unloaded value by the divider ratio
    gl = 1e-3
    g_on, g_pd = PERIPH["dac_g_on"], PERIPH["dac_g_pd"]
    Vl = pp.divider_voltages(np.array([L]), np.array([gl]), PERIPH)[0]
    assert abs(Vl / V[1] - (g_on + g_pd) / (g_on + g_pd + gl)) < 1e-14


def test_monotone_in_code_and_load():
    codes = np.arange(16)
    for gl in (0.0, 3.125e-5, 3.125e-4, 3e-3):        # the 32 kOhm and 3.2 kOhm loads among them
        V = pp.divider_voltages(codes, np.full(16, gl), PERIPH)
        assert np.all(np.diff(V) > 0)
    loads = np.array([0.0, 1e-5, 1e-4, 1e-3, 1e-2])
    V = pp.divider_voltages(np.full(5, 9), loads, PERIPH)
    assert np.all(np.diff(V) < 0)


def test_fc_path_with_one_row_crossbars_is_exact():
    """A layer on 1 x N crossbars: every array's currents from the fcm path
    equal the Thevenin network of that array for every input's code."""
    rng = np.random.default_rng(7)
    P, Q, N = 3, 5, 4
    W = rng.normal(0, 0.05, size=(P, Q)).astype(np.float32)
    X = rng.random(size=(6, P)).astype(np.float32)
    X[0, 0] = 0.0
    params = {"rows": 1, "cols": N, "g_min": 5e-6, "g_max": 50e-6, "r_driver": 0.0,
              "r_sense": 800.0, "r_row": 3.0, "r_col": 3.0, "weight_bits": 0,
              "bits_per_slice": 0, "w_max": 0.0}
    lay = omap.map_layer(W, params)
    _, dbg = ofcm.crossbar_vmm(X, lay, params, PERIPH, debug=True)
    codes = pp.dac_codes(X, PERIPH["dac_bits"], PERIPH["x_max"])
    w_max = omap.layer_w_max(W, params)
    for (r, c, a), (I, _) in dbg.items():
        G = omap.array_conductances(omap.tile_weights(W, params, r, c), params, w_max)[a]
        for b in range(X.shape[0]):
            v_th, r_th = thevenin(int(codes[b, r]), PERIPH)
            want = v_th * nw.gprime_nodal(G, r_th, 800.0, 3.0, 3.0)[0]
            np.testing.assert_allclose(I[b], want, rtol=1e-11, atol=1e-22)


def test_divider_needs_driver_free_mapping():
    W = np.ones((2, 2), dtype=np.float32)
    params = {"rows": 2, "cols": 2, "g_min": 5e-6, "g_max": 50e-6, "r_driver": 1000.0,
              "r_sense": 0.0, "r_row": 0.0, "r_col": 0.0, "weight_bits": 0,
              "bits_per_slice": 0, "w_max": 0.0}
    lay = omap.map_layer(W, params)
    with pytest.raises(AssertionError, match="driver"):
        ofcm.crossbar_vmm(np.ones((1, 2), np.float32), lay, params, PERIPH)
