"""GPU parity of the load-dependent divider DAC (the evaluation kernel's
per-array code -> voltage conversion from the rows' loads) against the
oracle, under the parity rules of tests/parity.py: G' per element, pre-ADC
currents within 1e-4 relative, ADC codes exact up to boundary flips, outputs
exact from the codes.  Every case prints its name before touching the GPU.
"""

import ctypes

import numpy as np
import pytest


torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402
from test_gpu_parity import compare_fc_debug, conv_compare, dev, fc_case, say  # noqa: E402

G_ON, G_PD = 5e-3, 5e-4   # 200 ohm full-scale branch, 2 kOhm pull-down


def divider(pp):
    return dict(pp, dac_bend=0.0, dac_g_on=G_ON, dac_g_pd=G_PD)


@pytest.mark.parametrize("P,Q,M,N,B,dac,adc,wb,sb", [
    (130, 70, 32, 32, 24, 6, 8, 0, 0),
    (70, 50, 13, 10, 37, 4, 8, 0, 0),        # sides off the 16-grid: padded rows and columns
    (256, 128, 64, 64, 16, 6, 8, 0, 0),
    (40, 20, 16, 16, 9, 8, 6, 8, 2),         # 8-bit weights in four 2-bit slices
    (130, 70, 32, 32, 24, 6, 0, 0, 0),       # ideal ADC: currents accumulate
    (300, 100, 128, 128, 20, 8, 8, 0, 0),
])
def test_fc_divider_parity(P, Q, M, N, B, dac, adc, wb, sb):
    W, X, xb, pp = fc_case(P, Q, M, N, B, dac=dac, adc=adc, wb=wb, sb=sb, seed=P + B,
                           r_driver=0.0)
    compare_fc_debug(W, X, xb, divider(pp),
                     f"fc divider {(P, Q, M, N, B, dac, adc, wb, sb)}")


def test_conv_divider_small():
    rng = np.random.default_rng(5)
    n, c_in, hw, c_out, k = 2, 5, 9, 7, 3
    weight = rng.normal(0, np.sqrt(2.0 / (c_in * k * k)), size=(c_out, c_in, k, k))
    W = np.ascontiguousarray(weight.reshape(c_out, -1).T).astype(np.float32)
    X = np.minimum(np.abs(rng.normal(size=(n, c_in, hw, hw))), 4.0).astype(np.float32)
    cv = {"n": n, "c_in": c_in, "h": hw, "w": hw, "c_out": c_out, "kh": k, "kw": k,
          "stride": 1, "pad": 1}
    conv_compare(cv, W, X, wl.xbar(16, 16, 2.5, r_driver=0.0), divider(wl.periph(6, 8, 4.0)),
                 label="conv divider small")


def test_conv3x3_64_56_b32_divider_sampled():
    w = wl.conv3x3_64_56()
    xb = dict(w["xbar"], r_driver=0.0)
    conv_compare(w["conv"], w["W"], w["X"], xb, divider(w["periph"]), images=[0, 31],
                 label="conv3x3 64->64 56x56 b32 divider")


def test_divider_loads_follow_remap():
    """After a remap the rows' loads are those of the new G': the evaluation
    equals that of a layer mapped from the new weights, bit for bit."""
    W, X, xb, pp = fc_case(130, 70, 32, 32, 24, dac=6, adc=8, seed=11, r_driver=0.0)
    pd = divider(pp)
    W2 = (W * np.float32(-0.7) + np.float32(0.01)).astype(np.float32)
    say("divider remap")
    L = rxnn.map_layer(dev(W), xb)
    rxnn.crossbar_vmm(L, pd, dev(X))
    rxnn.remap_layer(L, dev(W2))
    Y1 = rxnn.crossbar_vmm(L, pd, dev(X)).cpu().numpy()
    L2 = rxnn.map_layer(dev(W2), xb)
    Y2 = rxnn.crossbar_vmm(L2, pd, dev(X)).cpu().numpy()
    np.testing.assert_array_equal(Y1, Y2)
    L.free()
    L2.free()


def test_divider_rejections():
    W, X, xb, pp = fc_case(40, 20, 16, 16, 4, dac=4, adc=8, seed=2)   # r_driver 1 kOhm
    say("divider rejections")
    L = rxnn.map_layer(dev(W), xb)
    Xd = dev(X)
    with pytest.raises(rxnn.RxnnError, match="r_driver = 0"):
        rxnn.crossbar_vmm(L, divider(pp), Xd)
    for bad, msg in ((dict(divider(pp), dac_bend=0.1), "dac_bend"),
                     (dict(divider(pp), dac_bits=0), "dac_bits > 0"),
                     (dict(divider(pp), dac_g_on=0.0), "dac_g_on > 0"),
                     (dict(divider(pp), dac_g_pd=-1.0), "finite and >= 0"),
                     (dict(divider(pp), dac_g_on=float("nan")), "finite and >= 0")):
        with pytest.raises(rxnn.RxnnError, match=msg):
            rxnn.crossbar_vmm(L, bad, Xd)
    # dac_g_pd = 0 is the static DAC whatever dac_g_on says
    Y0 = rxnn.crossbar_vmm(L, pp, Xd).cpu().numpy()
    Y1 = rxnn.crossbar_vmm(L, dict(pp, dac_g_on=1.0), Xd).cpu().numpy()
    np.testing.assert_array_equal(Y0, Y1)
    assert ctypes.sizeof(rxnn.PeriphParams) == 64
    L.free()
