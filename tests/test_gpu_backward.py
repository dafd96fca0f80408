"""GPU parity of the re-training backward pass (rxnn_fc_backward,
rxnn_conv_backward) against the oracle's fp64 gradients (oracle/backward.py).

Tolerance: both sides read the same fp32 X, W and dY; the GPU forms each
gradient entry as an fp32 sum of k products (k = the contraction length plus,
for a convolution's dX, the kernel taps that meet at a pixel).  Any
summation order keeps |fl(sum) - sum| <= gamma_k sum |a b| with
gamma_k = k u / (1 - k u), u = 2^-24; the tests allow 1.01 k u sum |a b|,
where sum |a b| is the oracle's own gradient of |W|, |clip(X)| and |dY|.
Masked entries (inputs the DAC clips, weights beyond w_max) must be exactly
zero.  Every case prints its name before touching the GPU.
"""

import ctypes

import numpy as np
import pytest

from oracle import backward as ob

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402

U = 2.0 ** -24


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def say(*a):
    print("[case]", *a, flush=True)


def dac_range(pp):
    return float(pp["x_max"]) if pp["dac_bits"] else np.inf


def check(got, want, mag, k, masked):
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == want.shape
    assert np.all(got[masked] == 0.0), "masked gradients must be exactly zero"
    tol = 1.01 * k * U * mag + 1e-37
    err = np.abs(got - want)
    bad = err > tol
    assert not bad.any(), (
        f"{bad.sum()} entries beyond the fp32 bound; worst err {err.max():.3e}, "
        f"tol there {tol.flat[np.argmax(err)]:.3e}")


def fc_inputs(B, P, Q, x_max, seed):
    rng = np.random.default_rng(seed)
    W = rng.normal(0.0, 0.05, size=(P, Q)).astype(np.float32)
    # inputs spanning both ends of the DAC range, with exact edge values
    X = (rng.uniform(-0.25, 1.25, size=(B, P)) * x_max).astype(np.float32)
    if X.size >= 4:
        X.flat[0], X.flat[1] = 0.0, np.float32(x_max)
    dY = rng.normal(0.0, 1.0, size=(B, Q)).astype(np.float32)
    return W, X, dY


def fc_oracle(W, X, dY, x_max, w_max):
    dX, dW = ob.fc_backward(W, X, dY, x_max, w_max)
    Xc = np.clip(X.astype(np.float64), 0.0, x_max)
    mX, _ = ob.fc_backward(np.abs(W), np.zeros_like(X), np.abs(dY), np.inf, np.inf)
    _, mW = ob.fc_backward(W, Xc, np.abs(dY), np.inf, np.inf)
    return dX, dW, mX, np.abs(mW)


@pytest.mark.parametrize("B,P,Q,M,N,dac,w_max", [
    (1, 1, 1, 64, 64, 4, 0.0),
    (37, 300, 70, 64, 64, 4, 0.0),        # ragged everywhere
    (37, 300, 70, 64, 64, 0, 0.0),        # ideal DAC: only negative inputs clipped
    (64, 513, 129, 128, 128, 6, 0.08),    # fixed w_max below max|W|: weight mask
    (256, 1024, 512, 64, 64, 8, 0.0),
    (2048, 64, 32, 64, 64, 4, 0.0),       # dW split over 8 row ranges, then summed
])
def test_fc_backward_parity(B, P, Q, M, N, dac, w_max):
    label = f"fc_backward B={B} P={P} Q={Q} dac={dac} w_max={w_max}"
    x_max = 2.0
    W, X, dY = fc_inputs(B, P, Q, x_max, seed=B + P + Q)
    pp = wl.periph(dac, 8, x_max)
    say(label, "map")
    L = rxnn.map_layer(dev(W), wl.xbar(M, N, 2.5, w_max=w_max))
    wm = L.w_max()
    say(label, "backward")
    Wd, Xd, dYd = dev(W), dev(X), dev(dY)
    dX, dW = rxnn.fc_backward(L, pp, Wd, Xd, dYd)
    dX_only, _ = rxnn.fc_backward(L, pp, Wd, Xd, dYd, want_dw=False)
    _, dW_only = rxnn.fc_backward(L, pp, Wd, Xd, dYd, want_dx=False)
    torch.cuda.synchronize()
    xr = dac_range(pp)
    oX, oW, mX, mW = fc_oracle(W, X, dY, xr, wm)
    check(dX.cpu().numpy(), oX, mX, Q, ~((X >= 0) & (X <= xr)))
    check(dW.cpu().numpy(), oW, mW, B, ~(np.abs(W) <= wm))
    if w_max > 0.0:
        assert (np.abs(W) > wm).any()
    # the partial calls run the same kernels: identical results
    assert torch.equal(dX_only, dX) and torch.equal(dW_only, dW)
    L.free()


def test_fc_backward_noops_and_errors():
    say("fc_backward no-ops and errors")
    W, X, dY = fc_inputs(4, 40, 10, 1.0, seed=5)
    L = rxnn.map_layer(dev(W), wl.xbar(64, 64, 2.5))
    pp = wl.periph(4, 8, 1.0)
    lib = rxnn.load()
    ppc = ctypes.byref(rxnn.periph_params(pp))
    Wd, Xd, dYd = dev(W), dev(X), dev(dY)
    w, x, dy = rxnn._ptr(Wd), rxnn._ptr(Xd), rxnn._ptr(dYd)
    out = torch.full((4, 40), 7.0, device="cuda")
    # B = 0, and dX = dW = NULL, do nothing
    assert lib.rxnn_fc_backward(L.handle, ppc, w, x, dy, 0, rxnn._ptr(out), None,
                                None) == rxnn.RXNN_OK
    assert lib.rxnn_fc_backward(L.handle, ppc, w, x, dy, 4, None, None, None) == rxnn.RXNN_OK
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    assert lib.rxnn_fc_backward(L.handle, ppc, None, x, dy, 4, rxnn._ptr(out), None,
                                None) == rxnn.RXNN_EINVAL
    assert lib.rxnn_fc_backward(L.handle, ppc, w, x, dy, -1, None, None, None) == \
        rxnn.RXNN_EINVAL
    with pytest.raises(rxnn.RxnnError, match="dac_bits"):
        rxnn.fc_backward(L, dict(pp, dac_bits=99), Wd, Xd, dYd)
    L.free()


def conv_inputs(conv, x_max, seed):
    rng = np.random.default_rng(seed)
    c_in, c_out, k = conv["c_in"], conv["c_out"], conv["kh"]
    weight = rng.normal(0.0, np.sqrt(2.0 / (c_in * k * k)), size=(c_out, c_in, k, k))
    W = np.ascontiguousarray(weight.reshape(c_out, -1).T).astype(np.float32)
    X = (rng.uniform(-0.2, 1.2, size=(conv["n"], c_in, conv["h"], conv["w"])) *
         x_max).astype(np.float32)
    X.flat[0], X.flat[1] = 0.0, np.float32(x_max)
    ho, wo = rxnn.conv_out_hw(conv)
    dY = rng.normal(0.0, 1.0, size=(conv["n"], c_out, ho, wo)).astype(np.float32)
    return W, X, dY


def conv_oracle(W, X, dY, conv, x_max, w_max):
    dX, dW = ob.conv_backward(W, X, dY, conv, x_max, w_max)
    Xc = np.clip(X.astype(np.float64), 0.0, x_max)
    mX, _ = ob.conv_backward(np.abs(W), np.zeros_like(X), np.abs(dY), conv, np.inf, np.inf)
    _, mW = ob.conv_backward(W, Xc, np.abs(dY), conv, np.inf, np.inf)
    return dX, dW, mX, np.abs(mW)


def conv_dict(n, c_in, hw, c_out, k, s, p, w=None):
    return {"n": n, "c_in": c_in, "h": hw, "w": hw if w is None else w, "c_out": c_out,
            "kh": k, "kw": k, "stride": s, "pad": p}


@pytest.mark.parametrize("conv,dac,w_max", [
    (conv_dict(2, 3, 9, 5, 3, 1, 1), 4, 0.0),
    (conv_dict(1, 4, 11, 6, 5, 2, 2), 6, 0.0),
    (conv_dict(2, 2, 8, 3, 1, 1, 0), 0, 0.0),          # 1x1, ideal DAC
    (conv_dict(1, 3, 15, 4, 7, 2, 3), 8, 0.0),          # stem-like 7x7 / 2
    (conv_dict(3, 5, 10, 7, 3, 2, 0, w=13), 4, 0.0),    # non-square, no padding
    (conv_dict(4, 64, 28, 64, 3, 1, 1), 6, 0.1),        # several tiles, weight mask
    (conv_dict(2, 128, 14, 256, 3, 2, 1), 8, 0.0),
    (conv_dict(2, 20, 15, 70, 3, 1, 2), 4, 0.0),        # 3x3, odd widths: generic kernels
    (conv_dict(1, 4, 5, 3, 3, 1, 0, w=80), 0, 0.0),     # 3x3 rows wider than a chunk
    (conv_dict(3, 17, 7, 33, 3, 2, 1), 6, 0.0),         # 3x3 / 2 on 7 x 7 images
    (conv_dict(2, 20, 12, 68, 3, 1, 1), 4, 0.0),        # 3x3 halo kernels: ragged c_in, Q
    (conv_dict(2, 17, 16, 33, 3, 2, 1), 6, 0.1),        # 3x3 / 2 halo dW, weight mask
    (conv_dict(1, 8, 8, 12, 3, 1, 1, w=60), 0, 0.0),    # 3x3 halo, ideal DAC, 60-wide rows
    (conv_dict(1, 17, 8, 70, 3, 1, 1), 4, 0.1),         # 3x3 halo dW in one chunk: direct write
    (conv_dict(4, 16, 32, 8, 1, 1, 0), 6, 0.0),         # generic dW split over 16 pixel ranges
])
def test_conv_backward_parity(conv, dac, w_max):
    label = "conv_backward %s dac=%d w_max=%g" % (conv, dac, w_max)
    x_max = 4.0
    W, X, dY = conv_inputs(conv, x_max, seed=conv["c_in"] * 7 + conv["h"])
    pp = wl.periph(dac, 8, x_max)
    say(label, "map")
    L = rxnn.map_layer(dev(W), wl.xbar(64, 64, 2.5, w_max=w_max))
    wm = L.w_max()
    say(label, "backward")
    Wd, Xd, dYd = dev(W), dev(X), dev(dY)
    dX, dW = rxnn.conv_backward(L, pp, conv, Wd, Xd, dYd)
    dX_only, _ = rxnn.conv_backward(L, pp, conv, Wd, Xd, dYd, want_dw=False)
    _, dW_only = rxnn.conv_backward(L, pp, conv, Wd, Xd, dYd, want_dx=False)
    torch.cuda.synchronize()
    xr = dac_range(pp)
    oX, oW, mX, mW = conv_oracle(W, X, dY, conv, xr, wm)
    ho, wo = rxnn.conv_out_hw(conv)
    taps = -(-conv["kh"] // conv["stride"]) * -(-conv["kw"] // conv["stride"])
    check(dX.cpu().numpy(), oX, mX, conv["c_out"] + taps, ~((X >= 0) & (X <= xr)))
    check(dW.cpu().numpy(), oW, mW, conv["n"] * ho * wo, ~(np.abs(W) <= wm))
    assert torch.equal(dX_only, dX) and torch.equal(dW_only, dW)
    L.free()


def test_conv_backward_full_size():
    """The 3x3 64 -> 64 convolution on 32 x 56 x 56 inputs: dW over the whole
    batch, dX on sampled images (an image's dX depends on its own dY only)."""
    work = wl.conv3x3_64_56(32)
    conv, W, X = work["conv"], work["W"], work["X"]
    pp = work["periph"]
    dY = wl.normal(3003, (32, 64, 56, 56), 1.0)
    label = "conv_backward " + work["name"]
    say(label, "map")
    L = rxnn.map_layer(dev(W), work["xbar"])
    wm = L.w_max()
    say(label, "backward")
    dX, dW = rxnn.conv_backward(L, pp, conv, dev(W), dev(X), dev(dY))
    torch.cuda.synchronize()
    dX, dW = dX.cpu().numpy(), dW.cpu().numpy()
    L.free()
    say(label, "oracle dW")
    xr = dac_range(pp)
    _, oW = ob.conv_backward(W, X, dY, conv, xr, wm)
    _, mW = ob.conv_backward(W, np.clip(X.astype(np.float64), 0, xr), np.abs(dY), conv, np.inf,
                             np.inf)
    check(dW, oW, np.abs(mW), 32 * 56 * 56, ~(np.abs(W) <= wm))
    for img in (0, 31):
        say(label, "oracle dX image", img)
        one = dict(conv, n=1)
        oX, _ = ob.conv_backward(W, X[img:img + 1], dY[img:img + 1], one, xr, wm)
        mX, _ = ob.conv_backward(np.abs(W), np.zeros_like(X[:1]), np.abs(dY[img:img + 1]), one,
                                 np.inf, np.inf)
        check(dX[img:img + 1], oX, mX, 64 + 9, ~((X[img:img + 1] >= 0) & (X[img:img + 1] <= xr)))


def test_conv_backward_rejects_mismatch():
    say("conv_backward mismatch")
    conv = conv_dict(1, 3, 8, 4, 3, 1, 1)
    W, X, dY = conv_inputs(conv, 1.0, seed=3)
    L = rxnn.map_layer(dev(W), wl.xbar(64, 64, 2.5))
    lib = rxnn.load()
    ppc = ctypes.byref(rxnn.periph_params(wl.periph(4, 8, 1.0)))
    Wd, Xd, dYd = dev(W), dev(X), dev(dY)
    bad = rxnn.ConvDesc(1, 3, 8, 8, 5, 3, 3, 1, 1)      # c_out 5 on a 27 x 4 layer
    assert lib.rxnn_conv_backward(L.handle, ppc, ctypes.byref(bad), rxnn._ptr(Wd), rxnn._ptr(Xd),
                                  rxnn._ptr(dYd), None, rxnn._ptr(Wd), None) == rxnn.RXNN_EINVAL
    assert "convolution needs" in lib.rxnn_last_error().decode()
    assert lib.rxnn_conv_backward(L.handle, ppc, None, rxnn._ptr(Wd), rxnn._ptr(Xd),
                                  rxnn._ptr(dYd), None, rxnn._ptr(Wd), None) == rxnn.RXNN_EINVAL
    L.free()
