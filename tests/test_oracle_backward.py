"""Pins of the oracle's re-training backward pass (``oracle/backward.py``)."""

import numpy as np
import pytest

from oracle import backward as ob

torch = pytest.importorskip("torch")


def test_fc_matches_torch_linear_gradients():
    rng = np.random.default_rng(1)
    B, P, Q = 5, 7, 4
    W = rng.normal(size=(P, Q))
    X = rng.uniform(0.0, 1.0, size=(B, P))       # all inside [0, x_max]
    dY = rng.normal(size=(B, Q))
    dX, dW = ob.fc_backward(W, X, dY, x_max=1.0, w_max=10.0)
    Wt = torch.tensor(W, requires_grad=True)
    Xt = torch.tensor(X, requires_grad=True)
    (Xt @ Wt).backward(torch.tensor(dY))
    np.testing.assert_allclose(dX, Xt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-12, atol=1e-14)


def test_fc_masks():
    rng = np.random.default_rng(2)
    W = rng.normal(size=(4, 3))
    X = np.array([[-0.5, 0.2, 1.0, 1.7]])
    dY = rng.normal(size=(1, 3))
    dX, dW = ob.fc_backward(W, X, dY, x_max=1.0, w_max=0.8)
    assert dX[0, 0] == 0.0 and dX[0, 3] == 0.0          # clipped by the DAC range
    np.testing.assert_allclose(dX[0, 1:3], (dY @ W.T)[0, 1:3])
    # weights beyond w_max get no gradient; the clipped inputs enter as 0 and x_max
    assert np.all(dW[np.abs(W) > 0.8] == 0.0)
    Xc = np.array([[0.0, 0.2, 1.0, 1.0]])
    keep = np.abs(W) <= 0.8
    np.testing.assert_allclose(dW[keep], (Xc.T @ dY)[keep])


def test_fc_finite_differences():
    """dW is the gradient of the surrogate loss sum(dY * (clip(X) W))."""
    rng = np.random.default_rng(3)
    W = rng.normal(size=(6, 5))
    X = rng.uniform(-0.2, 1.2, size=(4, 6))
    dY = rng.normal(size=(4, 5))
    _, dW = ob.fc_backward(W, X, dY, x_max=1.0, w_max=100.0)
    loss = lambda Wv: float(np.sum(dY * (np.clip(X, 0, 1.0) @ Wv)))
    eps = 1e-6
    for p, q in [(0, 0), (3, 2), (5, 4)]:
        E = np.zeros_like(W)
        E[p, q] = eps
        fd = (loss(W + E) - loss(W - E)) / (2 * eps)
        assert abs(fd - dW[p, q]) < 1e-7


@pytest.mark.parametrize("n,c_in,hw,c_out,k,s,p", [
    (2, 3, 7, 4, 3, 1, 1),
    (1, 2, 9, 3, 3, 2, 0),
    (2, 2, 8, 5, 5, 2, 2),
    (1, 4, 6, 2, 1, 1, 0),
    (1, 1, 11, 2, 7, 2, 3),
])
def test_conv_matches_torch_conv_gradients(n, c_in, hw, c_out, k, s, p):
    rng = np.random.default_rng(n * 10 + c_in)
    weight = rng.normal(size=(c_out, c_in, k, k))
    W = weight.reshape(c_out, -1).T
    X = rng.uniform(0.0, 2.0, size=(n, c_in, hw, hw))       # inside [0, x_max = 2]
    ho = (hw + 2 * p - k) // s + 1
    dY = rng.normal(size=(n, c_out, ho, ho))
    conv = {"n": n, "c_in": c_in, "h": hw, "w": hw, "c_out": c_out, "kh": k, "kw": k,
            "stride": s, "pad": p}
    dX, dW = ob.conv_backward(W, X, dY, conv, x_max=2.0, w_max=100.0)
    Xt = torch.tensor(X, requires_grad=True)
    Wt = torch.tensor(weight, requires_grad=True)
    torch.nn.functional.conv2d(Xt, Wt, stride=s, padding=p).backward(torch.tensor(dY))
    np.testing.assert_allclose(dX, Xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy().reshape(c_out, -1).T, rtol=1e-10, atol=1e-12)


def test_conv_masks():
    rng = np.random.default_rng(5)
    weight = rng.normal(size=(2, 2, 3, 3))
    W = weight.reshape(2, -1).T
    X = rng.uniform(-1.0, 3.0, size=(1, 2, 6, 6))
    dY = rng.normal(size=(1, 2, 6, 6))
    conv = {"n": 1, "c_in": 2, "h": 6, "w": 6, "c_out": 2, "kh": 3, "kw": 3, "stride": 1,
            "pad": 1}
    dX, dW = ob.conv_backward(W, X, dY, conv, x_max=2.0, w_max=0.9)
    assert np.all(dX[(X < 0) | (X > 2.0)] == 0.0)
    assert np.all(dW[np.abs(W) > 0.9] == 0.0)
    # with the clipped input, the unmasked entries are torch's gradients
    Xt = torch.tensor(np.clip(X, 0, 2.0), requires_grad=True)
    Wt = torch.tensor(weight, requires_grad=True)
    torch.nn.functional.conv2d(Xt, Wt, padding=1).backward(torch.tensor(dY))
    keep = (X >= 0) & (X <= 2.0)
    np.testing.assert_allclose(dX[keep], Xt.grad.numpy()[keep], rtol=1e-10, atol=1e-12)
    wk = np.abs(W) <= 0.9
    np.testing.assert_allclose(dW[wk], Wt.grad.numpy().reshape(2, -1).T[wk], rtol=1e-10,
                               atol=1e-12)
