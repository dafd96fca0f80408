"""Oracle: the backward pass of model-in-the-loop re-training (Sec. VI, the
RxNN framework: its re-training paragraph, and the mapping of layers onto
matrix products).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

RxNN re-trains with a crossbar-based forward pass and a floating-point
backward pass, converting and scaling the data between the two so that
inputs, outputs and weights stay within their range constraints.  Readings
(the paper gives no formulas):

* The backward pass runs through the ideal weights W (fp64 here) with
  straight-through DAC and ADC: the quantisers pass gradients unchanged, but
  the DAC's range [0, x_max] clips its input, so an input outside it gets no
  gradient, and the forward input seen by the weights is clip(x, 0, x_max).
* With the ideal DAC (no quantisation) the range is [0, inf): the DAC only
  drops negative inputs (V = max(x, 0) v_read / x_max), so callers pass
  x_max = inf for it.
* The mapping's range [-w_max, w_max] clips the weights (the quantised
  mapping saturates at L_w), so a weight outside it gets no gradient.
* Fully connected layer, Y = X W (B x P times P x Q):
    dX = (dY W^T) * [0 <= X <= x_max]
    dW = clip(X, 0, x_max)^T dY * [|W| <= w_max]
* Convolution (patch column k = (ci kh + ky) kw + kx, Sec. VI): the same
  with X replaced by the unrolled patches, written out below as direct sums
  over kernel taps (no unrolled matrix).

Parity status: pinned against torch's CPU convolution and linear gradients
(an independent library), against finite differences of the linear surrogate
loss, and by the masks' special cases (tests/test_oracle_backward.py).
"""

from __future__ import annotations

import numpy as np


def fc_backward(W, X, dY, x_max, w_max):
    """dX (B x P) and dW (P x Q), fp64."""
    W = np.asarray(W, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    in_range = (X >= 0.0) & (X <= x_max)
    dX = (dY @ W.T) * in_range
    Xc = np.clip(X, 0.0, x_max)
    dW = (Xc.T @ dY) * (np.abs(W) <= w_max)
    return dX, dW


def conv_backward(W, X, dY, conv, x_max, w_max):
    """dX (NCHW like X) and dW (P x Q, P = c_in kh kw) of a convolution whose
    weight matrix is W[(ci kh + ky) kw + kx][co], fp64, by direct sums over
    the kernel taps."""
    W = np.asarray(W, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    n, c_in, h, w = X.shape
    kh, kw, s, pad = conv["kh"], conv["kw"], conv["stride"], conv["pad"]
    c_out = dY.shape[1]
    ho, wo = dY.shape[2], dY.shape[3]
    Wt = W.reshape(c_in, kh, kw, c_out)
    Xc = np.clip(X, 0.0, x_max)
    Xp = np.zeros((n, c_in, h + 2 * pad, w + 2 * pad))
    Xp[:, :, pad:pad + h, pad:pad + w] = Xc
    dXp = np.zeros_like(Xp)
    dW = np.zeros((c_in, kh, kw, c_out))
    for ky in range(kh):
        for kx in range(kw):
            # the input pixels this tap reads for every output pixel
            ys = slice(ky, ky + s * (ho - 1) + 1, s)
            xs = slice(kx, kx + s * (wo - 1) + 1, s)
            patch = Xp[:, :, ys, xs]                           # n, c_in, ho, wo
            dW[:, ky, kx, :] = np.einsum("nchw,nohw->co", patch, dY)
            dXp[:, :, ys, xs] += np.einsum("nohw,co->nchw", dY, Wt[:, ky, kx, :])
    in_range = (X >= 0.0) & (X <= x_max)
    dX = dXp[:, :, pad:pad + h, pad:pad + w] * in_range
    dW = dW.reshape(c_in * kh * kw, c_out) * (np.abs(W) <= w_max)
    return dX, dW
