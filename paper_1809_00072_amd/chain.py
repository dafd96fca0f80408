"""A whole ResNet-18 shaped network evaluated layer after layer on crossbars.

Every convolution and the classifier run through the crossbar path
(``rxnn.conv_layer`` / ``rxnn.crossbar_vmm``: DAC, V.G', ADC, accumulation on
the layer's mapped arrays); the digital glue between them (ReLU, the stem's
3x3 stride-2 max pool, the residual additions and the global average pool) is
ordinary tensor arithmetic in torch, as in the DNN framework the crossbar model
plugs into (Sec. VI).  Each layer's DAC range is the exact maximum of its
input.  No BatchNorm: the weights are random.
"""

from __future__ import annotations

from . import rxnn
from . import workloads as wl


def resnet18_forward(layers, specs, X, dac_bits=8, adc_bits=8, record=None, stream=None):
    """Forward pass of the ResNet-18 shaped stack.

    layers  mapped ``rxnn.Layer`` objects, one per entry of ``specs``
            (``workloads.resnet18_layers()`` order);
    X       device fp32 NCHW input (n x 3 x 224 x 224);
    record  optional list: receives (layer index, input, periph, output) of
            every crossbar layer, inputs and outputs as device tensors.
    Returns the classifier's outputs (n x 1000)."""
    import torch
    F = torch.nn.functional
    net = wl.resnet18_blocks()
    n = X.shape[0]

    def layer(l, x):
        pp = wl.periph(dac_bits, adc_bits, float(x.max()))
        spec = specs[l]
        if spec["kind"] == "conv":
            y = rxnn.conv_layer(layers[l], pp, wl.conv_desc(spec, n), x.contiguous(),
                                stream=stream)
        else:
            y = rxnn.crossbar_vmm(layers[l], pp, x.contiguous(), stream=stream)
        if record is not None:
            record.append((l, x, pp, y))
        return y

    x = F.max_pool2d(torch.relu(layer(net["stem"], X)), 3, stride=2, padding=1)
    for c1, c2, ds in net["blocks"]:
        h = layer(c2, torch.relu(layer(c1, x)))
        x = torch.relu(h + (layer(ds, x) if ds is not None else x))
    x = torch.flatten(F.adaptive_avg_pool2d(x, 1), 1)
    return layer(net["fc"], x)


def resnet18_ideal(Ws, specs, X):
    """The same network with ideal fp32 layers (the weights themselves, no
    crossbar): the reference for the end-to-end effect of the non-idealities."""
    import torch
    F = torch.nn.functional
    net = wl.resnet18_blocks()

    def layer(l, x):
        spec, W = specs[l], Ws[l]
        if spec["kind"] == "conv":
            k = spec["k"]
            w = W.t().contiguous().view(spec["c_out"], spec["c_in"], k, k)
            return F.conv2d(x, w, stride=spec["stride"], padding=spec["pad"])
        return x @ W

    x = F.max_pool2d(torch.relu(layer(net["stem"], X)), 3, stride=2, padding=1)
    for c1, c2, ds in net["blocks"]:
        h = layer(c2, torch.relu(layer(c1, x)))
        x = torch.relu(h + (layer(ds, x) if ds is not None else x))
    x = torch.flatten(F.adaptive_avg_pool2d(x, 1), 1)
    return layer(net["fc"], x)
