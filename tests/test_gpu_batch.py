"""rxnn_remap_layers (the G' rebuild of several layers in one launch
sequence) against rxnn_remap_layer per layer and against the oracle, through
the C ABI.  The batch runs the same elimination on every array, so its G' must
equal the per-layer rebuild bit for bit; the oracle checks a sample of arrays
under the parity rule.  Every case prints its name before touching the GPU."""

import numpy as np
import pytest

from oracle import mapping as omap

from parity import check_gprime

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402


def say(*a):
    print("[case]", *a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def all_gprime(L):
    return [L.gprime(r, c, a) for c in range(L.C) for r in range(L.R) for a in range(L.A)]


def layer_set(S, wire, seed):
    """Layers of one crossbar side: ragged shapes, sliced weights, a fixed
    w_max, generated variation and a device table."""
    rng = np.random.default_rng(seed)
    specs = [((3 * S + 5, 2 * S - 3), {}),
             ((S // 2, S + 7), {"weight_bits": 8, "bits_per_slice": 2}),
             ((2 * S, S), {"w_max": 0.08}),
             ((S + 1, 3), {"variation_sigma": 0.1, "variation_seed": 99}),
             ((70, 2 * S + 1), {"g_lut": [(k / 16.0) ** 0.6 for k in range(17)]})]
    out = []
    for (P, Q), extra in specs:
        xb = dict(wl.xbar(S, S, wire), **extra)
        W0 = rng.normal(0, 0.05, size=(P, Q)).astype(np.float32)
        W1 = rng.normal(0, 0.05, size=(P, Q)).astype(np.float32)
        out.append((xb, W0, W1))
    return out


@pytest.mark.parametrize("S,wire", [(16, 2.5), (32, 1.0), (64, 5.0), (128, 2.5), (256, 2.5)])
def test_remap_layers_matches_per_layer(S, wire):
    sets = layer_set(S, wire, seed=S)
    say("remap_layers S=%d wire=%g: map %d layers twice" % (S, wire, len(sets)))
    La = [rxnn.map_layer(dev(W0), xb) for xb, W0, _ in sets]
    Lb = [rxnn.map_layer(dev(W0), xb) for xb, W0, _ in sets]
    W1 = [dev(W1) for _, _, W1 in sets]
    say("remap_layers per layer")
    for L, W in zip(La, W1):
        rxnn.remap_layer(L, W)
    say("remap_layers batched")
    rxnn.remap_layers(Lb, W1)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(La, Lb)):
        assert a.w_max() == b.w_max()
        for ga, gb in zip(all_gprime(a), all_gprime(b)):
            np.testing.assert_array_equal(gb, ga)
    # the oracle on the first and last tile of every layer (the last one only
    # for the large sides, whose oracle build takes about a second per array)
    for (xb, _, W1n), L in zip(sets, Lb):
        first = [] if S >= 128 else [0]
        lay = omap.map_layer(W1n, xb, col_tiles=sorted(set(first + [L.C - 1])),
                             row_tiles=sorted(set(first + [L.R - 1])))
        for (r, c), g in lay["gp"].items():
            for a in range(L.A):
                check_gprime(L.gprime(r, c, a), g[a])
    for L in La + Lb:
        L.free()


def test_remap_layers_resnet50_s64_evaluates_like_per_layer():
    """The 54 ResNet-50 shaped layers on 64 x 64 crossbars (12,478 arrays in
    one batch): every layer's evaluation after the batched rebuild equals its
    evaluation after per-layer rebuilds, bit for bit."""
    layers, Ws, works = [], [], []
    say("remap_layers resnet50 S=64: map 54 layers")
    for l in range(len(wl.resnet50_layers())):
        w = wl.stack_layer("resnet50", l, crossbar=64, batch=2)
        Wd = dev(w["W"])
        layers.append(rxnn.map_layer(Wd, w["xbar"]))
        sigma = float(np.sqrt(2.0 / w["W"].shape[0]))
        Ws.append(dev(wl.weight_perturbation(3000, w["W"], sigma)))
        works.append(w)

    def evaluate():
        Ys = []
        for L, w in zip(layers, works):
            X = dev(w["X"])
            if w["kind"] == "conv":
                Ys.append(rxnn.conv_layer(L, w["periph"], w["conv"], X).cpu().numpy())
            else:
                Ys.append(rxnn.crossbar_vmm(L, w["periph"], X).cpu().numpy())
        return Ys

    say("remap_layers resnet50 S=64: per layer")
    for L, W in zip(layers, Ws):
        rxnn.remap_layer(L, W)
    Y0 = evaluate()
    g0 = [L.gprime(L.R - 1, L.C - 1, 1) for L in layers]
    for L, w in zip(layers, works):            # back to the base weights
        rxnn.remap_layer(L, dev(w["W"]))
    say("remap_layers resnet50 S=64: batched")
    rxnn.remap_layers(layers, Ws)
    Y1 = evaluate()
    for l, (a, b) in enumerate(zip(Y0, Y1)):
        np.testing.assert_array_equal(b, a, err_msg="layer %d" % l)
        np.testing.assert_array_equal(layers[l].gprime(layers[l].R - 1, layers[l].C - 1, 1),
                                      g0[l])
    for L in layers:
        L.free()


def test_remap_layers_rejections():
    say("remap_layers rejections")
    rng = np.random.default_rng(1)
    W = dev(rng.normal(0, 0.05, size=(40, 30)).astype(np.float32))
    L16 = rxnn.map_layer(W, wl.xbar(16, 16, 2.5))
    L32 = rxnn.map_layer(W, wl.xbar(32, 32, 2.5))
    Lw = rxnn.map_layer(W, wl.xbar(16, 16, 1.0))
    Lz = rxnn.map_layer(W, wl.xbar(16, 16, 0.0))          # row-sweep build
    for layers, msg in (([L16, L32], "differs"), ([L16, Lw], "differs"),
                        ([L16, Lz], "row-sweep"), ([L16, L16], "twice")):
        with pytest.raises(rxnn.RxnnError, match=msg):
            rxnn.remap_layers(layers, [W] * len(layers))
    with pytest.raises(ValueError):
        rxnn.remap_layers([], [])
    for L in (L16, L32, Lw, Lz):
        L.free()
