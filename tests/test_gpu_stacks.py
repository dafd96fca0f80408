"""GPU parity on the stacked workloads at their full sizes: the layers of a
ResNet-18 shaped stack on 128 x 128 crossbars, the VGG-16 shaped FC head with
bit-sliced weights on 64 x 64 crossbars, and ResNet-50 shaped layers swept over
crossbar sizes 32 ... 256 with the weights perturbed and G' rebuilt.

Each layer runs standalone on its seeded input (the chaining glue between
layers is not part of the crossbar path) over the whole batch, in the launch
configuration of a production call.  The oracle cannot map every array of
these layers in a test's time, so the check is sampled:

* the input is kept only on a few row tiles (other inputs are set to zero,
  so the other row tiles carry V = 0 and contribute code 0 exactly);
* the oracle maps the arrays of those row tiles for a few column tiles
  (first and last, the last one padded when Q is not a multiple of N);
* the GPU's G' of those arrays is checked element by element, and the GPU's
  layer outputs of the sampled images (rows) and columns are checked against
  the oracle's codes with ``parity.check_outputs_by_codes``.
"""

import numpy as np
import pytest

from oracle import fcm as ofcm
from oracle import mapping as omap
from oracle import periph as oper

from parity import array_weights, check_gprime, check_outputs_by_codes

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402


def say(*a):
    print("[case]", *a, flush=True)


def pick_row_tiles(R):
    return list(range(R)) if R <= 3 else [0, 1, R - 1]


def mask_inputs(work, rows):
    """Zero every input outside the row tiles ``rows`` (for a convolution,
    every input channel that is not wholly inside them)."""
    M = work["xbar"]["rows"]
    X = work["X"].copy()
    keep = np.zeros(work["W"].shape[0], dtype=bool)
    for r in rows:
        keep[r * M:(r + 1) * M] = True
    if work["kind"] == "fc":
        X[:, ~keep] = 0.0
    else:
        khw = work["conv"]["kh"] * work["conv"]["kw"]
        for ci in range(work["conv"]["c_in"]):
            if not keep[ci * khw:(ci + 1) * khw].all():
                X[:, ci] = 0.0
    assert X.any(), "the sample keeps no input"
    return X


def run_and_check(work, L=None, W=None, label=""):
    """Map (unless a mapped layer is given), evaluate on the GPU over the
    whole batch, and check the sample against the oracle."""
    xb, pp = work["xbar"], work["periph"]
    W = work["W"] if W is None else W
    P, Q = W.shape
    M, N = xb["rows"], xb["cols"]
    R, C = -(-P // M), -(-Q // N)
    rows = pick_row_tiles(R)
    cols = sorted({0, C - 1})
    X = mask_inputs(work, rows)
    say(label, "P=%d Q=%d M=%d R=%d C=%d row tiles %s col tiles %s" % (P, Q, M, R, C, rows, cols))
    if L is None:
        L = rxnn.map_layer(torch.from_numpy(W).cuda(), xb)
    Xd = torch.from_numpy(X).cuda()
    if work["kind"] == "conv":
        cv = work["conv"]
        Y = rxnn.conv_layer(L, pp, cv, Xd)
        sample = [cv["n"] - 1]
        Yg = Y[sample].cpu().numpy()                               # [1, Q, ho, wo]
        Yg = Yg.transpose(0, 2, 3, 1).reshape(-1, Q)               # patch rows x Q
    else:
        Y = rxnn.crossbar_vmm(L, pp, Xd)
        B = X.shape[0]
        sample = list(range(8)) + list(range(B - 8, B))
        Yg = Y.cpu().numpy()[sample]
    torch.cuda.synchronize()
    say(label, "oracle: %d arrays" % (len(rows) * len(cols) * L.A))
    lay = omap.map_layer(W, xb, col_tiles=cols, row_tiles=rows)
    for (r, c), g in lay["gp"].items():
        for a in range(L.A):
            check_gprime(L.gprime(r, c, a), g[a])
    if work["kind"] == "conv":
        _, dbg = ofcm.conv_layer(X, lay, xb, pp, work["conv"], images=sample, col_tiles=cols,
                                 row_tiles=rows, debug=True)
    else:
        _, dbg = ofcm.crossbar_vmm(X, lay, xb, pp, rows=sample, col_tiles=cols, row_tiles=rows,
                                   debug=True)
    thr = oper.adc_thresholds(int(pp["adc_bits"]), oper.adc_full_scale(pp, M, xb["g_max"]),
                              pp["adc_bend"])
    scale = oper.output_scale(pp, M, xb["g_max"], lay["s_w_eff"])
    weights = array_weights(L.A, omap.slicing(xb)[1])
    total_diff = total_codes = 0
    for c in cols:
        q0, q1 = c * N, min(Q, (c + 1) * N)
        part = {(r, a): (I[:, :q1 - q0], code[:, :q1 - q0])
                for (r, cc, a), (I, code) in dbg.items() if cc == c}
        nd, nc = check_outputs_by_codes(Yg[:, q0:q1], part, weights, thr, scale)
        total_diff += nd
        total_codes += nc
    say(label, "outputs differing by a threshold flip: %d (of %d codes)" % (total_diff, total_codes))
    return L


# ---------------------------------------------------------------------------
# ResNet-18 shaped stack: 128 x 128 crossbars, wire 1 Ohm, batch 64
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("l", [0, 1, 5, 7, 16, 20])
def test_resnet18_layer(l):
    work = wl.stack_layer("resnet18", l)
    L = run_and_check(work, label="resnet18 layer %d %s" % (l, work["spec"]["name"]))
    L.free()


# ---------------------------------------------------------------------------
# VGG-16 shaped FC head: 64 x 64 crossbars, 8-bit weights in 4 x 2-bit slices
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("l", [0, 1, 2])
def test_vgg16_fc_layer(l):
    work = wl.stack_layer("vgg16fc", l)
    L = run_and_check(work, label="vgg16fc layer %d %s" % (l, work["spec"]["name"]))
    L.free()


# ---------------------------------------------------------------------------
# ResNet-50 shaped layers over crossbar sizes and wire resistances
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("S,l,wire", [
    # every crossbar side at every wire resistance of the sweep
    (32, 12, 2.5),     # 3x3 stride 2, 128 channels
    (32, 53, 1.0),     # classifier
    (32, 6, 5.0),      # 3x3 64 -> 64 at 56 x 56
    (64, 3, 2.5),      # 1x1 64 -> 256
    (64, 25, 5.0),     # 3x3 stride 2, 256 channels
    (64, 14, 1.0),     # 1x1 stride 2 downsample 256 -> 512
    (128, 0, 2.5),     # 7x7 stride 2 stem
    (128, 46, 2.5),    # 1x1 stride 2 downsample to 2048
    (128, 5, 1.0),     # 1x1 256 -> 64
    (128, 9, 5.0),     # 3x3 64 -> 64 at 56 x 56
    (256, 2, 2.5),     # 3x3 64 -> 64 at 56 x 56
    (256, 45, 2.5),    # 1x1 512 -> 2048 at 7 x 7
    (256, 1, 1.0),     # 1x1 64 -> 64 at 56 x 56
    (256, 4, 5.0),     # 1x1 downsample 64 -> 256
])
def test_resnet50_layer(S, l, wire):
    work = wl.stack_layer("resnet50", l, crossbar=S, wire=wire)
    L = run_and_check(work, label="resnet50 S=%d wire=%g layer %d %s" % (
        S, wire, l, work["spec"]["name"]))
    L.free()


def test_resnet50_rebuild_after_update():
    """The model-in-the-loop step: perturb W, rebuild G' in place with
    rxnn_remap_layer, and evaluate again."""
    work = wl.stack_layer("resnet50", 16, crossbar=64)
    L = run_and_check(work, label="resnet50 S=64 layer 16 before update")
    sigma = float(np.sqrt(2.0 / work["W"].shape[0]))
    W1 = wl.weight_perturbation(3000, work["W"], sigma)
    assert not np.array_equal(W1, work["W"])
    rxnn.remap_layer(L, torch.from_numpy(W1).cuda())
    run_and_check(work, L=L, W=W1, label="resnet50 S=64 layer 16 after update")
    L.free()


# ---------------------------------------------------------------------------
# Real (unmasked) inputs: every row tile live
# ---------------------------------------------------------------------------

def sample_patch_rows(cv, n_rows, seed):
    """Seeded patch rows of a convolution: the first and last output pixel of
    the first and last image (borders) and random others, n_rows in all."""
    ho = (cv["h"] + 2 * cv["pad"] - cv["kh"]) // cv["stride"] + 1
    wo = (cv["w"] + 2 * cv["pad"] - cv["kw"]) // cv["stride"] + 1
    bv = cv["n"] * ho * wo
    fixed = [0, ho * wo - 1, bv - ho * wo, bv - 1]
    rng = np.random.default_rng(seed)
    rest = rng.choice(bv, size=n_rows, replace=False)
    rows = list(dict.fromkeys(fixed + [int(v) for v in rest]))[:n_rows]
    return np.array(sorted(rows)), ho, wo


def run_unmasked(work, n_rows=64, seed=0, label=""):
    """The layer on its real input over the whole batch (production launch);
    the oracle builds every row tile's G' for at most two column tiles (the
    first and the last, possibly padded one) and evaluates at most n_rows
    product rows; the outputs there are checked with
    ``parity.check_outputs_by_codes``."""
    xb, pp, W = work["xbar"], work["periph"], work["W"]
    P, Q = W.shape
    M, N = xb["rows"], xb["cols"]
    R, C = -(-P // M), -(-Q // N)
    cols = sorted({0, C - 1})
    say(label, "P=%d Q=%d M=%d R=%d C=%d: all row tiles, col tiles %s" % (P, Q, M, R, C, cols))
    L = rxnn.map_layer(torch.from_numpy(W).cuda(), xb)
    Xd = torch.from_numpy(work["X"]).cuda()
    if work["kind"] == "conv":
        cv = work["conv"]
        rows, ho, wo = sample_patch_rows(cv, n_rows, seed)
        Y = rxnn.conv_layer(L, pp, cv, Xd).cpu().numpy()
        img, pix = rows // (ho * wo), rows % (ho * wo)
        Yg = Y[img, :, pix // wo, pix % wo]                       # sampled rows x Q
        imgs = sorted(set(int(i) for i in img))
        patches = ofcm.im2col(work["X"], cv, imgs)                # rows of those images
        local = np.searchsorted(imgs, img) * (ho * wo) + pix
        Xs = patches[local]
    else:
        B = work["X"].shape[0]
        rng = np.random.default_rng(seed)
        rows = np.array(sorted(set([0, B - 1] + [int(v) for v in
                                                  rng.choice(B, size=min(n_rows, B), replace=False)])))[:n_rows]
        Y = rxnn.crossbar_vmm(L, pp, Xd).cpu().numpy()
        Yg = Y[rows]
        Xs = work["X"][rows]
    torch.cuda.synchronize()
    say(label, "oracle: %d arrays, %d rows" % (R * len(cols) * L.A, len(rows)))
    lay = omap.map_layer(W, xb, col_tiles=cols)
    for c in cols:
        for r in (0, R - 1):
            for a in range(L.A):
                check_gprime(L.gprime(r, c, a), lay["gp"][(r, c)][a])
    _, dbg = ofcm.crossbar_vmm(Xs, lay, xb, pp, col_tiles=cols, debug=True)
    thr = oper.adc_thresholds(int(pp["adc_bits"]), oper.adc_full_scale(pp, M, xb["g_max"]),
                              pp["adc_bend"])
    scale = oper.output_scale(pp, M, xb["g_max"], lay["s_w_eff"])
    weights = array_weights(L.A, omap.slicing(xb)[1])
    total_diff = total_codes = 0
    for c in cols:
        q0, q1 = c * N, min(Q, (c + 1) * N)
        part = {(r, a): (I[:, :q1 - q0], code[:, :q1 - q0])
                for (r, cc, a), (I, code) in dbg.items() if cc == c}
        nd, nc = check_outputs_by_codes(Yg[:, q0:q1], part, weights, thr, scale)
        total_diff += nd
        total_codes += nc
    say(label, "outputs differing by a threshold flip: %d (of %d codes)" % (total_diff, total_codes))
    L.free()


@pytest.mark.parametrize("config,l,S,wire", [
    ("resnet18", 1, None, None),       # 3x3 64 -> 64 at 56 x 56, 128 x 128 crossbars, 5 row tiles
    ("vgg16fc", 2, None, None),        # 4096 -> 1000, 64 row tiles, 8 arrays per position
    ("resnet50", 2, 256, 2.5),         # 3x3 64 -> 64 at 56 x 56 on 256 x 256 crossbars
    ("resnet50", 12, 32, 2.5),         # 3x3 stride 2, 128 channels, 36 row tiles (grouped walk)
])
def test_layer_unmasked_sampled(config, l, S, wire):
    work = wl.stack_layer(config, l, crossbar=S, wire=wire)
    run_unmasked(work, seed=l, label="%s unmasked layer %d %s S=%s wire=%s" % (
        config, l, work["spec"]["name"], S, wire))
