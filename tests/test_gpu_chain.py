"""The ResNet-18 shaped stack evaluated as one network (every layer's input is
the previous layers' crossbar output through ReLU, max pool, residual
additions and average pool), with teacher-forced layer parity: for sampled
layers the oracle takes the GPU's own input of that layer and checks the GPU's
output on sampled rows under the parity rule (every row tile's G' for the last
column tile).  The end-to-end deviation from the ideal fp32 network is
reported, not gated (it is the non-idealities' effect, not an error)."""

import numpy as np
import pytest

from oracle import fcm as ofcm
from oracle import mapping as omap
from oracle import periph as oper

from parity import array_weights, check_gprime, check_outputs_by_codes
from test_gpu_stacks import sample_patch_rows

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import chain, rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402

# layers whose oracle check stays within a few seconds each (up to 18 row
# tiles of 128 x 128): the stem, both blocks of the first stage, every
# downsample, the first convolution of each later stage and the classifier
CHECKED = (0, 1, 2, 3, 4, 5, 6, 7, 10, 12, 15, 17, 20)


def say(*a):
    print("[case]", *a, flush=True)


def test_resnet18_chained_teacher_forced():
    specs = wl.resnet18_layers()
    batch = 2
    xb = wl.xbar(128, 128, 1.0)
    say("resnet18 chained: map %d layers" % len(specs))
    Ws = [wl.he_weight(1003 + l, spec) for l, spec in enumerate(specs)]
    Wd = [torch.from_numpy(W).cuda() for W in Ws]
    layers = [rxnn.map_layer(W, xb) for W in Wd]
    X = torch.from_numpy(wl.uniform(2003, (batch, 3, 224, 224))).cuda()
    record = []
    say("resnet18 chained: forward")
    Y = chain.resnet18_forward(layers, specs, X, record=record)
    torch.cuda.synchronize()
    assert len(record) == len(specs) and torch.isfinite(Y).all()
    Yi = chain.resnet18_ideal(Wd, specs, X)
    rel = float(torch.linalg.norm(Y - Yi) / torch.linalg.norm(Yi))
    say("resnet18 chained: end-to-end relative deviation from the ideal network %.3g" % rel)
    total_diff = total_codes = 0
    for l, x, pp, y in record:
        if l not in CHECKED:
            continue
        spec, W = specs[l], Ws[l]
        P, Q = W.shape
        R, C = -(-P // 128), -(-Q // 128)
        c = C - 1
        x, y = x.cpu().numpy(), y.cpu().numpy()
        if spec["kind"] == "conv":
            cv = wl.conv_desc(spec, batch)
            rows, ho, wo = sample_patch_rows(cv, 32, seed=l)
            img, pix = rows // (ho * wo), rows % (ho * wo)
            imgs = sorted(set(int(i) for i in img))
            Xs = ofcm.im2col(x, cv, imgs)[np.searchsorted(imgs, img) * (ho * wo) + pix]
            Yg = y[img, :, pix // wo, pix % wo]
        else:
            Xs, Yg = x, y
        say("resnet18 chained: oracle on layer %d %s (%d arrays)" % (l, spec["name"], R * 2))
        lay = omap.map_layer(W, xb, col_tiles=[c])
        check_gprime(layers[l].gprime(R - 1, c, 1), lay["gp"][(R - 1, c)][1])
        _, dbg = ofcm.crossbar_vmm(Xs, lay, xb, pp, col_tiles=[c], debug=True)
        thr = oper.adc_thresholds(8, oper.adc_full_scale(pp, 128, xb["g_max"]), pp["adc_bend"])
        scale = oper.output_scale(pp, 128, xb["g_max"], lay["s_w_eff"])
        q0, q1 = c * 128, min(Q, (c + 1) * 128)
        part = {(r, a): (I[:, :q1 - q0], code[:, :q1 - q0])
                for (r, cc, a), (I, code) in dbg.items() if cc == c}
        nd, nc = check_outputs_by_codes(Yg[:, q0:q1], part, array_weights(2, 0), thr, scale)
        total_diff += nd
        total_codes += nc
    say("resnet18 chained: outputs off by a threshold flip: %d (of %d codes)"
        % (total_diff, total_codes))
    for L in layers:
        L.free()
