"""rxnn_crossbar_vmm_noalloc (the entry point for callers that cannot
allocate) against rxnn_crossbar_vmm through the C ABI: the same kernels on
buffers carved out of the library's fixed scratch array, so the outputs must
be identical bit for bit.  Two calls in a row on each layer, the second with a
smaller input; layers whose evaluation splits row tiles over workgroups (the
int32 workspace in the scratch), the divider DAC (row loads in the scratch)
and alternating layers that share the scratch.  A call that needs more
scratch than the array holds is rejected before any launch."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1809_00072_amd import rxnn  # noqa: E402
from paper_1809_00072_amd import workloads as wl  # noqa: E402


def say(*a):
    print("[case]", *a, flush=True)


def case(P, Q, M, N, B, dac, adc, seed, r_driver=wl.R_DRIVER):
    rng = np.random.default_rng(seed)
    W = torch.from_numpy(rng.normal(0, 0.05, size=(P, Q)).astype(np.float32)).cuda()
    X = torch.from_numpy(rng.random(size=(B, P)).astype(np.float32)).cuda()
    return W, X, wl.xbar(M, N, 2.5, r_driver=r_driver), wl.periph(dac, adc, 1.0)


def both(L, pp, X):
    Yr = rxnn.crossbar_vmm(L, pp, X)
    Yn = torch.full_like(Yr, float("nan"))
    rxnn.crossbar_vmm_noalloc(L, pp, X, Yn)
    torch.cuda.synchronize()
    return Yr.cpu().numpy(), Yn.cpu().numpy()


@pytest.mark.parametrize("P,Q,M,N,B,dac,adc,ldac", [
    (256, 128, 64, 64, 16, 4, 8, False),      # the FC 256 -> 128 workload
    (1200, 40, 16, 16, 40, 6, 8, False),      # many row tiles, few rows: split + int32 workspace
    (90, 70, 32, 32, 200, 8, 8, False),       # 32 x 32: grouped walk, odd R and C
    (300, 130, 128, 128, 20, 8, 0, False),    # ideal ADC
    (130, 70, 32, 32, 24, 6, 8, True),        # divider DAC: row loads in the scratch
])
def test_noalloc_matches_crossbar_vmm(P, Q, M, N, B, dac, adc, ldac):
    W, X, xb, pp = case(P, Q, M, N, B, dac, adc, seed=P + B,
                        r_driver=0.0 if ldac else wl.R_DRIVER)
    if ldac:
        pp = dict(pp, dac_bend=0.0, dac_g_on=5e-3, dac_g_pd=5e-4)
    say("noalloc", (P, Q, M, N, B, dac, adc, ldac), "map")
    L = rxnn.map_layer(W, xb)
    for b in (B, max(1, B // 3)):             # second call smaller than the first
        say("noalloc B=%d" % b)
        Yr, Yn = both(L, pp, X[:b].contiguous())
        np.testing.assert_array_equal(Yn, Yr)
    L.free()


def test_noalloc_layers_share_the_scratch():
    """Two layers alternate on the one scratch array (each call rebuilds its
    tables and clears its workspace), larger call first."""
    Wa, Xa, xba, ppa = case(1200, 40, 16, 16, 40, 6, 8, seed=1)
    Wb, Xb, xbb, ppb = case(200, 70, 64, 64, 130, 4, 6, seed=2)
    say("noalloc shared scratch map")
    La, Lb = rxnn.map_layer(Wa, xba), rxnn.map_layer(Wb, xbb)
    for L, pp, X in ((Lb, ppb, Xb), (La, ppa, Xa), (Lb, ppb, Xb[:37].contiguous()),
                     (La, ppa, Xa[:9].contiguous())):
        say("noalloc shared scratch B=%d P=%d" % (X.shape[0], L.P))
        Yr, Yn = both(L, pp, X)
        np.testing.assert_array_equal(Yn, Yr)
    La.free()
    Lb.free()


def test_noalloc_rejects_oversize():
    """B x (R M + 64) DAC outputs beyond the 64 MiB array: RXNN_EINVAL, nothing
    launched (Y keeps its contents); B = 0 is a no-op."""
    W, X, xb, pp = case(64, 16, 64, 16, 1, 4, 8, seed=3)
    L = rxnn.map_layer(W, xb)
    B = (64 << 20) // (4 * 128) + 1            # rows of 128 floats: just past 64 MiB
    say("noalloc oversize B=%d" % B)
    Xbig = torch.zeros((B, 64), dtype=torch.float32, device="cuda")
    Y = torch.full((B, 16), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(rxnn.RxnnError, match="scratch"):
        rxnn.crossbar_vmm_noalloc(L, pp, Xbig, Y)
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all())
    rxnn.crossbar_vmm_noalloc(L, pp, Xbig[:0], Y[:0])
    L.free()
