"""Pins of the oracle's device variation and characteristic table
(``oracle/variation.py``, ``oracle/mapping.py`` step 2)."""

import numpy as np
import pytest

from oracle import mapping as omap
from oracle import variation as ov


# ---------------------------------------------------------------------------
# Philox-4x64-10 against numpy's own implementation of the same generator
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("key", [(0, 0), (5, 7), (2**64 - 1, 12345), (0xDEADBEEF, 0)])
@pytest.mark.parametrize("ctr", [0, 1, 77, 2**40 + 3])
def test_philox_matches_numpy(key, ctr):
    # numpy's Philox advances its 256-bit counter before producing a block
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array([ctr, 0, 0, 0], dtype=np.uint64))
    want = [int(x) for x in bg.random_raw(4)]
    assert list(ov.philox4x64([ctr + 1, 0, 0, 0], key)) == want


def test_philox_array_matches_scalar():
    d = np.array([0, 1, 2, 1000, 2**33 + 5], dtype=np.uint64)
    words = ov.philox4x64_array(d, seed=99)
    for n, dv in enumerate(d):
        ref = ov.philox4x64([int(dv), 0, 0, 0], (99, 0))
        assert tuple(int(w[n]) for w in words) == ref


def test_philox_rounds_matter():
    assert ov.philox4x64([1, 0, 0, 0], (3, 0), rounds=10) != ov.philox4x64([1, 0, 0, 0], (3, 0),
                                                                           rounds=9)


# ---------------------------------------------------------------------------
# Normal draws and variation factors
# ---------------------------------------------------------------------------

def test_normal_moments():
    n = 200_000
    x0, x1, _, _ = ov.philox4x64_array(np.arange(n, dtype=np.uint64), seed=2024)
    z = ov.normal_from_words(x0, x1)
    assert abs(z.mean()) < 4.0 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 4.0 * np.sqrt(2.0 / n)
    assert abs(np.mean(np.abs(z) < 1.0) - 0.682689) < 0.005
    assert abs(np.mean(np.abs(z) < 2.0) - 0.954500) < 0.003


def test_uniform_edges():
    # u1 is never 0 (log finite), u2 never reaches 1
    z = ov.normal_from_words(np.array([0, 2**64 - 1], dtype=np.uint64),
                             np.array([0, 2**64 - 1], dtype=np.uint64))
    assert np.all(np.isfinite(z))


def test_generated_factors_statistics():
    n, sigma = 100_000, 0.1
    vf = ov.generated_factors(np.arange(n, dtype=np.uint64), seed=7, sigma=sigma)
    assert np.all(vf >= 0.0)
    assert abs(vf.mean() - 1.0) < 4.0 * sigma / np.sqrt(n)
    assert abs(vf.std() - sigma) < 0.01 * sigma * 4
    # different seeds give independent factors; the same seed the same ones
    assert np.array_equal(vf, ov.generated_factors(np.arange(n, dtype=np.uint64), 7, sigma))
    other = ov.generated_factors(np.arange(n, dtype=np.uint64), 8, sigma)
    assert abs(np.corrcoef(vf, other)[0, 1]) < 0.02


def test_device_indices_layout():
    d = ov.device_indices(6, 2, 3, 4)
    assert d.shape == (2, 3, 4)
    assert int(d[0, 0, 0]) == 6 * 12
    assert int(d[1, 2, 3]) == 7 * 12 + 2 * 4 + 3
    assert len(np.unique(d)) == d.size


# ---------------------------------------------------------------------------
# Characteristic table
# ---------------------------------------------------------------------------

def test_identity_table_is_linear_device():
    u = np.linspace(0.0, 1.0, 101)
    np.testing.assert_allclose(ov.characteristic(u, [0.0, 1.0]), u, rtol=0, atol=1e-15)
    np.testing.assert_allclose(ov.characteristic(u, np.linspace(0, 1, 9)), u, rtol=0, atol=1e-15)


def test_table_samples_and_interpolation():
    f = np.array([0.0, 0.3, 0.55, 0.8, 1.0])
    k = np.arange(5)
    np.testing.assert_array_equal(ov.characteristic(k / 4.0, f), f)
    mid = (k[:-1] + 0.5) / 4.0
    np.testing.assert_allclose(ov.characteristic(mid, f), 0.5 * (f[:-1] + f[1:]), atol=1e-15)
    # levels beyond the range clamp to the end samples
    np.testing.assert_array_equal(ov.characteristic([-0.5, 1.5], f), [0.0, 1.0])


# ---------------------------------------------------------------------------
# Step 2 with variation and a characteristic table
# ---------------------------------------------------------------------------

def base_params(wb=0, sb=0):
    return {"rows": 4, "cols": 3, "g_min": 5e-6, "g_max": 50e-6, "r_driver": 1000.0,
            "r_sense": 1000.0, "r_row": 2.5, "r_col": 2.5, "weight_bits": wb,
            "bits_per_slice": sb, "w_max": 0.0}


def test_unit_variation_reproduces_base():
    rng = np.random.default_rng(3)
    W = rng.normal(0, 0.05, size=(10, 7)).astype(np.float32)
    for wb, sb in ((0, 0), (8, 2), (4, 0)):
        p = base_params(wb, sb)
        base = omap.map_layer(W, p)
        R, C, A = base["R"], base["C"], base["A"]
        ones = np.ones((C, R, A, 4, 3))
        for extra in ({"variation": ones}, {"variation_sigma": 0.0, "variation_seed": 5}):
            var = omap.map_layer(W, dict(p, **extra))
            for key in base["gp"]:
                np.testing.assert_array_equal(var["gp"][key], base["gp"][key])


def test_supplied_variation_scales_conductances():
    rng = np.random.default_rng(4)
    W = rng.normal(0, 0.05, size=(8, 6)).astype(np.float32)
    p = base_params()
    frag = omap.tile_weights(W, p, 1, 0)
    w_max = omap.layer_w_max(W, p)
    vf = rng.uniform(0.8, 1.2, size=(2, 4, 3))
    np.testing.assert_array_equal(omap.array_conductances(frag, p, w_max, vf),
                                  omap.array_conductances(frag, p, w_max) * vf)


def test_identity_table_reproduces_linear_mapping():
    rng = np.random.default_rng(5)
    W = rng.normal(0, 0.05, size=(8, 6)).astype(np.float32)
    for wb, sb in ((0, 0), (8, 2), (6, 3)):
        p = base_params(wb, sb)
        frag = omap.tile_weights(W, p, 0, 1)
        w_max = omap.layer_w_max(W, p)
        lin = omap.array_conductances(frag, p, w_max)
        tab = omap.array_conductances(frag, dict(p, g_lut=[0.0, 1.0]), w_max)
        np.testing.assert_allclose(tab, lin, rtol=1e-14, atol=0)


def test_table_levels_of_slices():
    # a 2-bit slice digit d reads the table at d / 3; with 4 samples exactly
    f = [0.0, 0.5, 0.75, 1.0]
    p = dict(base_params(2, 2), g_lut=f)
    W = np.array([[0.0, 1 / 3, 2 / 3, 1.0]], dtype=np.float32)
    p["rows"], p["cols"] = 1, 4
    G = omap.array_conductances(omap.tile_weights(W, p, 0, 0), p, 1.0)
    want = 5e-6 + 45e-6 * np.array(f)
    np.testing.assert_allclose(G[0, 0], want, rtol=1e-15)
    np.testing.assert_allclose(G[1, 0], 5e-6, rtol=0)


def test_mean_conductance_over_samples():
    """E[VF] = 1: the mean over many seeds of a varied device's conductance
    is its nominal conductance."""
    rng = np.random.default_rng(6)
    W = rng.normal(0, 0.05, size=(4, 3)).astype(np.float32)
    p = base_params()
    frag = omap.tile_weights(W, p, 0, 0)
    w_max = omap.layer_w_max(W, p)
    nominal = omap.array_conductances(frag, p, w_max)
    n, sigma = 4000, 0.1
    acc = np.zeros_like(nominal)
    for seed in range(n):
        acc += omap.array_conductances(
            frag, p, w_max, omap.variation_factors(dict(p, variation_sigma=sigma,
                                                        variation_seed=seed), 0, 0, 1, 2, 4, 3))
    np.testing.assert_allclose(acc / n, nominal, rtol=4 * sigma / np.sqrt(n))
