"""Host-side checks of librxnn that need no GPU: the library loads, exports
every function include/rxnn.h declares, and rejects invalid arguments before
any HIP call is made."""

import ctypes
import os
import re

import pytest

from paper_1809_00072_amd import rxnn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "rxnn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rxnn_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rxnn.LIB_PATH):
        pytest.fail("librxnn.so is not built (run __graft_entry__.build())")
    return rxnn.load()


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(rxnn.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for st, text in ((0, b"ok"), (-1, b"invalid argument"), (-2, b"out of device memory"),
                     (-3, b"HIP runtime error"), (-4, b"unsupported by this library")):
        assert lib.rxnn_status_string(st) == text


def good_params(**kw):
    d = dict(rows=64, cols=64, g_min=5e-6, g_max=50e-6, r_driver=1e3, r_sense=1e3, r_row=2.5,
             r_col=2.5, weight_bits=0, bits_per_slice=0, w_max=0.0)
    d.update(kw)
    return rxnn.xbar_params(d)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


@pytest.mark.parametrize("kw,status,msg", [
    (dict(rows=0), rxnn.RXNN_EINVAL, "positive"),
    (dict(cols=-3), rxnn.RXNN_EINVAL, "positive"),
    (dict(rows=300), rxnn.RXNN_EINVAL, "256"),
    (dict(rows=128, r_row=0.0), rxnn.RXNN_EUNSUPPORTED, "positive wire"),
    (dict(g_min=0.0), rxnn.RXNN_EINVAL, "g_min"),
    (dict(g_min=6e-5), rxnn.RXNN_EINVAL, "g_min"),
    (dict(r_row=-1.0), rxnn.RXNN_EINVAL, "resistances"),
    (dict(r_sense=float("nan")), rxnn.RXNN_EINVAL, "resistances"),
    (dict(weight_bits=17), rxnn.RXNN_EINVAL, "weight_bits"),
    (dict(weight_bits=0, bits_per_slice=2), rxnn.RXNN_EINVAL, "bits_per_slice"),
    (dict(weight_bits=8, bits_per_slice=3), rxnn.RXNN_EINVAL, "multiple"),
    (dict(w_max=float("inf")), rxnn.RXNN_EINVAL, "w_max"),
])
def test_map_rejects_bad_params(lib, kw, status, msg):
    p = good_params(**kw)
    h = ctypes.c_void_p()
    st = lib.rxnn_map_layer(ctypes.byref(p), FAKE, 10, 10, None, ctypes.byref(h))
    assert st == status
    assert msg in lib.rxnn_last_error().decode()
    assert not h.value


def test_map_rejects_null_and_sizes(lib):
    p = good_params()
    h = ctypes.c_void_p()
    assert lib.rxnn_map_layer(None, FAKE, 10, 10, None, ctypes.byref(h)) == rxnn.RXNN_EINVAL
    assert lib.rxnn_map_layer(ctypes.byref(p), None, 10, 10, None, ctypes.byref(h)) == rxnn.RXNN_EINVAL
    assert lib.rxnn_map_layer(ctypes.byref(p), FAKE, 0, 10, None, ctypes.byref(h)) == rxnn.RXNN_EINVAL
    assert lib.rxnn_map_layer(ctypes.byref(p), FAKE, 10, -1, None, ctypes.byref(h)) == rxnn.RXNN_EINVAL
    assert lib.rxnn_map_layer(ctypes.byref(p), FAKE, 10, 10, None, None) == rxnn.RXNN_EINVAL


@pytest.mark.parametrize("setup,msg", [
    (lambda p: (setattr(p, "variation", 0x2000), setattr(p, "variation_sigma", 0.1)), "not both"),
    (lambda p: setattr(p, "variation_sigma", -0.1), "variation_sigma"),
    (lambda p: setattr(p, "variation_sigma", float("nan")), "variation_sigma"),
    (lambda p: setattr(p, "g_lut_n", 3), "without g_lut"),
])
def test_map_rejects_bad_variation(lib, setup, msg):
    p = good_params()
    setup(p)
    h = ctypes.c_void_p()
    assert lib.rxnn_map_layer(ctypes.byref(p), FAKE, 10, 10, None, ctypes.byref(h)) == \
        rxnn.RXNN_EINVAL
    assert msg in lib.rxnn_last_error().decode()


@pytest.mark.parametrize("vals,msg", [
    ([0.5], "g_lut_n"),
    ([0.0, 1.5], "not in [0, 1]"),
    ([0.0, float("nan"), 1.0], "not in [0, 1]"),
    ([-0.1, 1.0], "not in [0, 1]"),
])
def test_map_rejects_bad_characteristic(lib, vals, msg):
    arr = (ctypes.c_double * len(vals))(*vals)
    p = good_params()
    p.g_lut = ctypes.cast(arr, ctypes.c_void_p)
    p.g_lut_n = len(vals)
    h = ctypes.c_void_p()
    assert lib.rxnn_map_layer(ctypes.byref(p), FAKE, 10, 10, None, ctypes.byref(h)) == \
        rxnn.RXNN_EINVAL
    assert msg in lib.rxnn_last_error().decode()


def test_calls_reject_unknown_handles(lib):
    pp = rxnn.periph_params(dict(dac_bits=4, x_max=1.0, v_read=0.2, dac_bend=0.1, adc_bits=8,
                                 adc_bend=0.05))
    bogus = ctypes.c_void_p(0x3000)
    assert lib.rxnn_crossbar_vmm(bogus, ctypes.byref(pp), FAKE, 4, FAKE, None) == rxnn.RXNN_EINVAL
    assert "handle" in lib.rxnn_last_error().decode()
    cd = rxnn.ConvDesc(1, 1, 4, 4, 1, 3, 3, 1, 1)
    assert lib.rxnn_conv_layer(bogus, ctypes.byref(pp), ctypes.byref(cd), FAKE, FAKE, None) == \
        rxnn.RXNN_EINVAL
    assert lib.rxnn_fc_backward(bogus, ctypes.byref(pp), FAKE, FAKE, FAKE, 4, FAKE, FAKE,
                                None) == rxnn.RXNN_EINVAL
    assert lib.rxnn_conv_backward(bogus, ctypes.byref(pp), ctypes.byref(cd), FAKE, FAKE, FAKE,
                                  FAKE, FAKE, None) == rxnn.RXNN_EINVAL
    assert "handle" in lib.rxnn_last_error().decode()
    buf = (ctypes.c_float * 16)()
    assert lib.rxnn_get_gprime(bogus, 0, 0, 0, buf) == rxnn.RXNN_EINVAL
    assert lib.rxnn_set_gprime(bogus, 0, 0, 0, buf) == rxnn.RXNN_EINVAL
    info = (ctypes.c_int64 * 7)()
    assert lib.rxnn_layer_info(bogus, info) == rxnn.RXNN_EINVAL
    assert lib.rxnn_layer_info(None, info) == rxnn.RXNN_EINVAL
    lib.rxnn_free_layer(None)
    lib.rxnn_free_layer(bogus)  # unknown handles are ignored


def test_profile_read_rejects_null(lib):
    assert lib.rxnn_profile_read(None, None, None) == rxnn.RXNN_EINVAL
