"""Python binding of librxnn (ctypes).

Argument marshalling only: every step of the crossbar path runs in the HIP
library.  Tensors are torch tensors on the HIP device; their data pointers
and the current torch stream are handed to the C ABI declared in
``include/rxnn.h``.  Loading fails loudly when the library has not been built.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librxnn.so")

RXNN_OK, RXNN_EINVAL, RXNN_ENOMEM, RXNN_EHIP, RXNN_EUNSUPPORTED = 0, -1, -2, -3, -4

EXPORTS = (
    "rxnn_map_layer", "rxnn_remap_layer", "rxnn_crossbar_vmm", "rxnn_conv_layer", "rxnn_get_gprime",
    "rxnn_set_gprime", "rxnn_vmm_debug", "rxnn_layer_info", "rxnn_layer_wmax",
    "rxnn_free_layer", "rxnn_profile_enable", "rxnn_profile_reset", "rxnn_profile_read",
    "rxnn_status_string", "rxnn_last_error", "rxnn_fc_backward", "rxnn_conv_backward",
    "rxnn_profile_bytes", "rxnn_crossbar_vmm_noalloc", "rxnn_remap_layers",
)


class XbarParams(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int32), ("cols", ctypes.c_int32),
        ("g_min", ctypes.c_double), ("g_max", ctypes.c_double),
        ("r_driver", ctypes.c_double), ("r_sense", ctypes.c_double),
        ("r_row", ctypes.c_double), ("r_col", ctypes.c_double),
        ("weight_bits", ctypes.c_int32), ("bits_per_slice", ctypes.c_int32),
        ("w_max", ctypes.c_double),
        ("variation", ctypes.c_void_p),
        ("variation_sigma", ctypes.c_double),
        ("variation_seed", ctypes.c_uint64),
        ("g_lut", ctypes.c_void_p),
        ("g_lut_n", ctypes.c_int32),
    ]


class PeriphParams(ctypes.Structure):
    _fields_ = [
        ("dac_bits", ctypes.c_int32),
        ("x_max", ctypes.c_double), ("v_read", ctypes.c_double), ("dac_bend", ctypes.c_double),
        ("adc_bits", ctypes.c_int32),
        ("adc_bend", ctypes.c_double),
        ("dac_g_on", ctypes.c_double), ("dac_g_pd", ctypes.c_double),
    ]


class ConvDesc(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in
                ("n", "c_in", "h", "w", "c_out", "kh", "kw", "stride", "pad")]


class RxnnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"rxnn status {status}: {message}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH):
    """Load librxnn.so (once).  Raises if it is missing: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run paper_1809_00072_amd.build first")
    lib = ctypes.CDLL(path)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    sig = {
        "rxnn_map_layer": ([ctypes.POINTER(XbarParams), vp, i64, i64, vp, ctypes.POINTER(vp)], i32),
        "rxnn_remap_layer": ([vp, vp, vp], i32),
        "rxnn_remap_layers": ([ctypes.POINTER(vp), ctypes.POINTER(vp), i32, vp], i32),
        "rxnn_crossbar_vmm": ([vp, ctypes.POINTER(PeriphParams), vp, i64, vp, vp], i32),
        "rxnn_crossbar_vmm_noalloc": ([vp, ctypes.POINTER(PeriphParams), vp, i64, vp, vp], i32),
        "rxnn_conv_layer": ([vp, ctypes.POINTER(PeriphParams), ctypes.POINTER(ConvDesc), vp, vp, vp], i32),
        "rxnn_get_gprime": ([vp, i64, i64, i64, vp], i32),
        "rxnn_set_gprime": ([vp, i64, i64, i64, vp], i32),
        "rxnn_vmm_debug": ([vp, ctypes.POINTER(PeriphParams), vp, i64, vp, vp, vp, vp], i32),
        "rxnn_layer_info": ([vp, ctypes.POINTER(i64)], i32),
        "rxnn_layer_wmax": ([vp, ctypes.POINTER(ctypes.c_double)], i32),
        "rxnn_free_layer": ([vp], None),
        "rxnn_profile_enable": ([i32], i32),
        "rxnn_profile_reset": ([], i32),
        "rxnn_profile_read": ([ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)], i32),
        "rxnn_profile_bytes": ([ctypes.c_char_p, ctypes.POINTER(ctypes.c_double)], i32),
        "rxnn_fc_backward": ([vp, ctypes.POINTER(PeriphParams), vp, vp, vp, i64, vp, vp, vp], i32),
        "rxnn_conv_backward": ([vp, ctypes.POINTER(PeriphParams), ctypes.POINTER(ConvDesc), vp, vp,
                                vp, vp, vp, vp], i32),
        "rxnn_status_string": ([i32], ctypes.c_char_p),
        "rxnn_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status):
    if status != RXNN_OK:
        lib = load()
        raise RxnnError(status, lib.rxnn_last_error().decode())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, dtype=None, what="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be on the HIP device")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def xbar_params(d, variation=None, lut=None) -> XbarParams:
    """The C struct of a parameter dict.  ``variation``: device address of the
    factor array (or None); ``lut``: a ctypes double array the caller keeps
    alive during the call (or None)."""
    return XbarParams(int(d["rows"]), int(d["cols"]), float(d["g_min"]), float(d["g_max"]),
                      float(d["r_driver"]), float(d["r_sense"]), float(d["r_row"]),
                      float(d["r_col"]), int(d.get("weight_bits", 0)),
                      int(d.get("bits_per_slice", 0)), float(d.get("w_max", 0.0)), variation,
                      float(d.get("variation_sigma", 0.0) or 0.0),
                      int(d.get("variation_seed", 0) or 0),
                      ctypes.cast(lut, ctypes.c_void_p) if lut is not None else None,
                      len(lut) if lut is not None else 0)


def periph_params(d) -> PeriphParams:
    return PeriphParams(int(d["dac_bits"]), float(d["x_max"]), float(d["v_read"]),
                        float(d["dac_bend"]), int(d["adc_bits"]), float(d["adc_bend"]),
                        float(d.get("dac_g_on", 0.0) or 0.0),
                        float(d.get("dac_g_pd", 0.0) or 0.0))


@dataclass
class Layer:
    """A mapped layer (handle to the library's G' buffer)."""
    handle: ctypes.c_void_p
    P: int
    Q: int
    M: int
    N: int
    R: int
    C: int
    A: int
    _freed: bool = field(default=False, repr=False)

    def free(self):
        if not self._freed and self.handle:
            load().rxnn_free_layer(self.handle)
        self._freed = True

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    def gprime(self, r, c, a):
        import numpy as np
        out = np.empty((self.M, self.N), dtype=np.float32)
        _check(load().rxnn_get_gprime(self.handle, r, c, a, out.ctypes.data_as(ctypes.c_void_p)))
        return out

    def set_gprime(self, r, c, a, g):
        import numpy as np
        g = np.ascontiguousarray(g, dtype=np.float32)
        assert g.shape == (self.M, self.N)
        _check(load().rxnn_set_gprime(self.handle, r, c, a, g.ctypes.data_as(ctypes.c_void_p)))

    def w_max(self):
        v = ctypes.c_double()
        _check(load().rxnn_layer_wmax(self.handle, ctypes.byref(v)))
        return v.value


def map_layer(W, params, stream=None) -> Layer:
    """rxnn_map_layer: W is a device fp32 P x Q tensor; params a dict."""
    import torch
    lib = load()
    if W.dim() != 2:
        raise ValueError("W must be 2-D (P x Q)")
    P, Q = W.shape
    h = ctypes.c_void_p()
    var = params.get("variation")
    vptr = None
    if var is not None:
        # one factor per device, [C][R][A][M][N], on W's device
        if not (isinstance(var, torch.Tensor) and var.dtype == torch.float32 and var.is_contiguous()
                and var.device == W.device):
            raise ValueError("variation must be a contiguous fp32 tensor on W's device")
        vptr = var.data_ptr()
    lut = params.get("g_lut")
    lut_arr = None
    if lut is not None:
        vals = [float(v) for v in lut]
        lut_arr = (ctypes.c_double * len(vals))(*vals)
    p = xbar_params(params, vptr, lut_arr)
    _check(lib.rxnn_map_layer(ctypes.byref(p), _ptr(W, torch.float32, "W"), P, Q,
                              _stream(stream), ctypes.byref(h)))
    info = (ctypes.c_int64 * 7)()
    _check(lib.rxnn_layer_info(h, info))
    return Layer(h, *[int(v) for v in info])


def remap_layer(layer: Layer, W, stream=None):
    """rxnn_remap_layer: rebuild the layer's G' in place from new weights W."""
    import torch
    if tuple(W.shape) != (layer.P, layer.Q):
        raise ValueError(f"W must be {layer.P} x {layer.Q}")
    _check(load().rxnn_remap_layer(layer.handle, _ptr(W, torch.float32, "W"), _stream(stream)))


def remap_layers(layers, Ws, stream=None):
    """rxnn_remap_layers: rebuild the G' of every layer from its new weights
    in one launch sequence (layers of one crossbar size and resistances)."""
    import torch
    if len(layers) != len(Ws) or not layers:
        raise ValueError("one weight tensor per layer, at least one layer")
    for L, W in zip(layers, Ws):
        if tuple(W.shape) != (L.P, L.Q):
            raise ValueError(f"W must be {L.P} x {L.Q}")
    n = len(layers)
    hs = (ctypes.c_void_p * n)(*[L.handle.value if isinstance(L.handle, ctypes.c_void_p)
                                  else L.handle for L in layers])
    ws = (ctypes.c_void_p * n)(*[_ptr(W, torch.float32, "W").value for W in Ws])
    _check(load().rxnn_remap_layers(hs, ws, n, _stream(stream)))


def crossbar_vmm(layer: Layer, periph, X, Y=None, stream=None):
    """rxnn_crossbar_vmm: X device fp32 B x P -> Y device fp32 B x Q."""
    import torch
    B = X.shape[0]
    if X.dim() != 2 or X.shape[1] != layer.P:
        raise ValueError(f"X must be B x {layer.P}")
    if Y is None:
        Y = torch.empty((B, layer.Q), dtype=torch.float32, device=X.device)
    pp = periph_params(periph)
    _check(load().rxnn_crossbar_vmm(layer.handle, ctypes.byref(pp), _ptr(X, torch.float32, "X"),
                                    B, _ptr(Y, torch.float32, "Y"), _stream(stream)))
    return Y


def crossbar_vmm_noalloc(layer: Layer, periph, X, Y, stream=None):
    """rxnn_crossbar_vmm_noalloc: like crossbar_vmm, into the caller's Y
    (device fp32 B x Q); the library allocates nothing."""
    import torch
    B = X.shape[0]
    if X.dim() != 2 or X.shape[1] != layer.P:
        raise ValueError(f"X must be B x {layer.P}")
    if tuple(Y.shape) != (B, layer.Q):
        raise ValueError(f"Y must be {B} x {layer.Q}")
    pp = periph_params(periph)
    _check(load().rxnn_crossbar_vmm_noalloc(layer.handle, ctypes.byref(pp),
                                            _ptr(X, torch.float32, "X"), B,
                                            _ptr(Y, torch.float32, "Y"), _stream(stream)))
    return Y


def vmm_debug(layer: Layer, periph, X, stream=None):
    """rxnn_vmm_debug: returns (Y, I_preadc, codes) with I/codes [R][C][A][B][N]."""
    import torch
    B = X.shape[0]
    Y = torch.empty((B, layer.Q), dtype=torch.float32, device=X.device)
    I = torch.empty((layer.R, layer.C, layer.A, B, layer.N), dtype=torch.float32, device=X.device)
    codes = torch.empty_like(I, dtype=torch.int32)
    pp = periph_params(periph)
    _check(load().rxnn_vmm_debug(layer.handle, ctypes.byref(pp), _ptr(X, torch.float32, "X"), B,
                                 _ptr(Y), _ptr(I), _ptr(codes), _stream(stream)))
    return Y, I, codes


def conv_out_hw(conv):
    ho = (conv["h"] + 2 * conv["pad"] - conv["kh"]) // conv["stride"] + 1
    wo = (conv["w"] + 2 * conv["pad"] - conv["kw"]) // conv["stride"] + 1
    return ho, wo


def conv_layer(layer: Layer, periph, conv, X, Y=None, stream=None):
    """rxnn_conv_layer: X device fp32 NCHW -> Y device fp32 NCHW."""
    import torch
    cd = ConvDesc(*[int(conv[k]) for k in ("n", "c_in", "h", "w", "c_out", "kh", "kw",
                                           "stride", "pad")])
    if tuple(X.shape) != (conv["n"], conv["c_in"], conv["h"], conv["w"]):
        raise ValueError("X shape does not match the convolution")
    ho, wo = conv_out_hw(conv)
    if Y is None:
        Y = torch.empty((conv["n"], conv["c_out"], ho, wo), dtype=torch.float32, device=X.device)
    pp = periph_params(periph)
    _check(load().rxnn_conv_layer(layer.handle, ctypes.byref(pp), ctypes.byref(cd),
                                  _ptr(X, torch.float32, "X"), _ptr(Y, torch.float32, "Y"),
                                  _stream(stream)))
    return Y


def _grad_out(buf, like, want, what):
    import torch
    if buf is not None:
        if tuple(buf.shape) != tuple(like.shape):
            raise ValueError(f"{what} must have shape {tuple(like.shape)}")
        return buf
    return torch.empty_like(like) if want else None


def fc_backward(layer: Layer, periph, W, X, dY, want_dx=True, want_dw=True, dX=None, dW=None,
                stream=None):
    """rxnn_fc_backward: (dX B x P or None, dW P x Q or None), device fp32,
    written into the given buffers or new ones."""
    import torch
    B = X.shape[0]
    if tuple(W.shape) != (layer.P, layer.Q):
        raise ValueError(f"W must be {layer.P} x {layer.Q}")
    if X.dim() != 2 or X.shape[1] != layer.P:
        raise ValueError(f"X must be B x {layer.P}")
    if tuple(dY.shape) != (B, layer.Q):
        raise ValueError(f"dY must be {B} x {layer.Q}")
    dX = _grad_out(dX, X, want_dx, "dX")
    dW = _grad_out(dW, W, want_dw, "dW")
    pp = periph_params(periph)
    _check(load().rxnn_fc_backward(layer.handle, ctypes.byref(pp), _ptr(W, torch.float32, "W"),
                                   _ptr(X, torch.float32, "X"), _ptr(dY, torch.float32, "dY"), B,
                                   _ptr(dX), _ptr(dW), _stream(stream)))
    return dX, dW


def conv_backward(layer: Layer, periph, conv, W, X, dY, want_dx=True, want_dw=True, dX=None,
                  dW=None, stream=None):
    """rxnn_conv_backward: (dX NCHW or None, dW P x Q or None), device fp32,
    written into the given buffers or new ones."""
    import torch
    cd = ConvDesc(*[int(conv[k]) for k in ("n", "c_in", "h", "w", "c_out", "kh", "kw",
                                           "stride", "pad")])
    if tuple(W.shape) != (layer.P, layer.Q):
        raise ValueError(f"W must be {layer.P} x {layer.Q}")
    if tuple(X.shape) != (conv["n"], conv["c_in"], conv["h"], conv["w"]):
        raise ValueError("X shape does not match the convolution")
    ho, wo = conv_out_hw(conv)
    if tuple(dY.shape) != (conv["n"], conv["c_out"], ho, wo):
        raise ValueError("dY shape does not match the convolution")
    dX = _grad_out(dX, X, want_dx, "dX")
    dW = _grad_out(dW, W, want_dw, "dW")
    pp = periph_params(periph)
    _check(load().rxnn_conv_backward(layer.handle, ctypes.byref(pp), ctypes.byref(cd),
                                     _ptr(W, torch.float32, "W"), _ptr(X, torch.float32, "X"),
                                     _ptr(dY, torch.float32, "dY"), _ptr(dX), _ptr(dW),
                                     _stream(stream)))
    return dX, dW


def profile_enable(on=True):
    """on: False/0 off, True/1 every kernel, 2 the evaluation kernel only."""
    _check(load().rxnn_profile_enable(int(on)))


def profile_reset():
    _check(load().rxnn_profile_reset())


def profile_read(kernel):
    """(total milliseconds, launches) of one kernel name since the last reset."""
    t = ctypes.c_double()
    n = ctypes.c_int64()
    _check(load().rxnn_profile_read(kernel.encode(), ctypes.byref(t), ctypes.byref(n)))
    return t.value, n.value


def profile_bytes(kernel):
    """Algorithmic HBM bytes of the timed launches of one kernel name since the
    last reset (0 where the library does not count them)."""
    b = ctypes.c_double()
    _check(load().rxnn_profile_bytes(kernel.encode(), ctypes.byref(b)))
    return b.value
