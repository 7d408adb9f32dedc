"""Thin Python binding of libhatq (ctypes).

Argument marshalling only: every step of the operator runs in the library's HIP
kernels.  PyTorch supplies device memory (tensors passed by ``data_ptr()``) and
the stream (``torch.cuda.current_stream()``).  There is no fallback: if the
library is missing or cannot be loaded, every call raises.

The function names mirror the C ABI in ``include/hatq.h``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

from . import build as _build

HATQ_OK, HATQ_EINVAL, HATQ_EUNSUPPORTED, HATQ_EWORKSPACE, HATQ_EHIP = range(5)
HATQ_DH, HATQ_WH = 0, 1
HATQ_OUT_I32, HATQ_OUT_F32, HATQ_OUT_I8 = 0, 1, 2
HATQ_PAIRED, HATQ_XQ_C64, HATQ_YQ_C64 = 1, 2, 4
FORMS = {"DH": HATQ_DH, "WH": HATQ_WH}


class HatqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class ConvDesc(ctypes.Structure):
    _fields_ = [("cin", ctypes.c_int32), ("cout", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("out_pad", ctypes.c_int32),
                ("transposed", ctypes.c_int32), ("hblock", ctypes.c_int32)]


class Weights(ctypes.Structure):
    _fields_ = [("d", ConvDesc), ("form", ctypes.c_int32), ("cin_pad", ctypes.c_int32),
                ("cout_pad", ctypes.c_int32), ("k_total", ctypes.c_int32),
                ("k_stride", ctypes.c_int32), ("wq", ctypes.c_void_p),
                ("w_scale", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("wpack", ctypes.c_void_p), ("pack_stride", ctypes.c_int32)]


EXPORTS = ["hatq_status_string", "hatq_conv_out_hw", "hatq_weights_bytes", "hatq_prepare_weights",
           "hatq_export_weights", "hatq_pack_weights", "hatq_fwht_quant_ws_bytes", "hatq_fwht_quant_act",
           "hatq_fwht_quant_act_noalloc", "hatq_fwht_quant_act_c64", "hatq_conv_int8",
           "hatq_conv_int8_requant", "hatq_int_table_len", "hatq_int_transition_params",
           "hatq_conv_int8_int_transition", "hatq_range_expansion", "hatq_select_form", "hatq_hadamard_order",
           "hatq_fwht_quant_affine_ws_bytes", "hatq_fwht_quant_act_affine", "hatq_tapsum_len",
           "hatq_weight_tapsums", "hatq_conv_int8_affine",
           "hatq_layer_ws_bytes", "hatq_layer_forward"]

_lib = None


def lib_path() -> str:
    return _build.LIB


def load(build_if_missing: bool = False):
    """Load libhatq.so; raise if it is absent (no silent fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        if not build_if_missing:
            raise RuntimeError(f"libhatq.so not built ({path}); run __graft_entry__.build()")
        _build.build()
    L = ctypes.CDLL(path)
    P, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    L.hatq_status_string.argtypes = [i32]
    L.hatq_status_string.restype = ctypes.c_char_p
    L.hatq_conv_out_hw.argtypes = [ctypes.POINTER(ConvDesc), i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.hatq_conv_out_hw.restype = i32
    L.hatq_weights_bytes.argtypes = [ctypes.POINTER(ConvDesc), i32]
    L.hatq_weights_bytes.restype = sz
    L.hatq_prepare_weights.argtypes = [ctypes.POINTER(ConvDesc), i32, P, P, P, sz, ctypes.POINTER(Weights), P]
    L.hatq_prepare_weights.restype = i32
    L.hatq_export_weights.argtypes = [ctypes.POINTER(Weights), P, P, P, P]
    L.hatq_export_weights.restype = i32
    L.hatq_pack_weights.argtypes = [ctypes.POINTER(Weights), P]
    L.hatq_pack_weights.restype = i32
    L.hatq_fwht_quant_ws_bytes.argtypes = [i32]
    L.hatq_fwht_quant_ws_bytes.restype = sz
    L.hatq_fwht_quant_act.argtypes = [P, i32, i32, i32, i32, i32, P, P, P, P, sz, P]
    L.hatq_fwht_quant_act.restype = i32
    L.hatq_fwht_quant_act_noalloc.argtypes = [P, i32, i32, i32, i32, i32, P, P, P]
    L.hatq_fwht_quant_act_noalloc.restype = i32
    L.hatq_fwht_quant_act_c64.argtypes = [P, i32, i32, i32, i32, i32, P, P, P, P, sz, P]
    L.hatq_fwht_quant_act_c64.restype = i32
    L.hatq_conv_int8.argtypes = [ctypes.POINTER(Weights), P, P, i32, i32, i32, i32, P, P, i32, P, i32, P]
    L.hatq_conv_int8.restype = i32
    L.hatq_conv_int8_requant.argtypes = [ctypes.POINTER(Weights), P, P, i32, i32, i32, i32, P, P, P, i32, P]
    L.hatq_conv_int8_requant.restype = i32
    L.hatq_int_table_len.argtypes = [ctypes.POINTER(Weights)]
    L.hatq_int_table_len.restype = sz
    L.hatq_int_transition_params.argtypes = [ctypes.POINTER(Weights), ctypes.c_float, ctypes.c_float, i32, P, P]
    L.hatq_int_transition_params.restype = i32
    L.hatq_conv_int8_int_transition.argtypes = [ctypes.POINTER(Weights), P, i32, i32, i32, i32, P, P, i32, P]
    L.hatq_conv_int8_int_transition.restype = i32
    L.hatq_range_expansion.argtypes = [P, i32, i32, i32, i32, i32, P, P, P, P]
    L.hatq_fwht_quant_affine_ws_bytes.argtypes = [i32]
    L.hatq_fwht_quant_affine_ws_bytes.restype = sz
    L.hatq_fwht_quant_act_affine.argtypes = [P, i32, i32, i32, i32, i32, P, P, P, P, sz, P]
    L.hatq_fwht_quant_act_affine.restype = i32
    L.hatq_tapsum_len.argtypes = [ctypes.POINTER(Weights)]
    L.hatq_tapsum_len.restype = sz
    L.hatq_weight_tapsums.argtypes = [ctypes.POINTER(Weights), P, P]
    L.hatq_weight_tapsums.restype = i32
    L.hatq_conv_int8_affine.argtypes = [ctypes.POINTER(Weights), P, P, P, P, i32, i32, i32, i32, P, P]
    L.hatq_conv_int8_affine.restype = i32
    L.hatq_range_expansion.restype = i32
    L.hatq_select_form.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_double, ctypes.POINTER(i32)]
    L.hatq_select_form.restype = i32
    L.hatq_hadamard_order.argtypes = [i32]
    L.hatq_hadamard_order.restype = i32
    L.hatq_layer_ws_bytes.argtypes = [ctypes.POINTER(Weights), i32, i32, i32]
    L.hatq_layer_ws_bytes.restype = sz
    L.hatq_layer_forward.argtypes = [ctypes.POINTER(Weights), i32, P, i32, i32, i32, P, P, P, i32, P, P,
                                     sz, P]
    L.hatq_layer_forward.restype = i32
    _lib = L
    return L


def status_string(s: int) -> str:
    return load().hatq_status_string(int(s)).decode()


def _check(status: int, where: str):
    if status != HATQ_OK:
        raise HatqError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def _need(t: Optional[torch.Tensor], name: str, dtype: torch.dtype, numel: int, optional: bool = False):
    """Raise ValueError unless t is a contiguous device tensor of `dtype` with at
    least `numel` elements (the library trusts the pointers it is given)."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name}: tensor required")
    if not t.is_cuda:
        raise ValueError(f"{name}: device tensor expected")
    if t.dtype != dtype:
        raise ValueError(f"{name}: {dtype} expected, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: contiguous tensor expected")
    if t.numel() < numel:
        raise ValueError(f"{name}: {numel} elements needed, got {t.numel()}")


def _nhwc(t: torch.Tensor, name: str, dtype: torch.dtype, channels: Optional[int] = None):
    if t.dim() != 4:
        raise ValueError(f"{name}: NHWC tensor expected, got shape {tuple(t.shape)}")
    if channels is not None and t.shape[3] != channels:
        raise ValueError(f"{name}: {channels} channels expected, got {t.shape[3]}")
    _need(t, name, dtype, 0)
    return t.shape


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def desc(cin, cout, k, stride, pad, hblock, transposed=False, out_pad=0) -> ConvDesc:
    return ConvDesc(int(cin), int(cout), int(k), int(stride), int(pad), int(out_pad),
                    int(bool(transposed)), int(hblock))


def hatq_conv_out_hw(d: ConvDesc, h: int, w: int) -> Tuple[int, int]:
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    _check(load().hatq_conv_out_hw(ctypes.byref(d), h, w, ctypes.byref(ho), ctypes.byref(wo)),
           "hatq_conv_out_hw")
    return ho.value, wo.value


def hatq_weights_bytes(d: ConvDesc, form) -> int:
    return int(load().hatq_weights_bytes(ctypes.byref(d), FORMS.get(form, form)))


@dataclass
class PreparedLayer:
    """Prepared weights of one layer: the device buffer and the C view into it."""
    buf: torch.Tensor
    w: Weights
    form: int

    @property
    def cout_pad(self) -> int:
        return self.w.cout_pad

    @property
    def cin_pad(self) -> int:
        return self.w.cin_pad

    @property
    def k_stride(self) -> int:
        return self.w.k_stride

    def wq(self) -> torch.Tensor:
        """int8 [cout_pad, k_stride] view of the packed codes."""
        n = self.w.cout_pad * self.w.k_stride
        return self.buf[:n].view(self.w.cout_pad, self.w.k_stride)

    def w_scale(self) -> torch.Tensor:
        off = self.w.w_scale - self.buf.data_ptr()
        return self.buf[off:off + 4 * self.w.cout_pad].view(torch.float32)

    def bias(self) -> torch.Tensor:
        off = self.w.bias - self.buf.data_ptr()
        return self.buf[off:off + 4 * self.w.cout_pad].view(torch.float32)

    def wpack(self) -> torch.Tensor:
        """int8 [pack_stride/64, cout_pad, 64] view of the kernel-order copy."""
        off = self.w.wpack - self.buf.data_ptr()
        n = self.w.cout_pad * self.w.pack_stride
        return self.buf[off:off + n].view(self.w.pack_stride // 64, self.w.cout_pad, 64)


def hatq_prepare_weights(d: ConvDesc, form, w: torch.Tensor, bias: Optional[torch.Tensor] = None,
                         stream=None) -> PreparedLayer:
    f = FORMS.get(form, form)
    nbytes = hatq_weights_bytes(d, f)
    if nbytes == 0:
        raise HatqError(HATQ_EINVAL, "hatq_weights_bytes")
    buf = torch.zeros(nbytes, dtype=torch.int8, device=w.device)
    out = Weights()
    w = w.contiguous().float()
    b = None if bias is None else bias.contiguous().float()
    _need(w, "w", torch.float32, d.cout * d.cin * d.k * d.k)
    _need(b, "bias", torch.float32, d.cout, optional=True)
    _check(load().hatq_prepare_weights(ctypes.byref(d), f, _ptr(w), _ptr(b), _ptr(buf), nbytes,
                                       ctypes.byref(out), _stream(stream)), "hatq_prepare_weights")
    return PreparedLayer(buf, out, f)


def hatq_export_weights(layer: PreparedLayer, stream=None):
    """Host copies of the prepared operator: (codes int8 [cout_pad, k, k, cin_pad],
    w_scale fp32 [cout_pad], bias fp32 [cout_pad]); waits for the stream."""
    k, cp, co = layer.w.d.k, layer.w.cin_pad, layer.w.cout_pad
    wq = torch.empty((co, k, k, cp), dtype=torch.int8, pin_memory=True)
    sc = torch.empty(co, dtype=torch.float32, pin_memory=True)
    b = torch.empty(co, dtype=torch.float32, pin_memory=True)
    s = stream if stream is not None else torch.cuda.current_stream()
    _check(load().hatq_export_weights(ctypes.byref(layer.w), ctypes.c_void_p(wq.data_ptr()),
                                      ctypes.c_void_p(sc.data_ptr()), ctypes.c_void_p(b.data_ptr()), _stream(s)),
           "hatq_export_weights")
    s.synchronize()
    return wq, sc, b


def hatq_pack_weights(layer: PreparedLayer, stream=None) -> None:
    """Rebuild the kernel-order copy after codes were written into ``layer.wq()``."""
    _check(load().hatq_pack_weights(ctypes.byref(layer.w), _stream(stream)), "hatq_pack_weights")


def hatq_fwht_quant_act(x: torch.Tensor, hblock: int, absmax: Optional[torch.Tensor] = None,
                        xq: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """x fp32 NHWC -> (int8 codes NHWC, per-sample scale fp32 [n]).  Output and
    workspace tensors may be passed in to avoid allocation."""
    n, h, w, c = _nhwc(x, "x", torch.float32)
    if xq is None:
        xq = torch.empty((n, h, w, c), dtype=torch.int8, device=x.device)
    sc = scale if scale is not None else torch.empty(n, dtype=torch.float32, device=x.device)
    _need(xq, "xq", torch.int8, x.numel())
    _need(sc, "scale", torch.float32, n)
    _need(absmax, "absmax", torch.float32, n, optional=True)
    wsb = int(load().hatq_fwht_quant_ws_bytes(n))
    if ws is None:
        ws = torch.empty(max(wsb, 4), dtype=torch.int8, device=x.device)
    _need(ws, "ws", torch.int8, 0)
    wsb = ws.numel()
    _check(load().hatq_fwht_quant_act(_ptr(x), n, h, w, c, int(hblock), _ptr(absmax), _ptr(xq), _ptr(sc),
                                      _ptr(ws), wsb, _stream(stream)), "hatq_fwht_quant_act")
    return xq, sc


HATQ_NOALLOC_MAX_SAMPLES = 4096


def hatq_fwht_quant_act_noalloc(x: torch.Tensor, hblock: int, xq: torch.Tensor, scale: torch.Tensor,
                                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """hatq_fwht_quant_act (two passes) with the library's static scratch: the
    caller passes the outputs; nothing is allocated."""
    n, h, w, c = _nhwc(x, "x", torch.float32)
    _need(xq, "xq", torch.int8, x.numel())
    _need(scale, "scale", torch.float32, n)
    _check(load().hatq_fwht_quant_act_noalloc(_ptr(x), n, h, w, c, int(hblock), _ptr(xq), _ptr(scale),
                                              _stream(stream)), "hatq_fwht_quant_act_noalloc")
    return xq, scale


def hatq_fwht_quant_act_c64(x: torch.Tensor, hblock: int, absmax: Optional[torch.Tensor] = None,
                            xq: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                            ws: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """hatq_fwht_quant_act with the codes chunk-major: int8 [n, c/64, h, w, 64]."""
    n, h, w, c = _nhwc(x, "x", torch.float32)
    if c % 64:
        raise HatqError(HATQ_EUNSUPPORTED, "hatq_fwht_quant_act_c64 (c % 64)")
    if xq is None:
        xq = torch.empty((n, c // 64, h, w, 64), dtype=torch.int8, device=x.device)
    sc = scale if scale is not None else torch.empty(n, dtype=torch.float32, device=x.device)
    _need(xq, "xq", torch.int8, x.numel())
    _need(sc, "scale", torch.float32, n)
    _need(absmax, "absmax", torch.float32, n, optional=True)
    if ws is None:
        ws = torch.empty(max(int(load().hatq_fwht_quant_ws_bytes(n)), 4), dtype=torch.int8, device=x.device)
    _need(ws, "ws", torch.int8, 0)
    _check(load().hatq_fwht_quant_act_c64(_ptr(x), n, h, w, c, int(hblock), _ptr(absmax), _ptr(xq), _ptr(sc),
                                          _ptr(ws), ws.numel(), _stream(stream)), "hatq_fwht_quant_act_c64")
    return xq, sc


def to_c64(q: torch.Tensor) -> torch.Tensor:
    """NHWC codes [n, h, w, c] -> chunk-major [n, c/64, h, w, 64] (a copy)."""
    n, h, w, c = q.shape
    return q.view(n, h, w, c // 64, 64).permute(0, 3, 1, 2, 4).contiguous()


def from_c64(q: torch.Tensor) -> torch.Tensor:
    """Chunk-major codes [n, c/64, h, w, 64] -> NHWC [n, h, w, c] (a copy)."""
    n, m, h, w, _ = q.shape
    return q.permute(0, 2, 3, 1, 4).reshape(n, h, w, m * 64).contiguous()


def _codes_in(xq: torch.Tensor, cin_pad: int):
    """(n, h, w, flag) of a layer's input codes: NHWC [n, h, w, cin_pad], or
    chunk-major [n, cin_pad/64, h, w, 64] (HATQ_XQ_C64)."""
    if xq.dim() == 5:
        n, m, h, w, c64 = xq.shape
        if m * 64 != cin_pad or c64 != 64:
            raise ValueError(f"xq: chunk-major shape {tuple(xq.shape)} for cin_pad {cin_pad}")
        _need(xq, "xq", torch.int8, n * h * w * cin_pad)
        return n, h, w, HATQ_XQ_C64
    n, h, w, _ = _nhwc(xq, "xq", torch.int8, cin_pad)
    return n, h, w, 0


def _codes_out_shape(n: int, ho: int, wo: int, c: int, c64: bool):
    return (n, c // 64, ho, wo, 64) if c64 else (n, ho, wo, c)


def _flags(paired: bool) -> int:
    return HATQ_PAIRED if paired else 0


def hatq_conv_int8(layer: PreparedLayer, xq: torch.Tensor, act_scale: torch.Tensor, out_mode=HATQ_OUT_F32,
                   next_hblock: int = 0, next_absmax: Optional[torch.Tensor] = None, y=None, stream=None,
                   absmax_only: bool = False, out_scale: Optional[torch.Tensor] = None, paired: bool = False,
                   yq_c64: bool = False):
    """absmax_only: F32 mode with y = NULL, producing next_absmax alone (returns None).
    out_mode HATQ_OUT_I8: y receives the next operand's codes with the static
    per-sample scale out_scale (chunk-major with yq_c64).  paired: the
    HATQ_PAIRED flag.  A 5-d xq is chunk-major (HATQ_XQ_C64)."""
    n, h, w, xf = _codes_in(xq, layer.w.cin_pad)
    fl = _flags(paired) | xf | (HATQ_YQ_C64 if yq_c64 else 0)
    _need(act_scale, "act_scale", torch.float32, n)
    _need(next_absmax, "next_absmax", torch.float32, n, optional=True)
    _need(out_scale, "out_scale", torch.float32, n, optional=True)
    ho, wo = hatq_conv_out_hw(layer.w.d, h, w)
    if absmax_only:
        _check(load().hatq_conv_int8(ctypes.byref(layer.w), _ptr(xq), _ptr(act_scale), n, h, w, int(out_mode),
                                     _ptr(out_scale), None, int(next_hblock), _ptr(next_absmax), fl,
                                     _stream(stream)),
               "hatq_conv_int8")
        return None
    if out_mode == HATQ_OUT_I32:
        shape, dt = (n, ho, wo, layer.w.cout_pad), torch.int32
    elif out_mode == HATQ_OUT_I8:
        shape, dt = _codes_out_shape(n, ho, wo, layer.w.d.cout, yq_c64), torch.int8
    else:
        shape, dt = (n, ho, wo, layer.w.d.cout), torch.float32
    if y is None:
        y = torch.empty(shape, dtype=dt, device=xq.device)
    _need(y, "y", dt, n * ho * wo * (layer.w.cout_pad if out_mode == HATQ_OUT_I32 else layer.w.d.cout))
    _check(load().hatq_conv_int8(ctypes.byref(layer.w), _ptr(xq), _ptr(act_scale), n, h, w, int(out_mode),
                                 _ptr(out_scale), _ptr(y), int(next_hblock), _ptr(next_absmax), fl,
                                 _stream(stream)),
           "hatq_conv_int8")
    return y


def hatq_conv_int8_requant(layer: PreparedLayer, xq: torch.Tensor, act_scale: torch.Tensor, next_hblock: int,
                           next_absmax: Optional[torch.Tensor] = None, next_scale: Optional[torch.Tensor] = None,
                           yq: Optional[torch.Tensor] = None, stream=None, paired: bool = False,
                           yq_c64: bool = False):
    """Conv with the requantizing epilogue: returns (yq, next_scale), the next
    layer's codes (chunk-major with yq_c64) and scale.  A 5-d xq is chunk-major."""
    n, h, w, xf = _codes_in(xq, layer.w.cin_pad)
    _need(act_scale, "act_scale", torch.float32, n)
    _need(next_absmax, "next_absmax", torch.float32, n, optional=True)
    ho, wo = hatq_conv_out_hw(layer.w.d, h, w)
    if yq is None:
        yq = torch.empty(_codes_out_shape(n, ho, wo, layer.w.d.cout, yq_c64), dtype=torch.int8, device=xq.device)
    if next_scale is None:
        next_scale = torch.empty((n,), dtype=torch.float32, device=xq.device)
    _need(yq, "yq", torch.int8, n * ho * wo * layer.w.d.cout)
    _need(next_scale, "next_scale", torch.float32, n)
    _check(load().hatq_conv_int8_requant(ctypes.byref(layer.w), _ptr(xq), _ptr(act_scale), n, h, w,
                                         int(next_hblock), _ptr(next_absmax), _ptr(next_scale), _ptr(yq),
                                         _flags(paired) | xf | (HATQ_YQ_C64 if yq_c64 else 0), _stream(stream)),
           "hatq_conv_int8_requant")
    return yq, next_scale


def hatq_int_table_len(layer: PreparedLayer) -> int:
    return int(load().hatq_int_table_len(ctypes.byref(layer.w)))


def hatq_int_transition_params(layer: PreparedLayer, s_x: float, s_y: float, next_hblock: int,
                               table: Optional[torch.Tensor] = None, device="cuda", stream=None):
    """Integer transition table (M, b_int, shift) from static scales: returns
    (table, shift).  The library call does not wait; this wrapper reads the shift
    back (-1: none fits, then the call is reported as HATQ_EUNSUPPORTED here)."""
    if table is None:
        table = torch.empty((hatq_int_table_len(layer),), dtype=torch.int32, device=device)
    _need(table, "table", torch.int32, hatq_int_table_len(layer))
    _check(load().hatq_int_transition_params(ctypes.byref(layer.w), float(s_x), float(s_y), int(next_hblock),
                                             _ptr(table), _stream(stream)),
           "hatq_int_transition_params")
    shift = int(table[2 * layer.w.cout_pad].item())
    if shift < 0:
        raise HatqError(HATQ_EUNSUPPORTED, "hatq_int_transition_params (no shift fits)")
    return table, shift


def hatq_conv_int8_int_transition(layer: PreparedLayer, xq: torch.Tensor, next_hblock: int, table: torch.Tensor,
                                  yq: Optional[torch.Tensor] = None, stream=None, paired: bool = False,
                                  yq_c64: bool = False) -> torch.Tensor:
    """Conv with the integer-only epilogue: the next layer's codes (chunk-major
    with yq_c64).  A 5-d xq is chunk-major."""
    n, h, w, xf = _codes_in(xq, layer.w.cin_pad)
    _need(table, "table", torch.int32, hatq_int_table_len(layer))
    ho, wo = hatq_conv_out_hw(layer.w.d, h, w)
    if yq is None:
        yq = torch.empty(_codes_out_shape(n, ho, wo, layer.w.d.cout, yq_c64), dtype=torch.int8, device=xq.device)
    _need(yq, "yq", torch.int8, n * ho * wo * layer.w.d.cout)
    _check(load().hatq_conv_int8_int_transition(ctypes.byref(layer.w), _ptr(xq), n, h, w, int(next_hblock),
                                                _ptr(table), _ptr(yq), _flags(paired) | xf |
                                                (HATQ_YQ_C64 if yq_c64 else 0), _stream(stream)),
           "hatq_conv_int8_int_transition")
    return yq


def hatq_fwht_quant_act_affine(x: torch.Tensor, hblock: int, xq: Optional[torch.Tensor] = None,
                               scale: Optional[torch.Tensor] = None, zero: Optional[torch.Tensor] = None,
                               ws: Optional[torch.Tensor] = None, stream=None):
    """x fp32 NHWC -> (int8 codes, per-sample scale fp32 [n], zero point int32 [n])."""
    n, h, w, c = _nhwc(x, "x", torch.float32)
    if xq is None:
        xq = torch.empty((n, h, w, c), dtype=torch.int8, device=x.device)
    if scale is None:
        scale = torch.empty(n, dtype=torch.float32, device=x.device)
    if zero is None:
        zero = torch.empty(n, dtype=torch.int32, device=x.device)
    if ws is None:
        ws = torch.empty(int(load().hatq_fwht_quant_affine_ws_bytes(n)), dtype=torch.int8, device=x.device)
    _need(xq, "xq", torch.int8, x.numel())
    _need(scale, "scale", torch.float32, n)
    _need(zero, "zero", torch.int32, n)
    _need(ws, "ws", torch.int8, 0)
    _check(load().hatq_fwht_quant_act_affine(_ptr(x), n, h, w, c, int(hblock), _ptr(xq), _ptr(scale), _ptr(zero),
                                             _ptr(ws), ws.numel(), _stream(stream)), "hatq_fwht_quant_act_affine")
    return xq, scale, zero


def hatq_weight_tapsums(layer: PreparedLayer, tapsum: Optional[torch.Tensor] = None, device="cuda", stream=None):
    need = int(load().hatq_tapsum_len(ctypes.byref(layer.w)))
    if tapsum is None:
        tapsum = torch.empty(need, dtype=torch.int32, device=device)
    _need(tapsum, "tapsum", torch.int32, need)
    _check(load().hatq_weight_tapsums(ctypes.byref(layer.w), _ptr(tapsum), _stream(stream)), "hatq_weight_tapsums")
    return tapsum


def hatq_conv_int8_affine(layer: PreparedLayer, xq: torch.Tensor, act_scale: torch.Tensor, act_zero: torch.Tensor,
                          tapsum: torch.Tensor, out_mode=HATQ_OUT_F32, y=None, stream=None) -> torch.Tensor:
    n, h, w, _ = _nhwc(xq, "xq", torch.int8, layer.w.cin_pad)
    _need(act_scale, "act_scale", torch.float32, n)
    _need(act_zero, "act_zero", torch.int32, n)
    _need(tapsum, "tapsum", torch.int32, int(load().hatq_tapsum_len(ctypes.byref(layer.w))))
    ho, wo = hatq_conv_out_hw(layer.w.d, h, w)
    if out_mode == HATQ_OUT_I32:
        shape, dt = (n, ho, wo, layer.w.cout_pad), torch.int32
    else:
        shape, dt = (n, ho, wo, layer.w.d.cout), torch.float32
    if y is None:
        y = torch.empty(shape, dtype=dt, device=xq.device)
    _need(y, "y", dt, n * ho * wo * shape[3])
    _check(load().hatq_conv_int8_affine(ctypes.byref(layer.w), _ptr(xq), _ptr(act_scale), _ptr(act_zero),
                                        _ptr(tapsum), n, h, w, int(out_mode), _ptr(y), _stream(stream)),
           "hatq_conv_int8_affine")
    return y


def hatq_range_expansion(x: torch.Tensor, hblock: int, amax: Optional[torch.Tensor] = None,
                         flags: Optional[torch.Tensor] = None, count: Optional[torch.Tensor] = None,
                         stream=None):
    """Per-sample range-expansion indicator of x (fp32 NHWC): returns (amax [2n], flags [n]).
    count, if given, accumulates the number of expanding samples."""
    n, h, w, c = _nhwc(x, "x", torch.float32)
    if amax is None:
        amax = torch.empty(2 * n, dtype=torch.float32, device=x.device)
    if flags is None:
        flags = torch.empty(n, dtype=torch.int32, device=x.device)
    _need(amax, "amax", torch.float32, 2 * n)
    _need(flags, "flags", torch.int32, n)
    _need(count, "count", torch.int32, 1, optional=True)
    _check(load().hatq_range_expansion(_ptr(x), n, h, w, c, int(hblock), _ptr(amax), _ptr(flags), _ptr(count),
                                       _stream(stream)), "hatq_range_expansion")
    return amax, flags


def hatq_select_form(expansions: int, images: int, tau: float = 0.8) -> str:
    f = ctypes.c_int32(-1)
    _check(load().hatq_select_form(int(expansions), int(images), float(tau), ctypes.byref(f)), "hatq_select_form")
    return "WH" if f.value == HATQ_WH else "DH"


def hatq_hadamard_order(c: int) -> int:
    """m(c) of the transform order rule (0: c outside [1, 4096])."""
    return int(load().hatq_hadamard_order(int(c)))


def hatq_layer_ws_bytes(layer: PreparedLayer, n: int, h: int, w: int) -> int:
    return int(load().hatq_layer_ws_bytes(ctypes.byref(layer.w), n, h, w))


def hatq_layer_forward(layer: PreparedLayer, form, x: torch.Tensor, x_absmax: Optional[torch.Tensor] = None,
                       next_hblock: int = 0, next_absmax: Optional[torch.Tensor] = None,
                       act_scale: Optional[torch.Tensor] = None, y: Optional[torch.Tensor] = None,
                       ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    n, h, w, _ = _nhwc(x, "x", torch.float32, layer.w.d.cin)
    _need(x_absmax, "x_absmax", torch.float32, n, optional=True)
    _need(next_absmax, "next_absmax", torch.float32, n, optional=True)
    _need(act_scale, "act_scale", torch.float32, n, optional=True)
    ho, wo = hatq_conv_out_hw(layer.w.d, h, w)
    if y is None:
        y = torch.empty((n, ho, wo, layer.w.d.cout), dtype=torch.float32, device=x.device)
    _need(y, "y", torch.float32, n * ho * wo * layer.w.d.cout)
    need = hatq_layer_ws_bytes(layer, n, h, w)
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.int8, device=x.device)
    _need(ws, "ws", torch.int8, 0)
    _check(load().hatq_layer_forward(ctypes.byref(layer.w), FORMS.get(form, form), _ptr(x), n, h, w,
                                     _ptr(x_absmax), _ptr(y), _ptr(act_scale), int(next_hblock),
                                     _ptr(next_absmax), _ptr(ws), ws.numel(), _stream(stream)),
           "hatq_layer_forward")
    return y
