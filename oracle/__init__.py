"""CPU oracle for the HaTQ Hadamard-domain INT8 linear operator.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product package.  It shares no code
with the HIP library.  The arithmetic lives in ``hatq_oracle.c`` (plain C, fp64
sums, IEEE fp32 division, RNE); this file only marshals numpy arrays and composes
the per-step functions in the order the paper gives them:

    activation operand (DH: S = B_C x; WH: S = x)       Eq. input_hadamard_transform
    per-sample symmetric INT8 quantization               Eq. symmetric_q, Eq. current_scale
    (or affine: scale and zero point from min / max)     Eq. uniform_q, Eq. affine_q
    INT8 x INT8 -> INT32 direct convolution              Eq. integer_accumulation
    dequant (s_x s_w,c / b), bias, WH basis restore      Eq. accumulator_scale,
                                                         Eq. supp_padded_dh, Eq. supp_padded_wh
    integer-only transition (M, b_int, shift; int64)     Eq. integer_fixed_point_scale,
                                                         Eq. integer_hadamard_transition
    range-expansion statistic and the DH/WH rule         Eq. hadamard_sensitivity,
                                                         Eq. layerwise_hadamard_selection
    Paley / Kronecker orders and the order rule          Eq. hadamard_order,
                                                         Eq. supp_hadamard_order

Parity status: every function is pinned by the CPU tests (identities of the
Hadamard matrix, a library special case for the convolution, function
preservation of the unquantized layer, the quantizer's own invariants and a
quantization-error bound).  The exact quantized values of a full layer have no
printed worked example in the paper; they are pinned only through those
properties.  The free-running multi-layer stack beyond teacher-forced layers is
parity unpinned (a report, not a gate).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hatq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2 -fopenmp -ffp-contract=off, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                               "-std=c11", "-Wall", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int, ctypes.c_int64
        L.orc_set_threads.argtypes = [i32]
        L.orc_sylvester.argtypes = [i32, P]
        L.orc_block_transform_f64.argtypes = [i32, P, P, i64, i32]
        L.orc_activation_transform.argtypes = [P, i64, i32, i32, P]
        L.orc_quantize_symmetric.argtypes = [P, i64, i64, P, P]
        L.orc_quantize_symmetric.restype = None
        L.orc_prepare_weights.argtypes = [i32, i32, i32, i32, i32, i32, P, P, P, P, P, P]
        L.orc_out_size.argtypes = [i32, i32, i32, i32, i32, i32]
        L.orc_conv_int8.argtypes = [P, P, i32, i32, i32, i32, P, i32, i32, i32, i32, i32, i32, P]
        L.orc_quantize_affine.argtypes = [P, i64, i64, P, P, P]
        L.orc_conv_int8.restype = None
        L.orc_conv_f64.argtypes = [P, i32, i32, i32, i32, P, i32, i32, i32, i32, i32, i32, P]
        L.orc_conv_f64.restype = None
        L.orc_epilogue.argtypes = [P, i32, i64, i32, i32, i32, i32, P, P, P, P]
        L.orc_int_requant_params.argtypes = [i32, ctypes.c_float, P, P, ctypes.c_float, i32, i32, i32, i32, P, P]
        L.orc_int_transition.argtypes = [P, i64, i32, i32, P, P, i32, i32, i32, P]
        L.orc_range_expansion.argtypes = [P, i32, i64, i32, i32, P, P, P]
        L.orc_paley.argtypes = [i32, i32, P]
        L.orc_wh_z.argtypes = [P, i32, i64, i32, P, P, P, P]
        L.orc_hadamard.argtypes = [i32, P]
        L.orc_hadamard_base.argtypes = [i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.orc_order.argtypes = [i32, i32]
        L.orc_hadamard_split.argtypes = [i32]
        L.orc_select_form.argtypes = [i64, i64, ctypes.c_double]
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def set_threads(n: int = 0) -> int:
    """Set the OpenMP thread count of the oracle's loops (n <= 0: leave it);
    returns the count in effect."""
    return int(lib().orc_set_threads(int(n)))


def round_up(v: int, m: int) -> int:
    return (v + m - 1) // m * m


# --------------------------------------------------------------------------
# O1  Hadamard matrix (Eq. supp_sylvester)
# --------------------------------------------------------------------------
def sylvester(b: int) -> np.ndarray:
    H = np.zeros((b, b), np.int8)
    if lib().orc_sylvester(b, _p(H)) != 0:
        raise ValueError(f"Sylvester order must be a power of two, got {b}")
    return H


def block_transform_f64(x: np.ndarray, b: int) -> np.ndarray:
    """Dense B_C along the last axis in fp64 (width must be a multiple of b)."""
    x = _c(x, np.float64)
    out = np.empty_like(x)
    width = x.shape[-1]
    if lib().orc_block_transform_f64(b, _p(x), _p(out), x.size // width, width) != 0:
        raise ValueError("bad block size")
    return out


# --------------------------------------------------------------------------
# O3  Activation operand and quantizer
# --------------------------------------------------------------------------
def activation_transform(x: np.ndarray, b: int) -> np.ndarray:
    """S = fl32(B_C x_pad) per pixel (b = 1 gives S = x)."""
    x = _c(x, np.float32)
    C = x.shape[-1]
    Cp = round_up(C, b)
    S = np.empty(x.shape[:-1] + (Cp,), np.float32)
    if lib().orc_activation_transform(_p(x), x.size // C, C, b, _p(S)) != 0:
        raise ValueError("bad block size")
    return S


def quantize_symmetric(S: np.ndarray, per_sample: bool = True):
    """Codes and scale(s) of Eq. symmetric_q; one scale per leading-axis sample."""
    S = _c(S, np.float32)
    nsamp = S.shape[0] if per_sample else 1
    q = np.empty(S.shape, np.int8)
    s = np.empty(nsamp, np.float32)
    lib().orc_quantize_symmetric(_p(S), nsamp, S.size // nsamp, _p(q), _p(s))
    return q, s


def quantize_affine(S: np.ndarray, per_sample: bool = True):
    """Codes, scale(s) and zero point(s) of Eq. affine_q / Eq. uniform_q on the
    signed grid [-128, 127]; one (s, z) per leading-axis sample."""
    S = _c(S, np.float32)
    nsamp = S.shape[0] if per_sample else 1
    q = np.empty(S.shape, np.int8)
    s = np.empty(nsamp, np.float32)
    z = np.empty(nsamp, np.int32)
    lib().orc_quantize_affine(_p(S), nsamp, S.size // nsamp, _p(q), _p(s), _p(z))
    return q, s, z


def activation_operand(x: np.ndarray, form: str, hblock: int):
    """Steps a2-a4: (S, codes, per-sample scale)."""
    S = activation_transform(x, hblock if form == "DH" else 1)
    q, s = quantize_symmetric(S)
    return S, q, s


# --------------------------------------------------------------------------
# O2  Weights
# --------------------------------------------------------------------------
@dataclass
class PreparedWeights:
    wq: np.ndarray        # [cout_p, k, k, cin_p] int8 (OHWI)
    w_scale: np.ndarray   # [cout_p] fp32
    w_bias: np.ndarray    # [cout_p] fp32 (transformed for WH)
    w_real: np.ndarray    # [cout_p, k, k, cin_p] fp32, unquantized W'
    cin: int
    cout: int
    cin_p: int
    cout_p: int
    k: int
    stride: int
    pad: int
    transposed: bool
    out_pad: int
    form: str
    hblock: int


def prepare_weights(w: np.ndarray, bias: Optional[np.ndarray], *, cin, cout, k, stride, pad,
                    form, hblock, transposed=False, out_pad=0) -> PreparedWeights:
    w = _c(w, np.float32)
    b = None if bias is None else _c(bias, np.float32)
    fcode = {"DH": 0, "WH": 1}[form]
    cin_p = round_up(cin, hblock) if form == "DH" else cin
    cout_p = round_up(cout, hblock) if form == "WH" else cout
    wq = np.empty((cout_p, k, k, cin_p), np.int8)
    wr = np.empty((cout_p, k, k, cin_p), np.float32)
    ws = np.empty(cout_p, np.float32)
    wb = np.empty(cout_p, np.float32)
    rc = lib().orc_prepare_weights(cin, cout, k, int(transposed), hblock, fcode, _p(w), _p(b),
                                   _p(wq), _p(ws), _p(wb), _p(wr))
    if rc != 0:
        raise ValueError("bad weight descriptor")
    return PreparedWeights(wq, ws, wb, wr, cin, cout, cin_p, cout_p, k, stride, pad,
                           bool(transposed), out_pad, form, hblock)


# --------------------------------------------------------------------------
# O4  Convolution
# --------------------------------------------------------------------------
def out_size(n_in, k, stride, pad, transposed=False, out_pad=0) -> int:
    return lib().orc_out_size(n_in, k, stride, pad, int(transposed), out_pad)


def conv_int8(xq: np.ndarray, wq: np.ndarray, *, stride, pad, transposed=False, out_pad=0, zx=None):
    """Direct INT8 conv, INT32 accumulate.  xq NHWC [n,h,w,cin_p], wq OHWI;
    zx: per-sample activation zero points (affine codes), or None."""
    xq = _c(xq, np.int8)
    wq = _c(wq, np.int8)
    n, h, w, cin_p = xq.shape
    cout_p, k, k2, cin_w = wq.shape
    assert k == k2 and cin_w == cin_p
    ho = out_size(h, k, stride, pad, transposed, out_pad)
    wo = out_size(w, k, stride, pad, transposed, out_pad)
    acc = np.empty((n, ho, wo, cout_p), np.int32)
    zxa = None if zx is None else _c(zx, np.int32)
    assert zxa is None or zxa.shape == (n,)
    lib().orc_conv_int8(_p(xq), _p(zxa), n, h, w, cin_p, _p(wq), cout_p, k, stride, pad,
                        int(transposed), out_pad, _p(acc))
    return acc


def conv_f64(x: np.ndarray, w_ohwi: np.ndarray, *, stride, pad, transposed=False, out_pad=0):
    x = _c(x, np.float64)
    w_ohwi = _c(w_ohwi, np.float64)
    n, h, w, cin = x.shape
    cout, k, _, _ = w_ohwi.shape
    ho = out_size(h, k, stride, pad, transposed, out_pad)
    wo = out_size(w, k, stride, pad, transposed, out_pad)
    y = np.empty((n, ho, wo, cout), np.float64)
    lib().orc_conv_f64(_p(x), n, h, w, cin, _p(w_ohwi), cout, k, stride, pad,
                       int(transposed), out_pad, _p(y))
    return y


def torch_layout_to_ohwi(w: np.ndarray, transposed: bool) -> np.ndarray:
    """OIHW (conv) or IOHW (transposed) -> OHWI, a pure relabelling of axes."""
    return np.ascontiguousarray(w.transpose(1, 2, 3, 0) if transposed else w.transpose(0, 2, 3, 1))


# --------------------------------------------------------------------------
# O5  Epilogue and O6 layer composition
# --------------------------------------------------------------------------
def epilogue(acc: np.ndarray, sx: np.ndarray, pw: PreparedWeights) -> np.ndarray:
    acc = _c(acc, np.int32)
    n = acc.shape[0]
    pix = acc.size // (n * pw.cout_p)
    y = np.empty(acc.shape[:-1] + (pw.cout,), np.float32)
    rc = lib().orc_epilogue(_p(acc), n, pix, pw.cout, pw.cout_p, {"DH": 0, "WH": 1}[pw.form],
                            pw.hblock, _p(_c(sx, np.float32)), _p(pw.w_scale), _p(pw.w_bias), _p(y))
    if rc != 0:
        raise ValueError("bad epilogue geometry")
    return y


def wh_z(acc: np.ndarray, sx: np.ndarray, pw: PreparedWeights) -> np.ndarray:
    """A WH layer's dequantized accumulators before the output restore
    [.., cout_p]: the next operand when the next transform uses the same blocks
    (B_next y = z exactly, Table I)."""
    assert pw.form == "WH"
    acc = _c(acc, np.int32)
    n = acc.shape[0]
    pix = acc.size // (n * pw.cout_p)
    z = np.empty(acc.shape, np.float32)
    lib().orc_wh_z(_p(acc), n, pix, pw.cout_p, _p(_c(sx, np.float32)), _p(pw.w_scale), _p(pw.w_bias), _p(z))
    return z


@dataclass
class LayerResult:
    S: np.ndarray
    xq: np.ndarray
    sx: np.ndarray
    acc: np.ndarray
    y: np.ndarray


def layer_forward(x: np.ndarray, pw: PreparedWeights) -> LayerResult:
    """One quantized layer: a2-a4, a5, a6."""
    S, xq, sx = activation_operand(x, pw.form, pw.hblock)
    acc = conv_int8(xq, pw.wq, stride=pw.stride, pad=pw.pad, transposed=pw.transposed,
                    out_pad=pw.out_pad)
    y = epilogue(acc, sx, pw)
    return LayerResult(S, xq, sx, acc, y)


def layer_unquantized(x: np.ndarray, pw: PreparedWeights) -> np.ndarray:
    """The same layer with quantization switched off (fp32 S and W' in place of the
    codes, fp64 contraction): by Eq. hadamard_linear_equivalence and Eq.
    weight_only_hadamard_equivalence it must equal the plain float layer."""
    S = activation_transform(x, pw.hblock if pw.form == "DH" else 1)
    acc = conv_f64(S, pw.w_real, stride=pw.stride, pad=pw.pad, transposed=pw.transposed,
                   out_pad=pw.out_pad)
    if pw.form == "DH":
        y = acc / pw.hblock + pw.w_bias[: pw.cout].astype(np.float64)
    else:
        z = acc + pw.w_bias.astype(np.float64)
        # restore with B^T (B^T B = b I): row vectors times H
        H = hadamard(pw.hblock).astype(np.float64)
        y = (z.reshape(z.shape[:-1] + (-1, pw.hblock)) @ H).reshape(z.shape)[..., : pw.cout] / pw.hblock
    return y


def float_layer(x: np.ndarray, w: np.ndarray, bias: Optional[np.ndarray], *, stride, pad,
                transposed=False, out_pad=0) -> np.ndarray:
    """The original float operator Y = X W^T + b, fp64 (no transform, no quantizer)."""
    y = conv_f64(x, torch_layout_to_ohwi(w, transposed), stride=stride, pad=pad,
                 transposed=transposed, out_pad=out_pad)
    if bias is not None:
        y = y + bias.astype(np.float64)
    return y


# --------------------------------------------------------------------------
# O7  Integer-only inter-layer transition (static scales)
# --------------------------------------------------------------------------
@dataclass
class IntRequant:
    M: np.ndarray       # [cout_p] int32 multipliers
    b_int: np.ndarray   # [cout_p] int32 integer bias
    shift: int          # shared right shift n


def int_requant_params(pw: PreparedWeights, s_x: float, s_y: float, next_b: int) -> IntRequant:
    """Eq. integer_accumulation (b_int), Eq. integer_fixed_point_scale (M, n) for
    static input scale s_x and next-operand scale s_y (see the C source, O6)."""
    K = pw.k * pw.k * pw.cin_p
    gain = (pw.hblock if pw.form == "WH" else 1) * next_b
    M = np.empty(pw.cout_p, np.int32)
    b = np.empty(pw.cout_p, np.int32)
    beta_in, beta_out = (pw.hblock, 1) if pw.form == "DH" else (1, pw.hblock)
    n = lib().orc_int_requant_params(pw.cout_p, float(s_x), _p(pw.w_scale), _p(pw.w_bias), float(s_y),
                                     beta_in, beta_out, K, gain, _p(M), _p(b))
    if n < 0:
        raise ValueError("no shift fits the multiplier and overflow bounds")
    return IntRequant(M, b, int(n))


def int_transition(acc: np.ndarray, pw: PreparedWeights, rq: IntRequant, next_b: int) -> np.ndarray:
    """Eq. integer_hadamard_transition with phi = identity: the next layer's INT8
    operand [.., cout] from the accumulators [.., cout_p]."""
    acc = _c(acc, np.int32)
    P = acc.size // pw.cout_p
    q = np.empty(acc.shape[:-1] + (pw.cout,), np.int8)
    wb = pw.hblock if pw.form == "WH" else 1
    if lib().orc_int_transition(_p(acc), P, pw.cout, pw.cout_p, _p(_c(rq.M, np.int32)),
                                _p(_c(rq.b_int, np.int32)), rq.shift, wb, next_b, _p(q)) != 0:
        raise ValueError("bad transition geometry")
    return q


# --------------------------------------------------------------------------
# O7  Range-expansion profiling and the form rule
# --------------------------------------------------------------------------
def range_expansion(x: np.ndarray, b: int):
    """Per sample of x [n, ..., C]: (max |x|, max |fl32(B_C x_pad)|, expands)
    with expands = max|S|^2 > b max|x|^2 (Eq. hadamard_sensitivity with the
    orthonormal transform B / sqrt(b))."""
    x = _c(x, np.float32)
    n, C = x.shape[0], x.shape[-1]
    P = x.size // (n * C)
    ax = np.empty(n, np.float32)
    ah = np.empty(n, np.float32)
    fl = np.empty(n, np.int32)
    if lib().orc_range_expansion(_p(x), n, P, C, b, _p(ax), _p(ah), _p(fl)) != 0:
        raise ValueError("bad block size or shape")
    return ax, ah, fl


def select_form(expansions: int, images: int, tau: float = 0.8) -> str:
    """Eq. layerwise_hadamard_selection: "WH" if expansions / images > tau, else "DH"."""
    r = lib().orc_select_form(int(expansions), int(images), float(tau))
    if r < 0:
        raise ValueError("bad counts")
    return "WH" if r else "DH"


# --------------------------------------------------------------------------
# O8  Hadamard orders beyond powers of two
# --------------------------------------------------------------------------
def paley(q: int, kind: int) -> np.ndarray:
    """Paley-I (kind 1, q = 3 mod 4, order q + 1) or Paley-II (kind 2, q = 1 mod 4,
    order 2(q + 1)) for an odd prime power q, over the field F_q."""
    n = (q + 1) * (1 if kind == 1 else 2)
    H = np.empty((n, n), np.int8)
    if lib().orc_paley(q, kind, _p(H)) != 0:
        raise ValueError("no Paley matrix of this kind for q")
    return H


def hadamard_base(m: int):
    """(b, kind, q): the base order of the construction of order m (P_b (x) H~_(m/b))
    and its Paley kind and prime power (kind 0: b = 1, Sylvester); None if m has no
    such form (it may still be a Kronecker product, see hadamard_split)."""
    kind, q = ctypes.c_int32(), ctypes.c_int32()
    b = lib().orc_hadamard_base(m, ctypes.byref(kind), ctypes.byref(q))
    return None if b < 0 else (int(b), int(kind.value), int(q.value))


def hadamard_split(m: int):
    """The smallest factor a of an order m = a * c reached only as a Kronecker
    product H_a (x) H_c of two supported orders; None otherwise."""
    a = lib().orc_hadamard_split(m)
    return None if a < 0 else int(a)


def hadamard(m: int) -> np.ndarray:
    H = np.empty((m, m), np.int8)
    if lib().orc_hadamard(m, _p(H)) != 0:
        raise ValueError("unsupported order")
    return H


def order(C: int, mmax: int = 4096) -> int:
    """Eq. hadamard_order: the smallest supported order >= 4 ceil(C / 4)."""
    m = lib().orc_order(C, mmax)
    if m < 0:
        raise ValueError("no supported order below mmax")
    return int(m)
