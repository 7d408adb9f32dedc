"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any launch (so
these run without a GPU; the pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2608_01653_amd import hatq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x10000)   # aligned, never dereferenced: validation fails first

# These calls pass fake device pointers that validation must reject.  Never run
# them where a GPU is visible: a validation bug would then launch on garbage.
try:
    import torch
    _HAS_GPU = torch.cuda.device_count() > 0
except Exception:  # pragma: no cover
    _HAS_GPU = False
pytestmark = pytest.mark.skipif(_HAS_GPU, reason="fake-pointer validation tests run on CPU-only hosts")


@pytest.fixture(scope="module")
def L():
    return hatq.load(build_if_missing=True)


def declared_symbols():
    txt = open(os.path.join(ROOT, "include", "hatq.h")).read()
    return sorted(set(re.findall(r"^\S.*?\b(hatq_\w+)\s*\(", txt, re.M)))


def test_exports_every_declared_symbol(L):
    syms = declared_symbols()
    assert len(syms) >= 9
    for s in syms:
        assert hasattr(L, s), s
    assert set(syms) == set(hatq.EXPORTS)


def test_status_strings(L):
    for s in range(5):
        assert hatq.status_string(s)
    assert hatq.status_string(99) == "unknown status"


@pytest.mark.parametrize("args,exp", [
    ((192, 192, 5, 2, 2, 64), (128, 128)),
    ((128, 128, 1, 1, 0, 128), (64, 64)),
    ((3, 192, 5, 2, 2, 64), (128, 128)),
])
def test_out_hw(L, args, exp):
    assert hatq.hatq_conv_out_hw(hatq.desc(*args), 256 if args[3] == 2 else 64,
                                 256 if args[3] == 2 else 64) == exp


def test_out_hw_transposed(orc):
    d = hatq.desc(192, 192, 5, 2, 2, 64, transposed=True, out_pad=1)
    assert hatq.hatq_conv_out_hw(d, 64, 96) == (orc.out_size(64, 5, 2, 2, True, 1),
                                                orc.out_size(96, 5, 2, 2, True, 1)) == (128, 192)


def test_weights_bytes(L):
    assert hatq.hatq_weights_bytes(hatq.desc(192, 192, 5, 2, 2, 64), "DH") >= 192 * 4800 + 2 * 192 * 4
    assert hatq.hatq_weights_bytes(hatq.desc(3, 192, 5, 2, 2, 64), "WH") >= 192 * 128
    assert hatq.hatq_weights_bytes(hatq.desc(192, 192, 5, 2, 2, 48), "DH") == 0    # not a power of two
    assert hatq.hatq_weights_bytes(hatq.desc(192, 192, 5, 2, 2, 256), "DH") == 0   # above 128
    assert hatq.hatq_weights_bytes(hatq.desc(192, 192, 5, 2, 2, 64), 7) == 0


def test_prepare_rejects_before_launch(L):
    out = hatq.Weights()
    d = hatq.desc(192, 192, 5, 2, 2, 64)
    f = L.hatq_prepare_weights
    assert f(ctypes.byref(d), 0, None, None, FAKE, 1 << 30, ctypes.byref(out), None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(d), 0, FAKE, None, FAKE, 16, ctypes.byref(out), None) == hatq.HATQ_EWORKSPACE
    d2 = hatq.desc(96, 192, 5, 2, 2, 64)       # DH needs cin % hblock == 0
    assert f(ctypes.byref(d2), 0, FAKE, None, FAKE, 1 << 30, ctypes.byref(out), None) == hatq.HATQ_EUNSUPPORTED
    d3 = hatq.desc(192, 96, 5, 2, 2, 64)       # WH needs cout % hblock == 0
    assert f(ctypes.byref(d3), 1, FAKE, None, FAKE, 1 << 30, ctypes.byref(out), None) == hatq.HATQ_EUNSUPPORTED
    assert f(ctypes.byref(d), 0, FAKE, None, ctypes.c_void_p(0x10010), 1 << 30, ctypes.byref(out),
             None) == hatq.HATQ_EINVAL    # dst not 256-aligned


def test_fwht_quant_c64_rejects_before_launch(L):
    f = L.hatq_fwht_quant_act_c64
    assert f(None, 1, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 96, 32, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED   # c % 64
    assert f(FAKE, 1, 4, 4, 128, 128, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED  # block 128
    assert f(FAKE, 1, 4, 4, 192, 192, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED  # Kronecker
    assert f(FAKE, 1, 4, 4, 64, 64, None, ctypes.c_void_p(FAKE.value + 4), FAKE, FAKE, 256,
             None) == hatq.HATQ_EINVAL                                                            # xq not 16-aligned
    assert f(FAKE, 2, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 0, None) == hatq.HATQ_EWORKSPACE


def test_fwht_quant_rejects_before_launch(L):
    f = L.hatq_fwht_quant_act
    assert f(None, 1, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 48, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 96, 64, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED
    assert f(FAKE, 2, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 0, None) == hatq.HATQ_EWORKSPACE
    assert f(FAKE, 2, 4, 4, 64, 64, None, FAKE, FAKE, None, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.c_void_p(0x10004), 1, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 0, 4, 4, 64, 64, None, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL


def _fake_weights(cin=192, cout=192, k=5, s=2, p=2, hb=64, form=0, transposed=0, out_pad=0):
    d = hatq.desc(cin, cout, k, s, p, hb, transposed, out_pad)
    cin_p = -(-cin // hb) * hb if form == 0 else cin
    cout_p = -(-cout // hb) * hb if form == 1 else cout
    kt = k * k * cin_p
    ks = -(-kt // 64) * 64
    rowrun = not transposed and cin_p <= 4 and k * cin_p <= 16 and k <= 8 and s <= 2
    ps = -(-16 * k // 64) * 64 if rowrun else ks
    return hatq.Weights(d, form, cin_p, cout_p, kt, ks, 0x10000, 0x20000, 0x30000, 0x40000, ps)


def test_pack_rejects_before_launch(L):
    f = L.hatq_pack_weights
    assert f(None, None) == hatq.HATQ_EINVAL
    W = _fake_weights(cin=3, form=1)
    W.pack_stride = W.k_stride + 64                    # inconsistent view
    assert f(ctypes.byref(W), None) == hatq.HATQ_EINVAL
    W = _fake_weights()
    W.wpack = None
    assert f(ctypes.byref(W), None) == hatq.HATQ_EINVAL


def test_conv_rejects_before_launch(L):
    f = L.hatq_conv_int8

    def c(W, n, h, w, mode, y, nh, na, out_scale=None, flags=0):
        return f(W, FAKE, FAKE, n, h, w, mode, out_scale, y, nh, na, flags, None)
    W = _fake_weights()
    assert c(None, 1, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), 1, 8, 8, 5, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), 1, 8, 8, 0, FAKE, 64, FAKE) == hatq.HATQ_EINVAL          # I32 + absmax
    assert c(ctypes.byref(W), 1, 8, 8, 1, FAKE, 0, None, flags=8) == hatq.HATQ_EINVAL  # unknown flag
    # chunk-major codes: outputs only in code modes; input only for the 5x5 stride-2 window kernel
    assert c(ctypes.byref(W), 1, 8, 8, 1, FAKE, 0, None, flags=hatq.HATQ_YQ_C64) == hatq.HATQ_EINVAL
    W3 = _fake_weights(k=3, p=1)
    assert c(ctypes.byref(W3), 1, 8, 8, 1, FAKE, 0, None, flags=hatq.HATQ_XQ_C64) == hatq.HATQ_EUNSUPPORTED
    Wt = _fake_weights(transposed=1, out_pad=1)
    assert c(ctypes.byref(Wt), 1, 8, 8, 1, FAKE, 0, None, flags=hatq.HATQ_XQ_C64) == hatq.HATQ_EUNSUPPORTED
    W128 = _fake_weights(cout=128)
    assert c(ctypes.byref(W128), 1, 8, 8, 1, FAKE, 0, None, flags=hatq.HATQ_XQ_C64) == hatq.HATQ_EUNSUPPORTED
    # an order-320 transform in the epilogue runs on the general kernel's
    # 320-column tile: not with chunk-major codes, not for 3 input channels
    Wwh = _fake_weights(cout=320, hb=320, form=1)
    assert c(ctypes.byref(Wwh), 1, 8, 8, 1, FAKE, 0, None, flags=hatq.HATQ_XQ_C64) == hatq.HATQ_EUNSUPPORTED
    Wdh = _fake_weights(cout=320)
    assert c(ctypes.byref(Wdh), 1, 8, 8, 1, FAKE, 320, FAKE, flags=hatq.HATQ_XQ_C64) == hatq.HATQ_EUNSUPPORTED
    assert c(ctypes.byref(Wdh), 1, 8, 8, 1, FAKE, 192, FAKE) == hatq.HATQ_EUNSUPPORTED   # 192 does not tile 320
    Wrgb = _fake_weights(cin=3, cout=320, hb=320, form=1)
    assert c(ctypes.byref(Wrgb), 1, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    Wrgb64 = _fake_weights(cin=3, cout=320, hb=64, form=1)
    assert c(ctypes.byref(Wrgb64), 1, 8, 8, 1, FAKE, 320, FAKE) == hatq.HATQ_EUNSUPPORTED
    assert c(ctypes.byref(W), 1, 8, 8, 1, FAKE, 0, None, out_scale=FAKE) == hatq.HATQ_EINVAL   # scale outside I8
    bad = _fake_weights()
    bad.k_total += 1                                   # inconsistent view
    assert c(ctypes.byref(bad), 1, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EINVAL
    W32 = _fake_weights(cin=32, hb=32)                 # cin_pad 32: neither small nor a multiple of 64
    assert c(ctypes.byref(W32), 1, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    Wt3 = _fake_weights(transposed=1, s=3, out_pad=1)  # transposed needs stride 2
    assert c(ctypes.byref(Wt3), 1, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    assert c(ctypes.byref(W), 1, 8, 8, 1, FAKE, 128, FAKE) == hatq.HATQ_EUNSUPPORTED
    W0 = _fake_weights(p=0)                            # 5x5, no padding: a 2x2 input gives no output
    assert c(ctypes.byref(W0), 1, 2, 2, 1, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), 0, 8, 8, 1, FAKE, 0, None) == hatq.HATQ_EINVAL


def test_conv_absmax_only_needs_next_absmax(L):
    f = L.hatq_conv_int8
    W = _fake_weights()
    # y = NULL is only the absmax-only F32 call
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, 1, None, None, 0, None, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, 0, None, None, 0, None, 0, None) == hatq.HATQ_EINVAL


def test_conv_i8_mode_needs_static_scale(L):
    """HATQ_OUT_I8 through hatq_conv_int8: the codes need out_scale (a static
    per-sample scale) and an output; a next_absmax is not taken in this mode;
    the next operand's block follows the requantizing entry point's rules."""
    f = L.hatq_conv_int8
    W = _fake_weights()
    I8 = hatq.HATQ_OUT_I8
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, None, FAKE, 64, None, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, FAKE, None, 64, None, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, FAKE, FAKE, 64, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, FAKE, FAKE, 3, None, 0, None) == hatq.HATQ_EINVAL
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, FAKE, FAKE, 128, None, 0, None) == hatq.HATQ_EUNSUPPORTED
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, ctypes.c_void_p(FAKE.value + 2), FAKE, 64, None, 0,
             None) == hatq.HATQ_EINVAL                                                   # misaligned scale
    assert f(ctypes.byref(W), FAKE, FAKE, 1, 8, 8, I8, FAKE, FAKE, 64, None, 8, None) == hatq.HATQ_EINVAL


def test_requant_rejects_before_launch(L):
    f = L.hatq_conv_int8_requant
    W = _fake_weights()

    def r(W, n, nh, na, sc, yq, flags=0):
        return f(W, FAKE, FAKE, n, 8, 8, nh, na, sc, yq, flags, None)
    assert r(None, 1, 64, FAKE, FAKE, FAKE) == hatq.HATQ_EINVAL
    assert r(ctypes.byref(W), 1, 64, FAKE, None, FAKE) == hatq.HATQ_EINVAL   # no scale
    assert r(ctypes.byref(W), 1, 64, FAKE, FAKE, None) == hatq.HATQ_EINVAL   # no output
    assert r(ctypes.byref(W), 0, 64, FAKE, FAKE, FAKE) == hatq.HATQ_EINVAL
    assert r(ctypes.byref(W), 1, 3, FAKE, FAKE, FAKE) == hatq.HATQ_EINVAL    # block 3
    assert r(ctypes.byref(W), 1, 128, FAKE, FAKE, FAKE) == hatq.HATQ_EUNSUPPORTED
    assert r(ctypes.byref(W), 1, 64, ctypes.c_void_p(FAKE.value + 2), FAKE, FAKE) == hatq.HATQ_EINVAL  # misaligned
    assert r(ctypes.byref(W), 1, 64, FAKE, FAKE, FAKE, flags=8) == hatq.HATQ_EINVAL                   # unknown flag
    W96 = _fake_weights(cout=96, hb=32)
    assert r(ctypes.byref(W96), 1, 32, FAKE, FAKE, FAKE, flags=hatq.HATQ_YQ_C64) == hatq.HATQ_EUNSUPPORTED  # cout % 64
    assert r(ctypes.byref(W), 1, 64, FAKE, FAKE, ctypes.c_void_p(FAKE.value + 4),
             flags=hatq.HATQ_YQ_C64) == hatq.HATQ_EINVAL                                            # yq not 16-aligned


def test_int_transition_rejects_before_launch(L):
    W = _fake_weights()
    assert L.hatq_int_table_len(ctypes.byref(W)) == 2 * W.cout_pad + 1
    assert L.hatq_int_table_len(None) == 0
    p = L.hatq_int_transition_params
    assert p(None, 0.1, 0.1, 64, FAKE, None) == hatq.HATQ_EINVAL
    assert p(ctypes.byref(W), 0.0, 0.1, 64, FAKE, None) == hatq.HATQ_EINVAL           # s_x not positive
    assert p(ctypes.byref(W), 0.1, float("inf"), 64, FAKE, None) == hatq.HATQ_EINVAL  # s_y not finite
    assert p(ctypes.byref(W), 0.1, float("nan"), 64, FAKE, None) == hatq.HATQ_EINVAL
    assert p(ctypes.byref(W), 0.1, 0.1, 3, FAKE, None) == hatq.HATQ_EINVAL            # block 3
    assert p(ctypes.byref(W), 0.1, 0.1, 128, FAKE, None) == hatq.HATQ_EINVAL          # above 64
    assert p(ctypes.byref(W), 0.1, 0.1, 64, None, None) == hatq.HATQ_EINVAL           # no table
    assert p(ctypes.byref(W), 0.1, 0.1, 64, ctypes.c_void_p(FAKE.value + 4), None) \
        == hatq.HATQ_EINVAL                                                             # misaligned
    c = L.hatq_conv_int8_int_transition
    assert c(None, FAKE, 1, 8, 8, 64, FAKE, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), FAKE, 0, 8, 8, 64, FAKE, FAKE, 0, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 64, None, FAKE, 0, None) == hatq.HATQ_EINVAL      # no table
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 64, FAKE, None, 0, None) == hatq.HATQ_EINVAL      # no output
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 3, FAKE, FAKE, 0, None) == hatq.HATQ_EINVAL       # block 3
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 128, FAKE, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    # the Sylvester order 128 stays out of the integer epilogue, on either side
    Wwh = _fake_weights(cin=128, cout=128, hb=128, form=1)
    assert p(ctypes.byref(Wwh), 0.1, 0.1, 64, FAKE, None) == hatq.HATQ_EUNSUPPORTED
    assert c(ctypes.byref(Wwh), FAKE, 1, 8, 8, 64, FAKE, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    Wdh = _fake_weights(cin=64, cout=128)
    assert c(ctypes.byref(Wdh), FAKE, 1, 8, 8, 128, FAKE, FAKE, 0, None) == hatq.HATQ_EUNSUPPORTED
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 64, ctypes.c_void_p(FAKE.value + 4), FAKE, 0, None) \
        == hatq.HATQ_EINVAL                                                                   # misaligned table
    assert c(ctypes.byref(W), FAKE, 1, 8, 8, 64, FAKE, FAKE, 8, None) == hatq.HATQ_EINVAL      # unknown flag
    W3 = _fake_weights(k=3, p=1)
    assert c(ctypes.byref(W3), FAKE, 1, 8, 8, 64, FAKE, FAKE, hatq.HATQ_XQ_C64, None) == hatq.HATQ_EUNSUPPORTED


def test_noalloc_rejects_before_launch(L):
    f = L.hatq_fwht_quant_act_noalloc
    assert f(None, 1, 4, 4, 64, 64, FAKE, FAKE, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 64, None, FAKE, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 0, 4, 4, 64, 64, FAKE, FAKE, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 48, FAKE, FAKE, None) == hatq.HATQ_EINVAL           # not a supported order
    assert f(FAKE, 1, 4, 4, 96, 64, FAKE, FAKE, None) == hatq.HATQ_EUNSUPPORTED     # c % b
    assert f(ctypes.c_void_p(FAKE.value + 4), 1, 4, 4, 64, 64, FAKE, FAKE, None) == hatq.HATQ_EINVAL
    n = hatq.HATQ_NOALLOC_MAX_SAMPLES
    assert f(FAKE, n + 1, 4, 4, 64, 64, FAKE, FAKE, None) == hatq.HATQ_EUNSUPPORTED  # past the scratch


def test_export_rejects_before_copy(L):
    f = L.hatq_export_weights
    assert f(None, None, None, None, None) == hatq.HATQ_EINVAL
    bad = _fake_weights()
    bad.k_stride += 64                                 # inconsistent view
    assert f(ctypes.byref(bad), None, None, None, None) == hatq.HATQ_EINVAL
    W = _fake_weights()
    assert f(ctypes.byref(W), None, None, None, None) == hatq.HATQ_OK   # nothing to copy


def test_range_expansion_rejects_before_launch(L):
    f = L.hatq_range_expansion
    assert f(None, 1, 4, 4, 64, 64, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 64, None, None, None, None) == hatq.HATQ_EINVAL                 # no amax
    assert f(FAKE, 0, 4, 4, 64, 64, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 65536, 4, 4, 64, 64, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 0, 64, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 48, FAKE, None, None, None) == hatq.HATQ_EINVAL                 # not a power of two
    assert f(FAKE, 1, 4, 4, 64, 256, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(ctypes.c_void_p(FAKE.value + 4), 1, 4, 4, 64, 64, FAKE, None, None, None) == hatq.HATQ_EINVAL
    assert f(FAKE, 1, 4, 4, 64, 64, FAKE, ctypes.c_void_p(FAKE.value + 2), None, None) == hatq.HATQ_EINVAL


def test_select_form_matches_oracle(L, orc):
    out = ctypes.c_int32(-1)
    for k, m, tau in [(800, 1000, 0.8), (801, 1000, 0.8), (0, 1, 0.8), (1, 1, 0.8), (4, 5, 0.8), (5, 6, 0.8),
                      (3, 10, 0.3), (4, 10, 0.3), (7, 7, 1.0), (0, 3, -0.5), (2, 3, 2.0 / 3.0)]:
        assert L.hatq_select_form(k, m, tau, ctypes.byref(out)) == hatq.HATQ_OK
        assert ("WH" if out.value == hatq.HATQ_WH else "DH") == orc.select_form(k, m, tau), (k, m, tau)
    for k, m, tau in [(1, 0, 0.8), (-1, 4, 0.8), (5, 4, 0.8), (1, 2, float("nan")), (1, 2, float("inf"))]:
        assert L.hatq_select_form(k, m, tau, ctypes.byref(out)) == hatq.HATQ_EINVAL
    assert L.hatq_select_form(1, 2, 0.8, None) == hatq.HATQ_EINVAL


def test_affine_rejects_before_launch(L):
    q = L.hatq_fwht_quant_act_affine
    assert L.hatq_fwht_quant_affine_ws_bytes(4) >= 32 and L.hatq_fwht_quant_affine_ws_bytes(0) == 0
    assert q(None, 1, 4, 4, 64, 64, FAKE, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert q(FAKE, 1, 4, 4, 64, 64, FAKE, FAKE, None, FAKE, 256, None) == hatq.HATQ_EINVAL     # no zero points
    assert q(FAKE, 1, 4, 4, 64, 48, FAKE, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EINVAL
    assert q(FAKE, 4, 4, 4, 64, 64, FAKE, FAKE, FAKE, FAKE, 16, None) == hatq.HATQ_EWORKSPACE
    assert q(FAKE, 1, 4, 4, 48, 32, FAKE, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED  # c % b
    assert q(FAKE, 1, 3, 3, 3, 1, FAKE, FAKE, FAKE, FAKE, 256, None) == hatq.HATQ_EUNSUPPORTED    # h*w*c % 4
    W = _fake_weights()
    assert L.hatq_tapsum_len(ctypes.byref(W)) == (W.d.k * W.d.k + 1) * W.cout_pad
    assert L.hatq_tapsum_len(None) == 0
    assert L.hatq_weight_tapsums(ctypes.byref(W), None, None) == hatq.HATQ_EINVAL
    assert L.hatq_weight_tapsums(ctypes.byref(W), ctypes.c_void_p(FAKE.value + 4), None) == hatq.HATQ_EINVAL
    c = L.hatq_conv_int8_affine
    assert c(None, FAKE, FAKE, FAKE, FAKE, 1, 8, 8, 1, FAKE, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), FAKE, FAKE, None, FAKE, 1, 8, 8, 1, FAKE, None) == hatq.HATQ_EINVAL   # no zero points
    assert c(ctypes.byref(W), FAKE, FAKE, FAKE, None, 1, 8, 8, 1, FAKE, None) == hatq.HATQ_EINVAL   # no tap sums
    assert c(ctypes.byref(W), FAKE, FAKE, FAKE, FAKE, 1, 8, 8, hatq.HATQ_OUT_I8, FAKE, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), FAKE, FAKE, FAKE, FAKE, 0, 8, 8, 1, FAKE, None) == hatq.HATQ_EINVAL
    assert c(ctypes.byref(W), FAKE, FAKE, FAKE, ctypes.c_void_p(FAKE.value + 4), 1, 8, 8, 1, FAKE, None) \
        == hatq.HATQ_EINVAL


def test_layer_forward_form_flag_and_workspace(L):
    f = L.hatq_layer_forward
    W = _fake_weights()
    # the per-layer form flag must match the prepared weights
    assert f(ctypes.byref(W), 1, FAKE, 1, 16, 16, None, FAKE, None, 0, None, FAKE, 1 << 30,
             None) == hatq.HATQ_EINVAL
    need = L.hatq_layer_ws_bytes(ctypes.byref(W), 1, 16, 16)
    assert need >= 16 * 16 * 192
    assert f(ctypes.byref(W), 0, FAKE, 1, 16, 16, None, FAKE, None, 0, None, FAKE, need - 1,
             None) == hatq.HATQ_EWORKSPACE
    assert f(ctypes.byref(W), 0, FAKE, 1, 16, 16, None, FAKE, None, 0, None, None, need,
             None) == hatq.HATQ_EINVAL
