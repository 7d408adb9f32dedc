"""The synthetic learned-image-coding workloads: layer shapes, forms and input recipes.

Shapes only; no arithmetic of the method lives here.  Each workload is a list of
layers run in order; a layer's fp32 output is the next layer's input (identity
nonlinearity between layers).  ``form`` is the per-layer Hadamard form: "DH"
(double-Hadamard, Sec. IV-B) or "WH" (weight-only Hadamard, Sec. IV-B).  ``hblock``
is the block order of the block-diagonal transform (Sylvester blocks of 64 in the
specified workloads); it acts on C_in for DH and on C_out for WH.
``with_orders`` gives the same stack with one block of the paper's order m(C)
over each transformed axis (Eq. hadamard_order).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

import numpy as np

from . import synth


@dataclass(frozen=True)
class Layer:
    cin: int
    cout: int
    k: int
    stride: int
    pad: int
    form: str
    hblock: int
    transposed: bool = False
    out_pad: int = 0


@dataclass
class Workload:
    name: str
    input_shape: Tuple[int, int, int, int]   # NHWC
    input_kind: str                          # "heavy" | "rgb"
    layers: List[Layer]
    seed: int = 0
    note: str = ""

    def out_hw(self, i: int, h: int, w: int) -> Tuple[int, int]:
        L = self.layers[i]
        if L.transposed:
            return ((h - 1) * L.stride - 2 * L.pad + L.k + L.out_pad,
                    (w - 1) * L.stride - 2 * L.pad + L.k + L.out_pad)
        return ((h + 2 * L.pad - L.k) // L.stride + 1, (w + 2 * L.pad - L.k) // L.stride + 1)

    def shapes(self):
        """Per-layer (input NHWC, output NHWC)."""
        n, h, w, c = self.input_shape
        out = []
        for i, L in enumerate(self.layers):
            ho, wo = self.out_hw(i, h, w)
            out.append(((n, h, w, L.cin), (n, ho, wo, L.cout)))
            h, w = ho, wo
        return out

    def generate(self, with_bias: bool = True):
        """Input tensor then each layer's (weight, bias), all from one seeded rng."""
        rng = np.random.default_rng(self.seed)
        if self.input_kind == "rgb":
            x = synth.rgb_uniform(rng, self.input_shape)
        else:
            x = synth.heavy_tailed_activations(rng, self.input_shape)
        params = [synth.layer_params(rng, L.cin, L.cout, L.k, L.transposed, with_bias)
                  for L in self.layers]
        return x, params


def with_orders(wl: Workload, order) -> Workload:
    """The workload with each layer's block replaced by order(C), C the channel
    count of the transformed axis (C_in for DH, C_out for WH); ``order`` is the
    order rule m(C), passed in so this module stays free of the method."""
    layers = [replace(L, hblock=int(order(L.cin if L.form == "DH" else L.cout))) for L in wl.layers]
    return Workload(wl.name + "_paper_orders", wl.input_shape, wl.input_kind, layers, wl.seed,
                    "one block of order m(C) per transformed axis")


def conv_ops(wl: Workload, i: int) -> int:
    """Algorithmic MAC-pair count (2 ops per multiply-add) of layer i, dense taps."""
    (n, h, w, cin), (_, ho, wo, cout) = wl.shapes()[i]
    L = wl.layers[i]
    if L.transposed:
        return 2 * n * h * w * cin * cout * L.k * L.k
    return 2 * n * ho * wo * cout * L.k * L.k * cin


def _k5s2(cin, cout, form, hb=64):
    return Layer(cin, cout, 5, 2, 2, form, hb)


# Single 1x1 (linear) layer, double-Hadamard with one 128-point block.
LINEAR_1X1 = Workload("linear1x1_dh_b128_64x64x128", (1, 64, 64, 128), "heavy",
                [Layer(128, 128, 1, 1, 0, "DH", 128)])
# One analysis 5x5 stride-2 conv, 192->192, three 64-blocks; run in both forms.
ANALYSIS_K5S2_DH = Workload("analysis_k5s2_192_256x256_dh", (1, 256, 256, 192), "heavy",
                   [_k5s2(192, 192, "DH")])
ANALYSIS_K5S2_WH = Workload("analysis_k5s2_192_256x256_wh", (1, 256, 256, 192), "heavy",
                   [_k5s2(192, 192, "WH")])
# One synthesis 5x5 stride-2 transposed conv on a 1/16-resolution 1024x1536 latent.
SYNTHESIS_TCONV = Workload("synthesis_tconv_k5s2_192_64x96_dh", (1, 64, 96, 192), "heavy",
                [Layer(192, 192, 5, 2, 2, "DH", 64, transposed=True, out_pad=1)])
# Four-layer analysis stack, form mask WH, DH, DH, WH, on a Kodak-size RGB image.
_STACK = [_k5s2(3, 192, "WH"), _k5s2(192, 192, "DH"), _k5s2(192, 192, "DH"),
          _k5s2(192, 320, "WH")]
STACK_KODAK = Workload("analysis_stack4_rgb_512x768", (1, 512, 768, 3), "rgb", list(_STACK))
# The same stack at batch 16 on 1024x1024 RGB: the largest conv shapes.
STACK_B16 = Workload("analysis_stack4_rgb_b16_1024x1024", (16, 1024, 1024, 3), "rgb", list(_STACK))

ALL = {w.name: w for w in (LINEAR_1X1, ANALYSIS_K5S2_DH, ANALYSIS_K5S2_WH, SYNTHESIS_TCONV,
                             STACK_KODAK, STACK_B16)}
