"""A workload's layer stack on the GPU (step a7: Table I transitions, Fig.
hadamard_framework): prepared weights, device buffers allocated once, and one
step = every layer's activation transform + quantization, INT8 convolution and
epilogue, in order.

Composition (identity nonlinearity between layers, fp32 between layers):
  * The first layer quantizes its input with the two-pass kernel pair (absmax,
    then codes).
  * A layer with a small input-channel count (the row-run path, whose fp32
    output is the largest tensor of the stack) hands its output to the next
    layer as INT8 codes through the requantizing epilogue: an absmax-only pass,
    then the codes (the dynamic per-sample scale needs the whole sample's
    maximum first).  By default both transforms of a WH -> DH transition run
    (the WH output restore, then the next layer's butterfly); ``paired=True``
    takes the next operand as z instead (B_next B_Cout = b I, HATQ_PAIRED).
  * Every other layer writes fp32 and the next layer's per-sample absmax in its
    epilogue, so the next layer's quantization reads its input once.

Code layout: with ``c64`` (the default) a layer's input codes are kept in the
chunk-major layout [n][cin/64][h][w][64] (HATQ_XQ_C64) wherever the layer's
convolution reads it (5x5 stride 2, cin a multiple of 64) and its producer
writes it (the requantizing epilogue, HATQ_YQ_C64, or
hatq_fwht_quant_act_c64): the same codes, placed so the convolution's input
window refills read whole 128-byte lines.  ``codes(i)`` returns them NHWC.

Every step of the path runs in the library's kernels; this module only
allocates and sequences the calls.
"""
from __future__ import annotations

from typing import Callable, List, Optional

import numpy as np
import torch

from . import hatq, workloads


class Stack:
    def __init__(self, wl: workloads.Workload, params, device="cuda:0", c64: bool = True):
        self.wl = wl
        self.dev = torch.device(device)
        self.shapes = wl.shapes()
        self.n = wl.input_shape[0]
        self.nL = len(wl.layers)
        self.layers: List[hatq.PreparedLayer] = []
        for L, (w, b) in zip(wl.layers, params):
            d = hatq.desc(L.cin, L.cout, L.k, L.stride, L.pad, L.hblock, L.transposed, L.out_pad)
            bt = None if b is None else torch.from_numpy(b).to(self.dev)
            self.layers.append(hatq.hatq_prepare_weights(d, L.form, torch.from_numpy(w).to(self.dev), bt))
        # activation transform block of each layer's input (WH: none)
        self.act_hb = [L.hblock if L.form == "DH" else 1 for L in wl.layers]
        # layer i writes layer i+1's codes (small-cin producer: the row-run path)
        self.requant = [i + 1 < self.nL and wl.layers[i].cin <= 4 for i in range(self.nL)]
        # chunk-major input codes: read by the 5x5 stride-2 window kernel, written
        # by the requantizing epilogue or the chunk-major quantizer
        def c64_ok(i):
            L = wl.layers[i]
            pl = self.layers[i]
            # (an epilogue with an order-320 transform runs on the general
            # kernel, which reads NHWC codes)
            nxt = wl.layers[i + 1] if i + 1 < self.nL else None
            o320 = (L.form == "WH" and L.hblock == 320) or (nxt is not None and self.act_hb[i + 1] == 320)
            reads = (not L.transposed and L.k == 5 and L.stride == 2 and pl.cin_pad % 64 == 0
                     and pl.cout_pad in (192, 320) and not o320)
            hb = self.act_hb[i]
            writes = hb <= 64 and (hb & (hb - 1)) == 0 if not (i > 0 and self.requant[i - 1]) else True
            return i > 0 and reads and writes
        self.c64 = [c64 and c64_ok(i) for i in range(self.nL)]
        n = self.n
        self.xq, self.sc, self.amax, self.ys = [], [], [], []
        for i, (ishape, oshape) in enumerate(self.shapes):
            if self.c64[i]:
                nn, h, w, c = ishape
                ishape = (nn, c // 64, h, w, 64)
            self.xq.append(torch.empty(ishape, dtype=torch.int8, device=self.dev))
            self.sc.append(torch.empty(n, dtype=torch.float32, device=self.dev))
            self.amax.append(torch.empty(n, dtype=torch.float32, device=self.dev))
            # a requantizing layer writes no fp32 output
            self.ys.append(None if self.requant[i] else torch.empty(oshape, dtype=torch.float32, device=self.dev))
        self.ws = torch.empty(int(hatq.load().hatq_fwht_quant_ws_bytes(n)), dtype=torch.int8, device=self.dev)

    def quant_passes(self, i: int) -> int:
        """Reads of layer i's fp32 input by its quantization (0: codes from the producer)."""
        if i == 0:
            return 2
        return 0 if self.requant[i - 1] else 1

    def step(self, x0: torch.Tensor, mark: Optional[Callable[[str], None]] = None,
             paired: bool = False) -> torch.Tensor:
        """One pass over the batch.  mark(label), if given, is called on the host
        before each launch group and at the end ("L<i>.quant", "L<i>.conv" or,
        for a requantizing layer, "L<i>.absmax" and "L<i>.requant", then
        "end"); the benchmark records a stream event there."""
        def m(label):
            if mark is not None:
                mark(label)
        x = x0
        for i in range(self.nL):
            m(f"L{i + 1}.quant")
            if self.quant_passes(i):
                quant = hatq.hatq_fwht_quant_act_c64 if self.c64[i] else hatq.hatq_fwht_quant_act
                quant(x, self.act_hb[i], absmax=None if i == 0 else self.amax[i - 1], xq=self.xq[i],
                      scale=self.sc[i], ws=self.ws)
            nxt = i + 1 < self.nL
            if self.requant[i]:
                m(f"L{i + 1}.absmax")
                hatq.hatq_conv_int8(self.layers[i], self.xq[i], self.sc[i], hatq.HATQ_OUT_F32,
                                    next_hblock=self.act_hb[i + 1], next_absmax=self.amax[i], absmax_only=True,
                                    paired=paired)
                m(f"L{i + 1}.requant")
                hatq.hatq_conv_int8_requant(self.layers[i], self.xq[i], self.sc[i], self.act_hb[i + 1],
                                            next_absmax=self.amax[i], next_scale=self.sc[i + 1],
                                            yq=self.xq[i + 1], paired=paired, yq_c64=self.c64[i + 1])
            else:
                m(f"L{i + 1}.conv")
                hatq.hatq_conv_int8(self.layers[i], self.xq[i], self.sc[i], hatq.HATQ_OUT_F32,
                                    next_hblock=self.act_hb[i + 1] if nxt else 0,
                                    next_absmax=self.amax[i] if nxt else None, y=self.ys[i])
            x = self.ys[i]
        m("end")
        return self.ys[-1]

    def output(self) -> torch.Tensor:
        return self.ys[-1]

    def nhwc_buf(self, i: int) -> torch.Tensor:
        """Layer i's code buffer viewed NHWC (the same memory, for calls that
        write and read it in that layout themselves)."""
        return self.xq[i].view(self.shapes[i][0])

    def codes(self, i: int) -> torch.Tensor:
        """Layer i's input codes, NHWC (a copy when they are kept chunk-major)."""
        return hatq.from_c64(self.xq[i]) if self.c64[i] else self.xq[i]


def conv_bytes(st: Stack, i: int) -> int:
    """Algorithmic bytes of layer i's convolution: int8 input once, int8 weights,
    output (fp32, or int8 codes for a requantizing layer)."""
    (ishape, oshape) = st.shapes[i]
    L = st.layers[i]
    out_pix = oshape[0] * oshape[1] * oshape[2]
    return int(np.prod(ishape)) + L.cout_pad * L.k_stride + out_pix * st.wl.layers[i].cout * (
        1 if st.requant[i] else 4)
