#!/usr/bin/env python3
"""Benchmark of the Hadamard-domain INT8 operator on one MI355X.

One step = one pass of the whole hot path over one batch of the workload
(default: the four-layer analysis stack, 5x5 stride-2 convolutions
3->192->192->192->320, per-layer forms WH, DH, DH, WH, Sylvester blocks of 64,
at batch 16 on 1024x1024 RGB inputs).  Per layer: activation transform +
per-sample absmax + INT8 quantization, INT8 implicit-GEMM convolution with
INT32 accumulation, fused dequant / bias / WH restore epilogue.  The layer-1 ->
layer-2 transition runs both Table I transforms explicitly (the WH output
restore, then the next layer's butterfly) inside the requantizing epilogue;
the cancellation shortcut (HATQ_PAIRED) is timed separately as
``paired_shortcut``.  Inputs and prepared weights are resident in HBM before
timing.  Data: synthetic, seeded (uniform RGB, Student-t weights).

Prints one JSON line.  ``value`` is the whole step's algorithmic INT8 conv
throughput (TOP/s, dense taps, 2 ops per MAC).  Every kernel of the step is
timed with stream events at its launch boundaries; per-layer figures are under
``layers``.  ``roofline`` is for the step's longest kernel, ``roofline_act_quant``
for the fused transform + quantization pass in the step (its layer-3 input,
read once); ``act_quant_l2_input`` times the same pass standalone on the
805 M-element layer-2-shaped tensor.  ``other_workloads`` carries the single
layers and the 512x768 stack, warm (back to back) and flushed (a 1 GiB write
between steps, which evicts the 256 MB MALL).  ``cpu_baseline`` times the CPU
oracle (rank 0, N = 1 only).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
PEAK_INT8_TOPS = 5000.0      # MI355X dense INT8 MFMA, TOP/s
# fp32 vector ALU, one lane-operation per lane per clock: 256 CUs x 4 SIMDs x
# 16 lanes x 2.4 GHz (the 157.3 TFLOP/s figure counts an FMA as two flops and
# packed dual-rate issue twice)
PEAK_ALU_TLOPS = 256 * 4 * 16 * 2.4e9 / 1e12
RIDGE = PEAK_INT8_TOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # ops per byte
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_analysis_stack_b16.json")
DEFAULT_WORKLOAD = "analysis_stack4_rgb_b16_1024x1024"
OTHER_WORKLOADS = ["linear1x1_dh_b128_64x64x128", "analysis_k5s2_192_256x256_dh", "analysis_k5s2_192_256x256_wh",
                   "synthesis_tconv_k5s2_192_64x96_dh", "analysis_stack4_rgb_512x768"]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("act_quant.hip", "conv_i8.hip", "hatq_device.h", "hatq_launch.h", "api.cpp"):
        h.update(open(os.path.join(ROOT, "paper_2608_01653_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(key: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    try:
        d = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != kernel_source_hash():
        return None
    return d.get("kernels", {}).get(key)


def traffic_bytes(key: str):
    t = measured_traffic(key)
    return None if t is None else int(t["bytes"])


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Marks:
    """Stream events recorded at the labelled launch boundaries of each step."""

    def __init__(self):
        import torch
        self.torch = torch
        self.steps = []

    def new_step(self):
        self.steps.append([])

    def mark(self, label):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        self.steps[-1].append((label, e))

    def durations_us(self):
        """Average time from each label to the next one, in microseconds."""
        acc = defaultdict(float)
        for st in self.steps:
            for (lab, e0), (_, e1) in zip(st, st[1:]):
                acc[lab] += e0.elapsed_time(e1) * 1e3
        return {k: v / len(self.steps) for k, v in acc.items()}

    def step_us(self):
        return sum(st[0][1].elapsed_time(st[-1][1]) for st in self.steps) / len(self.steps) * 1e3


def kernel_label(st, key):
    """The kernel behind a mark label of the step (for reports)."""
    li, part = key.split(".")
    i = int(li[1:]) - 1
    L = st.wl.layers[i]
    shape = f"layer {i + 1}, {L.form} {L.cin}->{L.cout} k{L.k}s{L.stride}"
    if part == "quant":
        b = st.act_hb[i]
        two = st.quant_passes(i) == 2
        return f"{'absmax_kernel<%d> + ' % b if two else ''}quant_kernel<{b}> ({shape})"
    if part in ("absmax", "requant"):
        nb = st.act_hb[i + 1]
        # the 32 x 32 MFMA variant: 3 -> 192 channels, 5x5 or 6x6, WH blocks of 64
        # into a next operand with blocks of 64, or the order 192 on both sides
        rr32 = (L.cin == 3 and L.cout == 192 and L.k in (5, 6) and L.form == "WH"
                and (L.hblock, nb) in ((64, 64), (192, 192)))
        name = "conv_rr32_kernel" if rr32 else "conv_rowrun_kernel"
        what = "next-operand absmax only" if part == "absmax" else "codes of the next operand"
        return f"{name} ({shape}; {what}, WH restore + B_{nb} explicit)"
    nxt = i + 1 < st.nL
    wb = L.hblock if L.form == "WH" else 0
    nb = st.act_hb[i + 1] if nxt else 0
    if L.cin <= 4:
        name = "conv_rowrun_kernel"
    elif L.k == 5 and L.stride == 2 and not L.transposed and 320 not in (wb, nb):
        name = "conv_halo5_kernel"
    else:
        name = "conv_pipe_kernel"    # (an order-320 epilogue: the 320-column tile)
    return f"{name}<Epi<{wb},{nb}>> ({shape})"


def _log2(b):
    return max(int(b).bit_length() - 1, 0)


def _stages(b):
    """Add/sub passes over each element of a transform of order b: log2(b) for
    a Sylvester block; for P_q+1 (x) H~_16 the four butterfly stages, then q
    sums per output of the Paley factor."""
    return 4 + int(b) // 16 - 1 if int(b) in (192, 320) else _log2(b)


# Algorithmic vector-ALU lane-operations of the method per element:
QUANT_OPS = 4          # scale, round, clamp, convert of one code
DEQUANT_OPS = 2        # int -> fp32 conversion and the fused scale-and-bias


def kernel_work(st, key):
    """Algorithmic work of the kernel(s) behind a mark label: INT8 MFMA ops,
    HBM bytes and vector-ALU lane-operations (a transform's add/sub passes per
    element, _stages, dequantization, quantization, maxima)."""
    import numpy as np
    from paper_2608_01653_amd import stack as stk, workloads
    li, part = key.split(".")
    i = int(li[1:]) - 1
    L = st.wl.layers[i]
    (ishape, oshape) = st.shapes[i]
    if part == "quant":
        e = int(np.prod(ishape))
        passes = st.quant_passes(i)
        ops = e * (_stages(st.act_hb[i]) + QUANT_OPS) + (e * (_stages(st.act_hb[i]) + 1) if passes == 2 else 0)
        return {"mfma_ops": 0, "hbm_bytes": e * 5, "alu_lane_ops": ops}
    outs = int(np.prod(oshape[:3])) * L.cout
    wb = L.hblock if L.form == "WH" else 1
    nxt = i + 1 < st.nL
    nb = st.act_hb[i + 1] if nxt else 1
    base = DEQUANT_OPS + _stages(wb)
    mf = workloads.conv_ops(st.wl, i)
    wbytes = st.layers[i].cout_pad * st.layers[i].k_stride
    xin = int(np.prod(ishape))
    if part == "absmax":
        return {"mfma_ops": mf, "hbm_bytes": xin + wbytes, "alu_lane_ops": outs * (base + _stages(nb) + 1)}
    if part == "requant":
        return {"mfma_ops": mf, "hbm_bytes": xin + wbytes + outs,
                "alu_lane_ops": outs * (base + _stages(nb) + QUANT_OPS)}
    alu = outs * (base + ((_stages(nb) + 1) if nxt else 0))
    return {"mfma_ops": mf, "hbm_bytes": stk.conv_bytes(st, i), "alu_lane_ops": alu}


def roofline_of(work, us):
    """The bound with the longest ideal time, and the achieved fraction of it."""
    t = us * 1e-6
    cands = [("mfma", work["mfma_ops"] / (PEAK_INT8_TOPS * 1e12), work["mfma_ops"] / t / 1e12, PEAK_INT8_TOPS,
              "TOP/s"),
             ("hbm", work["hbm_bytes"] / (PEAK_HBM_GBS * 1e9), work["hbm_bytes"] / t / 1e9, PEAK_HBM_GBS, "GB/s"),
             ("alu", work["alu_lane_ops"] / (PEAK_ALU_TLOPS * 1e12), work["alu_lane_ops"] / t / 1e12, PEAK_ALU_TLOPS,
              "T lane-op/s")]
    bound, ideal, ach, peak, unit = max(cands, key=lambda c: c[1])
    return {"bound": bound, "achieved": round(ach, 1), "peak": round(peak, 1), "unit": unit,
            "frac": round(ach / peak, 4), "ideal_us": round(ideal * 1e6, 2)}


def layer_report(st, dur, img_pix):
    """Per-layer figures from the per-kernel durations (us)."""
    import numpy as np
    from paper_2608_01653_amd import stack as stk, workloads
    out = []
    for i, L in enumerate(st.wl.layers):
        (ishape, oshape) = st.shapes[i]
        elems = int(np.prod(ishape))
        passes = st.quant_passes(i)
        tq = dur.get(f"L{i + 1}.quant", 0.0)
        if st.requant[i]:
            parts = {f"{p}_pass": dict(us=round(dur[f"L{i + 1}.{p}"], 2),
                                       **roofline_of(kernel_work(st, f"L{i + 1}.{p}"), dur[f"L{i + 1}.{p}"]))
                     for p in ("absmax", "requant")}
            tc = dur[f"L{i + 1}.absmax"] + dur[f"L{i + 1}.requant"]
        else:
            parts = {"conv_roofline": roofline_of(kernel_work(st, f"L{i + 1}.conv"), dur[f"L{i + 1}.conv"])}
            tc = dur[f"L{i + 1}.conv"]
        ops = workloads.conv_ops(st.wl, i)
        cb = stk.conv_bytes(st, i)
        tops = ops / (tc * 1e-6) / 1e12
        gbs = cb / (tc * 1e-6) / 1e9
        out_pix = oshape[0] * oshape[1] * oshape[2]
        rec = {
            "layer": f"L{i + 1} {L.form} {L.cin}->{L.cout} k{L.k}s{L.stride}"
                     + (" transposed" if L.transposed else ""),
            "act_quant_us": round(tq, 2) if passes else None,
            "act_quant_passes": passes,
            "act_quant_gbs_alg": round(elems * 5 / (tq * 1e-6) / 1e9, 1) if passes else None,
            "act_quant_hbm_frac": round(elems * 5 / (tq * 1e-6) / 1e9 / PEAK_HBM_GBS, 4) if passes else None,
            "conv_us": round(tc, 2),
            "conv_output": "int8 codes of the next operand" if st.requant[i] else "fp32",
            "conv_tops": round(tops, 1),
            "conv_mfma_frac": round(tops / PEAK_INT8_TOPS, 4),
            "conv_gbs_alg": round(gbs, 1),
            "conv_ops_per_byte": round(ops / cb, 1),
            "mpix_per_s_image": round(img_pix / ((tq + tc) * 1e-6) / 1e6, 1),
            "mpix_per_s_output": round(out_pix / ((tq + tc) * 1e-6) / 1e6, 1),
        }
        if passes == 0:
            rec["act_quant_note"] = "codes written by the previous layer's epilogue"
        rec.update(parts)
        out.append(rec)
    return out


_SLEEP_CYCLES_PER_US = None


def gpu_hold(us):
    """Keep the GPU busy for about `us` microseconds with a spin kernel that
    touches no memory, so the launches the host enqueues meanwhile run back to
    back (host launch overhead then adds no idle time between them)."""
    import torch
    global _SLEEP_CYCLES_PER_US
    if _SLEEP_CYCLES_PER_US is None:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        a.record()
        torch.cuda._sleep(1 << 20)
        b.record()
        torch.cuda.synchronize()
        _SLEEP_CYCLES_PER_US = (1 << 20) / max(a.elapsed_time(b) * 1e3, 1.0)
    torch.cuda._sleep(int(us * _SLEEP_CYCLES_PER_US))


def run_steps(st, x0, steps, warmup, paired=False, flush=None):
    """Time `steps` steps.  Warm: back to back, the whole run between two events
    (and each kernel by the marks).  Flushed: a 1 GiB write before every step;
    the step is timed from its first mark to its last.  Either way the GPU is
    held busy while the host enqueues, so host overhead does not show."""
    import torch
    for _ in range(warmup):
        st.step(x0, paired=paired)
    torch.cuda.synchronize()
    mk = Marks()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    gpu_hold(3000 + 600 * steps * st.nL)
    if flush is None:
        t0.record()
    for _ in range(steps):
        if flush is not None:
            flush.fill_(1)
        mk.new_step()
        st.step(x0, mark=mk.mark, paired=paired)
    if flush is None:
        t1.record()
    torch.cuda.synchronize()
    total_us = t0.elapsed_time(t1) * 1e3 / steps if flush is None else mk.step_us()
    return mk, total_us


def workload_figures(st, x0, steps, warmup, flush_buf):
    """Warm and flushed per-layer figures of one workload."""
    from paper_2608_01653_amd import workloads
    n, H, W = st.wl.input_shape[:3]
    img_pix = n * H * W
    ops = sum(workloads.conv_ops(st.wl, i) for i in range(st.nL))
    res = {"workload": st.wl.name, "input": list(st.wl.input_shape),
           "layers_desc": [f"{L.form} {L.cin}->{L.cout} k{L.k}s{L.stride} b{L.hblock}"
                           + (" transposed" if L.transposed else "") for L in st.wl.layers]}
    for label, fl in (("warm", None), ("flushed", flush_buf)):
        mk, us = run_steps(st, x0, steps, warmup, flush=fl)
        dur = mk.durations_us()
        res[label] = {"us_per_step": round(us, 2), "tops": round(ops / (us * 1e-6) / 1e12, 2),
                      "mpix_per_s": round(img_pix / (us * 1e-6) / 1e6, 1),
                      "layers": layer_report(st, dur, img_pix)}
    res["note"] = ("warm: steps back to back (inputs and weights may sit in the 256 MB MALL / L2); flushed: a "
                   "1 GiB device write before every step, timed from the step's first kernel to its last")
    return res


def cpu_baseline(x_np, params, wl):
    """The oracle, as it stands, on sample 0 of the batch (all host threads),
    stage by stage, and on the 512x768 stack with one thread."""
    import numpy as np
    import oracle
    from paper_2608_01653_amd import workloads

    oracle.lib()

    def run(wl_, x, prm, tag):
        stages = {"transform_quant_s": 0.0, "conv_s": 0.0, "epilogue_s": 0.0}
        ops = 0
        frac = x.shape[0] / wl_.input_shape[0]
        for i, L in enumerate(wl_.layers):
            w, b = prm[i]
            pw = oracle.prepare_weights(w, b, cin=L.cin, cout=L.cout, k=L.k, stride=L.stride, pad=L.pad,
                                        form=L.form, hblock=L.hblock, transposed=L.transposed,
                                        out_pad=L.out_pad)           # offline, not timed (as on the GPU)
            t0 = time.perf_counter()
            _, xq, sx = oracle.activation_operand(x, L.form, L.hblock)
            t1 = time.perf_counter()
            acc = oracle.conv_int8(xq, pw.wq, stride=L.stride, pad=L.pad, transposed=L.transposed,
                                   out_pad=L.out_pad)
            t2 = time.perf_counter()
            x = oracle.epilogue(acc, sx, pw)
            t3 = time.perf_counter()
            stages["transform_quant_s"] += t1 - t0
            stages["conv_s"] += t2 - t1
            stages["epilogue_s"] += t3 - t2
            ops += int(workloads.conv_ops(wl_, i) * frac)
            log(f"cpu baseline ({tag}): layer {i + 1} done ({sum(stages.values()):.1f} s so far)")
        return ops, {k: round(v, 3) for k, v in stages.items()}

    cores = oracle.set_threads(0)
    ops, stages = run(wl, x_np[:1], params, f"{cores} threads")
    secs = sum(stages.values())
    out = {"value": ops / secs / 1e12, "unit": "TOP/s", "cores": cores, "kind": "oracle",
           "seconds": round(secs, 3), "stages": stages,
           "sample": f"sample 0 of the batch (1/{wl.input_shape[0]} of one step): the same layers on "
                     f"[1,{','.join(str(v) for v in wl.input_shape[1:])}]; weight preparation untimed, as on "
                     "the GPU"}
    kodak = workloads.STACK_KODAK
    if [(L.cin, L.cout, L.k, L.form) for L in kodak.layers] == [(L.cin, L.cout, L.k, L.form) for L in wl.layers]:
        xk, pk = kodak.generate()
        oracle.set_threads(1)
        try:
            ops1, st1 = run(kodak, xk, pk, "1 thread")
        finally:
            oracle.set_threads(cores)
        s1 = sum(st1.values())
        out["single_thread"] = {"value": ops1 / s1 / 1e12, "unit": "TOP/s", "cores": 1, "seconds": round(s1, 3),
                                "stages": st1, "sample": f"the same stack on one {kodak.input_shape} image "
                                                         f"({kodak.name}), one thread"}
    return out


def measure_integer_stack(st, x0, args, total_ops, img_pix):
    """The same stack with integer-only transitions between layers (static
    per-tensor scales, calibrated as the largest per-sample scale the dynamic
    step produced for each operand): one activation pass on the image, then each
    conv writes the next layer's INT8 codes through the fixed-point epilogue;
    the last layer writes fp32.  Both Table I transforms run in the integer
    epilogue; the HATQ_PAIRED variant (B_next B_Cout = b I, bit-identical codes)
    is timed beside it."""
    import torch
    from paper_2608_01653_amd import hatq
    n, nL, dev = st.n, st.nL, st.dev
    s_dyn = [float(st.sc[i].max()) for i in range(nL)]
    a0 = torch.full((n,), s_dyn[0] * 127.0, dtype=torch.float32, device=dev)
    s0 = torch.empty(n, dtype=torch.float32, device=dev)
    hatq.hatq_fwht_quant_act(x0, st.act_hb[0], absmax=a0, xq=st.xq[0], scale=s0, ws=st.ws)
    s_x = [float(s0[0])] + s_dyn[1:]
    tables, shifts = [], []
    for i in range(nL - 1):
        t, sh = hatq.hatq_int_transition_params(st.layers[i], s_x[i], s_x[i + 1], st.act_hb[i + 1], device=dev)
        tables.append(t)
        shifts.append(sh)
    s_last = torch.full((n,), s_x[-1], dtype=torch.float32, device=dev)
    y_last = st.ys[-1]

    def istep(mark=None, paired=False):
        m = mark or (lambda _l: None)
        m("quant_l1")
        hatq.hatq_fwht_quant_act(x0, st.act_hb[0], absmax=a0, xq=st.xq[0], scale=s0, ws=st.ws)
        for i in range(nL - 1):
            m(f"conv_l{i + 1}_int_transition")
            hatq.hatq_conv_int8_int_transition(st.layers[i], st.xq[i], st.act_hb[i + 1], tables[i],
                                               yq=st.xq[i + 1], paired=paired, yq_c64=st.c64[i + 1])
        m(f"conv_l{nL}_f32")
        hatq.hatq_conv_int8(st.layers[-1], st.xq[-1], s_last, hatq.HATQ_OUT_F32, y=y_last)
        m("end")

    res = {}
    for paired in (False, True):
        for _ in range(args.warmup):
            istep(paired=paired)
        torch.cuda.synchronize()
        mk = Marks()
        for _ in range(args.steps):
            mk.new_step()
            istep(mk.mark, paired)
        torch.cuda.synchronize()
        us = mk.step_us()
        res["paired" if paired else "explicit"] = {
            "ms_per_step": round(us / 1e3, 4), "tops": round(total_ops / (us * 1e-6) / 1e12, 2),
            "mpix_per_s": round(img_pix / (us * 1e-6) / 1e6, 1),
            "stages_us": {k: round(v, 2) for k, v in mk.durations_us().items()}}
    log(f"integer stack: {res['explicit']['ms_per_step']:.3f} ms/step explicit, "
        f"{res['paired']['ms_per_step']:.3f} paired")
    res.update({"static_scales": [float(f"{v:.6g}") for v in s_x], "shifts": shifts,
                "note": "integer-only transitions (fixed-point multiplier, integer bias, int64 Hadamard "
                        "transforms in the conv epilogue); static per-tensor scales; 'paired' folds the "
                        "layer-1 -> 2 transforms into B_next B_Cout = b I (exact in integers)"})
    return res


def layer1_f32_output(st):
    """Layer 1's fp32 output of the batch (the stack itself only forms its codes)
    and the next layer's fused absmax."""
    import torch
    from paper_2608_01653_amd import hatq
    y1 = torch.empty(st.shapes[0][1], dtype=torch.float32, device=st.dev)
    am = torch.empty(st.n, dtype=torch.float32, device=st.dev)
    hatq.hatq_conv_int8(st.layers[0], st.xq[0], st.sc[0], hatq.HATQ_OUT_F32, next_hblock=st.act_hb[1],
                        next_absmax=am, y=y1)
    return y1, am


def back_to_back(f, reps=20):
    import torch
    for _ in range(3):
        f()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        f()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps * 1e3   # us


def measure_act_quant_l2_input(st, y1, am):
    """The fused transform + quantization pass standalone on layer 2's input, the
    805 M-element fp32 tensor [16,512,512,192]: single read with the producer's
    absmax (5 B/element algorithmic), and the two-pass form (absmax kernel, then
    codes: 9 B/element moved, 5 algorithmic)."""
    from paper_2608_01653_amd import hatq
    hb = st.act_hb[1]
    e = y1.numel()
    q1 = st.nhwc_buf(1)
    t1 = back_to_back(lambda: hatq.hatq_fwht_quant_act(y1, hb, absmax=am, xq=q1, scale=st.sc[1], ws=st.ws))
    t2 = back_to_back(lambda: hatq.hatq_fwht_quant_act(y1, hb, xq=q1, scale=st.sc[1], ws=st.ws))
    alg = e * 5
    log(f"layer-2 input quantization: {t1:.1f} us single read, {t2:.1f} us two-pass")
    return {"tensor": list(y1.shape), "elements": e, "algorithmic_bytes": alg,
            "single_read": {"kernel": f"quant_kernel<{hb}>", "us": round(t1, 2),
                            "achieved": round(alg / (t1 * 1e-6) / 1e9, 1), "unit": "GB/s",
                            "frac": round(alg / (t1 * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)},
            "two_pass": {"kernels": f"absmax_kernel<{hb}> + quant_kernel<{hb}>", "us": round(t2, 2),
                         "achieved": round(alg / (t2 * 1e-6) / 1e9, 1), "unit": "GB/s",
                         "frac": round(alg / (t2 * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)},
            "note": "20 launches back to back on the resident tensor (layer 1's fp32 output, with the per-sample "
                    "absmax its epilogue produced)"}


def measure_form_selection(st, x0, y1, tau=0.8, reps=5):
    """The profiling pass of the form rule on this batch: per image, the
    range-expansion indicator of each layer's fp32 input with the layer's
    block, p_l over the batch and the form it selects; the pass over layer 2's
    input (the largest activation) is timed (one read, HBM bound)."""
    import torch
    from paper_2608_01653_amd import hatq
    n = st.n
    inputs = [x0, y1] + st.ys[1:st.nL - 1]
    p, sel = [], []
    amax = torch.empty(2 * n, dtype=torch.float32, device=st.dev)
    flags = torch.empty(n, dtype=torch.int32, device=st.dev)
    for L, xin in zip(st.wl.layers, inputs):
        count = torch.zeros(1, dtype=torch.int32, device=st.dev)
        hatq.hatq_range_expansion(xin, L.hblock, amax=amax, flags=flags, count=count)
        k = int(count.item())
        p.append(round(k / n, 4))
        sel.append(hatq.hatq_select_form(k, n, tau))
    us = back_to_back(lambda: hatq.hatq_range_expansion(y1, st.wl.layers[1].hblock, amax=amax, flags=flags),
                      reps)
    nbytes = y1.numel() * 4
    gbs = nbytes / (us * 1e-6) / 1e9
    log(f"form selection: p = {p}, selected {sel}; profiling pass {us:.1f} us")
    return {"tau": tau, "images": n, "p": p, "selected": sel, "configured": [L.form for L in st.wl.layers],
            "profile_pass": {"kernel": f"range_kernel<{st.wl.layers[1].hblock}> (layer 2 input)",
                             "us": round(us, 2), "bound": "hbm", "achieved": round(gbs, 1),
                             "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                             "work": f"{nbytes} bytes per call = {y1.numel()} fp32 elements read once"},
            "note": "random-init weights and synthetic inputs: the selection shows the mechanism, "
                    "not the paper's trained-model assignment"}


def measure_affine_layer(st, per_layer, li=2, reps=20):
    """Layer 3 with affine dynamic activations (the paper's PTQ setting): the
    min / max pass and the affine quantization of its fp32 input, then the
    convolution with the zero-point correction, F32 output."""
    import torch
    from paper_2608_01653_amd import hatq, workloads
    L = st.wl.layers[li]
    x = st.ys[li - 1]
    n = x.shape[0]
    scale = torch.empty(n, dtype=torch.float32, device=st.dev)
    zero = torch.empty(n, dtype=torch.int32, device=st.dev)
    ws = torch.empty(int(hatq.load().hatq_fwht_quant_affine_ws_bytes(n)), dtype=torch.int8, device=st.dev)
    tapsum = hatq.hatq_weight_tapsums(st.layers[li], device=st.dev)
    hb = st.act_hb[li]
    q = st.nhwc_buf(li)
    tq = back_to_back(lambda: hatq.hatq_fwht_quant_act_affine(x, hb, xq=q, scale=scale, zero=zero, ws=ws),
                      reps)
    tc = back_to_back(lambda: hatq.hatq_conv_int8_affine(st.layers[li], q, scale, zero, tapsum,
                                                         hatq.HATQ_OUT_F32, y=st.ys[li]), reps)
    ops = workloads.conv_ops(st.wl, li)
    z = zero.cpu().tolist()
    log(f"affine layer {li + 1}: quant {tq:.1f} us, conv {tc:.1f} us")
    return {"layer": per_layer[li]["layer"], "act_quant_affine_us": round(tq, 2),
            "act_quant_affine_gbs_alg": round(x.numel() * 5 / (tq * 1e-6) / 1e9, 1), "act_quant_affine_passes": 2,
            "conv_affine_us": round(tc, 2), "conv_affine_tops": round(ops / (tc * 1e-6) / 1e12, 1),
            "symmetric_act_quant_us": per_layer[li]["act_quant_us"], "symmetric_conv_us": per_layer[li]["conv_us"],
            "zero_points": [min(z), max(z)],
            "note": "dynamic per-sample affine activations (min/max pass + quantization), zero-point correction "
                    "in the conv epilogue; back to back on the resident layer input"}


def measure_order_layer(st, params, per_layer, li=2, reps=20):
    """Layer 3 (DH, 192 input channels) with the paper's transform order
    m(192) = 192 (one Kronecker block P_12 (x) H~_16 over all channels) in place
    of blocks of 64: the two-pass activation quantization of its fp32 input and
    the convolution."""
    import torch
    from paper_2608_01653_amd import hatq, workloads
    L = st.wl.layers[li]
    m = 192
    if L.form != "DH" or L.cin % m:
        return None
    w, b = params[li]
    layer = hatq.hatq_prepare_weights(hatq.desc(L.cin, L.cout, L.k, L.stride, L.pad, m, L.transposed, L.out_pad),
                                      "DH", torch.from_numpy(w).to(st.dev), torch.from_numpy(b).to(st.dev))
    x = st.ys[li - 1]
    q = st.nhwc_buf(li)
    tq = back_to_back(lambda: hatq.hatq_fwht_quant_act(x, m, xq=q, scale=st.sc[li], ws=st.ws), reps)
    tc = back_to_back(lambda: hatq.hatq_conv_int8(layer, q, st.sc[li], hatq.HATQ_OUT_F32, y=st.ys[li]),
                      reps)
    log(f"order-{m} layer {li + 1}: quant {tq:.1f} us, conv {tc:.1f} us")
    return {"layer": per_layer[li]["layer"], "order": m, "construction": "P_12 (x) H~_16 (Paley-I q = 11)",
            "act_quant_us": round(tq, 2), "act_quant_passes": 2,
            "act_quant_gbs_alg": round(x.numel() * 5 / (tq * 1e-6) / 1e9, 1),
            "conv_us": round(tc, 2),
            "conv_tops": round(workloads.conv_ops(st.wl, li) / (tc * 1e-6) / 1e12, 1),
            "block64_act_quant_us": per_layer[li]["act_quant_us"], "block64_conv_us": per_layer[li]["conv_us"],
            "note": "two-pass quantization, back to back on the resident layer input; algorithmic bytes 5 per "
                    "element (4 B fp32 read + 1 B int8 written)"}


def measure_paper_order_stack(wl, params, x0, steps, warmup, dev, block64_step_us):
    """The same four layers with one block of the paper's order m(C) per
    transformed axis (Eq. hadamard_order: 192, 192, 192, 320), the rest of the
    step unchanged (explicit transforms, dynamic per-sample scales)."""
    from paper_2608_01653_amd import hatq, stack, workloads
    owl = workloads.with_orders(wl, hatq.hatq_hadamard_order)
    ost = stack.Stack(owl, params, dev)
    mk, us = run_steps(ost, x0, steps, warmup)
    n, H, W = owl.input_shape[:3]
    img_pix = n * H * W
    ops = sum(workloads.conv_ops(owl, i) for i in range(ost.nL))
    res = {"workload": owl.name, "orders": [L.hblock for L in owl.layers],
           "layers_desc": [f"{L.form} {L.cin}->{L.cout} k{L.k}s{L.stride} b{L.hblock}" for L in owl.layers],
           "ms_per_step": round(us / 1e3, 4), "tops": round(ops / (us * 1e-6) / 1e12, 2),
           "mpix_per_s": round(img_pix / (us * 1e-6) / 1e6, 1),
           "block64_ms_per_step": round(block64_step_us / 1e3, 4),
           "layers": layer_report(ost, mk.durations_us(), img_pix),
           "note": "192 = P_12 (x) H~_16, 320 = P_20 (x) H~_16; layer 1's two passes on the row-run kernel "
                   "(the 32x32 variant takes blocks of 64), layer 4 on the general kernel's 320-column tile"}
    log(f"paper-order stack {res['orders']}: {us / 1e3:.3f} ms/step")
    del ost
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="only the step (no other legs or workloads)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device-to-device copy (scales the HBM byte counters)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("copied 1 GiB three times")
        return
    if args.gpus != 1:
        print("bench.py: this operator is measured on one GPU only; --gpus must be 1 "
              f"(got {args.gpus}). Batch sharding across GPUs needs no communication and is "
              "not run here.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_01653_amd import build, hatq, stack, workloads

    if build.stale() and not os.path.exists(build.LIB):
        build.build()
    hatq.load()
    wl = workloads.ALL[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    x_np, params = wl.generate()
    log(f"inputs generated: {wl.name} {wl.input_shape}")
    st = stack.Stack(wl, params, dev)
    x0 = torch.from_numpy(x_np).to(dev)
    n, H, W = wl.input_shape[:3]
    img_pix = n * H * W
    total_ops = sum(workloads.conv_ops(wl, i) for i in range(st.nL))

    mk, step_us = run_steps(st, x0, args.steps, args.warmup)
    log(f"timed {args.steps} steps: {step_us / 1e3:.3f} ms/step")
    dur = mk.durations_us()
    per_layer = layer_report(st, dur, img_pix)

    # the step's longest kernel, against its roofline (the bound with the
    # longest ideal time: INT8 MFMA ops, HBM bytes or vector-ALU lane-ops)
    key = max((k for k in dur if k != "end"), key=lambda k: dur[k])
    work = kernel_work(st, key)
    tkey = "conv_l2" if key == "L2.conv" else None
    roof = {"kernel": kernel_label(st, key), **roofline_of(work, dur[key]),
            "traffic": traffic_bytes(tkey) if tkey else None,
            "traffic_detail": measured_traffic(tkey) if tkey else None, "avg_us": round(dur[key], 2),
            "work": {**work, "per": "launch"}}
    kernels = [{"kernel": kernel_label(st, k), "us": round(v, 2), **roofline_of(kernel_work(st, k), v)}
               for k, v in dur.items() if k != "end" and v > 0 and not (k.endswith(".quant") and
                                                                         not st.quant_passes(int(k[1]) - 1))]
    out = {
        "metric": "Hadamard-INT8 conv TOPS + Mpixel/s per layer; % of INT8 MFMA / HBM peak",
        "value": round(total_ops / (step_us * 1e-6) / 1e12, 2),
        "unit": "TOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_us / 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded " + ("uniform RGB input" if wl.input_kind == "rgb" else
                                        "heavy-tailed Student-t activations") + ", Student-t weights)",
        "config": {"workload": wl.name, "input": list(wl.input_shape),
                   "layers": [f"{L.form} {L.cin}->{L.cout} k{L.k}s{L.stride} b{L.hblock}"
                              + (" transposed" if L.transposed else "") for L in wl.layers],
                   "form_mask": ",".join(L.form for L in wl.layers),
                   "transition": "Table I transforms explicit (WH restore, then the next butterfly)",
                   "parallelism": "none"},
        "mpix_per_s": round(img_pix / (step_us * 1e-6) / 1e6, 1),
        "layers": per_layer,
        "kernels": kernels,
        "roofline": roof,
    }
    # the fused transform + quantization pass in the step (first single-read layer)
    import numpy as np
    qi = next((i for i in range(1, st.nL) if st.quant_passes(i) == 1), 0)
    if st.quant_passes(qi):
        eq = int(np.prod(st.shapes[qi][0]))
        t_q = dur[f"L{qi + 1}.quant"] * 1e-6
        achq = eq * 5 / t_q / 1e9
        kq = (f"quant_kernel<{st.act_hb[qi]}> (layer {qi + 1}, single read, in the step)" if qi else
              f"absmax_kernel<{st.act_hb[0]}> + quant_kernel<{st.act_hb[0]}> (layer 1, two passes, in the step)")
        out["roofline_act_quant"] = {
            "kernel": kq, "bound": "hbm",
            "achieved": round(achq, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achq / PEAK_HBM_GBS, 4),
            "traffic": traffic_bytes(f"quant_l{qi + 1}"), "traffic_detail": measured_traffic(f"quant_l{qi + 1}"),
            "avg_us": round(t_q * 1e6, 2),
            "work": f"{eq * 5} bytes per launch = {eq} elements x (4 B fp32 in + 1 B int8 out)"}

    if not args.no_extras:
        if any(st.requant):
            mkp, us_p = run_steps(st, x0, args.steps, args.warmup, paired=True)
            dp = mkp.durations_us()
            i1 = st.requant.index(True)
            out["paired_shortcut"] = {
                "ms_per_step": round(us_p / 1e3, 4), "tops": round(total_ops / (us_p * 1e-6) / 1e12, 2),
                "mpix_per_s": round(img_pix / (us_p * 1e-6) / 1e6, 1),
                "absmax_pass_us": round(dp[f"L{i1 + 1}.absmax"], 2),
                "requant_pass_us": round(dp[f"L{i1 + 1}.requant"], 2),
                "note": "layer 1 -> 2 through the cancellation B_next B_Cout = b I (HATQ_PAIRED): the next "
                        "operand taken as z, neither transform run; valid only with identity between the layers"}
            log(f"paired shortcut: {us_p / 1e3:.3f} ms/step")
        if wl.name == DEFAULT_WORKLOAD:
            out["integer_stack"] = measure_integer_stack(st, x0, args, total_ops, img_pix)
            st.step(x0)                      # restore the dynamic step's buffers
            y1, am = layer1_f32_output(st)
            out["act_quant_l2_input"] = measure_act_quant_l2_input(st, y1, am)
            out["form_selection"] = measure_form_selection(st, x0, y1)
            del y1, am
            st.step(x0)
            out["affine_layer"] = measure_affine_layer(st, per_layer)
            out["paper_order_layer"] = measure_order_layer(st, params, per_layer)
            out["paper_order_stack"] = measure_paper_order_stack(wl, params, x0, args.steps, args.warmup, dev,
                                                                 step_us)
            flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
            others = []
            for name in OTHER_WORKLOADS:
                owl = workloads.ALL[name]
                oxn, opar = owl.generate()
                ost = stack.Stack(owl, opar, dev)
                others.append(workload_figures(ost, torch.from_numpy(oxn).to(dev), args.steps, args.warmup, flush))
                log(f"workload {name}: warm {others[-1]['warm']['us_per_step']:.1f} us, "
                    f"flushed {others[-1]['flushed']['us_per_step']:.1f} us")
                del ost
            out["other_workloads"] = others
            del flush
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(x_np, params, wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
