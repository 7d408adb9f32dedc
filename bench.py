#!/usr/bin/env python3
"""Benchmark of the Hadamard-domain INT8 operator on one MI355X.

One step = one pass of the whole hot path over one batch: the four-layer
analysis stack (5x5 stride-2 convolutions 3->192->192->192->320, per-layer forms
WH, DH, DH, WH, Sylvester blocks of 64) at batch 16 on 1024x1024 RGB inputs.
Per layer: activation transform + per-sample absmax + INT8 quantization, INT8
implicit-GEMM convolution with INT32 accumulation, fused dequant/bias/WH-restore
epilogue; each convolution's epilogue also produces the next layer's per-sample
absmax, so layers 2-4 read their fp32 input once.  Inputs and prepared weights
are resident in HBM before timing.  Data: synthetic, seeded (uniform RGB,
Student-t weights).

Prints one JSON line.  ``value`` is the whole step's algorithmic INT8 conv
throughput (TOP/s, dense taps, 2 ops per MAC); per-layer time, TOP/s, GB/s and
Mpixel/s are under ``layers``.  ``roofline`` is for the dominant kernel (layer-2
convolution, INT8 MFMA bound); ``roofline_act_quant`` for layer 3's fused
transform+quantization pass (HBM bound; the first layer quantized from a stored
fp32 output, read once).  Both are timed inside the steps; their ``isolated``
entries time the same kernel on the same resident input launched back to back.  ``cpu_baseline`` times the CPU oracle
on one sample of the batch (rank 0, N = 1 only).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
PEAK_INT8_TOPS = 5000.0      # MI355X dense INT8 MFMA, TOP/s
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_analysis_stack_b16.json")


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
    """HBM bytes (read + written) per launch, or None."""
    t = measured_traffic(key)
    return None if t is None else int(t["bytes"])


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(wl, x_np, params):
    """The oracle, as it stands, on sample 0 of the batch (1/n of a step)."""
    import numpy as np
    import oracle
    from paper_2608_01653_amd import workloads

    oracle.lib()
    x = x_np[:1]
    ops = 0
    dt = 0.0
    for i, L in enumerate(wl.layers):
        w, b = params[i]
        pw = oracle.prepare_weights(w, b, cin=L.cin, cout=L.cout, k=L.k, stride=L.stride, pad=L.pad,
                                    form=L.form, hblock=L.hblock, transposed=L.transposed,
                                    out_pad=L.out_pad)           # offline, not timed (as on the GPU)
        t0 = time.perf_counter()
        r = oracle.layer_forward(x, pw)
        dt += time.perf_counter() - t0
        x = r.y
        ops += workloads.conv_ops(wl, i) // wl.input_shape[0]
        log(f"cpu baseline: layer {i + 1} done ({dt:.1f} s so far)")
    cores = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    return {"value": ops / dt / 1e12, "unit": "TOP/s", "cores": cores, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"sample 0 of the batch (1/{wl.input_shape[0]} of one step): the same four "
                      f"layers on [1,{wl.input_shape[1]},{wl.input_shape[2]},3]; weight "
                      "preparation untimed, as on the GPU"}


def measure_integer_stack(args, wl, layers, x0, xq, sc, ys, ws, act_hb, total_ops, img_pix):
    """The same stack with integer-only transitions between layers (static
    per-tensor scales, calibrated as the largest per-sample scale the dynamic
    step just produced for each operand): one activation pass on the image, then
    each conv writes the next layer's INT8 codes through the fixed-point
    epilogue; the last layer writes fp32.  Timed separately from the step."""
    import torch
    from paper_2608_01653_amd import hatq
    n = x0.shape[0]
    nL = len(layers)
    dev = x0.device
    s_dyn = [float(sc[i].max()) for i in range(nL)]
    # static input scale: every sample quantized with the batch's absmax
    a0 = torch.full((n,), s_dyn[0] * 127.0, dtype=torch.float32, device=dev)
    s0 = torch.empty(n, dtype=torch.float32, device=dev)
    hatq.hatq_fwht_quant_act(x0, act_hb[0], absmax=a0, xq=xq[0], scale=s0, ws=ws)
    s_x = [float(s0[0])] + s_dyn[1:]
    tables, shifts = [], []
    for i in range(nL - 1):
        t, sh = hatq.hatq_int_transition_params(layers[i], s_x[i], s_x[i + 1], act_hb[i + 1], device=dev)
        tables.append(t)
        shifts.append(sh)
    s_last = torch.full((n,), s_x[-1], dtype=torch.float32, device=dev)

    def istep(events=None):
        if events:
            events[0].record()
        hatq.hatq_fwht_quant_act(x0, act_hb[0], absmax=a0, xq=xq[0], scale=s0, ws=ws)
        for i in range(nL - 1):
            if events:
                events[i + 1].record()
            hatq.hatq_conv_int8_int_transition(layers[i], xq[i], act_hb[i + 1], tables[i], yq=xq[i + 1])
        if events:
            events[nL].record()
        hatq.hatq_conv_int8(layers[-1], xq[-1], s_last, hatq.HATQ_OUT_F32, y=ys[-1])
        if events:
            events[nL + 1].record()

    for _ in range(args.warmup):
        istep()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(nL + 2)] for _ in range(args.steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for k in range(args.steps):
        istep(ev[k])
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    log(f"integer stack: {ms:.3f} ms/step")

    def avg_us(a, b):
        return round(sum(ev[k][a].elapsed_time(ev[k][b]) for k in range(args.steps)) / args.steps * 1e3, 2)
    stages = {"act_quant_l1": avg_us(0, 1)}
    for i in range(nL - 1):
        stages[f"conv_l{i + 1}_int_transition"] = avg_us(i + 1, i + 2)
    stages[f"conv_l{nL}_f32"] = avg_us(nL, nL + 1)
    return {"ms_per_step": round(ms, 4),
            "tops": round(total_ops / (ms * 1e-3) / 1e12, 2),
            "mpix_per_s": round(img_pix / (ms * 1e-3) / 1e6, 1),
            "stages_us": stages,
            "static_scales": [float(f"{v:.6g}") for v in s_x],
            "shifts": shifts,
            "note": "integer-only transitions (fixed-point multiplier, integer bias, int64 "
                    "Hadamard transforms in the conv epilogue); static per-tensor scales"}


def measure_form_selection(args, wl, layers, x0, xq, sc, ys, tau=0.8):
    """The profiling pass of the form rule on this batch: for each layer's fp32
    input, the per-image range-expansion indicator with the layer's block, the
    probability p_l over the batch's images and the form it selects.  The pass
    over layer 2's input (the largest activation) is timed: it is one read of
    the tensor, HBM bound."""
    import torch
    from paper_2608_01653_amd import hatq
    n = x0.shape[0]
    # layer 1's fp32 output (the stack itself only forms its codes), from
    # dynamically quantized input codes
    L1 = wl.layers[0]
    hatq.hatq_fwht_quant_act(x0, L1.hblock if L1.form == "DH" else 1, xq=xq[0], scale=sc[0])
    hatq.hatq_conv_int8(layers[0], xq[0], sc[0], hatq.HATQ_OUT_F32, y=ys[0])
    inputs = [x0] + ys[:len(layers) - 1]
    p, sel = [], []
    amax = torch.empty(2 * n, dtype=torch.float32, device=x0.device)
    flags = torch.empty(n, dtype=torch.int32, device=x0.device)
    for L, xin in zip(wl.layers, inputs):
        count = torch.zeros(1, dtype=torch.int32, device=x0.device)
        hatq.hatq_range_expansion(xin, L.hblock, amax=amax, flags=flags, count=count)
        k = int(count.item())
        p.append(round(k / n, 4))
        sel.append(hatq.hatq_select_form(k, n, tau))
    x2 = inputs[1]
    reps = max(args.steps, 5)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    hatq.hatq_range_expansion(x2, wl.layers[1].hblock, amax=amax, flags=flags)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(reps):
        hatq.hatq_range_expansion(x2, wl.layers[1].hblock, amax=amax, flags=flags)
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) / reps * 1e3
    nbytes = x2.numel() * 4
    gbs = nbytes / (us * 1e-6) / 1e9
    log(f"form selection: p = {p}, selected {sel}; profiling pass {us:.1f} us")
    return {"tau": tau, "images": n, "p": p, "selected": sel,
            "configured": [L.form for L in wl.layers],
            "profile_pass": {"kernel": f"range_kernel<{wl.layers[1].hblock}> (layer 2 input)",
                             "us": round(us, 2), "bound": "hbm", "achieved": round(gbs, 1),
                             "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                             "work": f"{nbytes} bytes per call = {x2.numel()} fp32 elements read once"},
            "note": "random-init weights and synthetic inputs: the selection shows the mechanism, "
                    "not the paper's trained-model assignment"}


def measure_affine_layer(args, wl, layers, xq, ys, per_layer, li=2):
    """Layer 3 with affine dynamic activations (the paper's PTQ setting): the
    min / max pass and the affine quantization of its fp32 input, then the
    convolution with the zero-point correction, F32 output.  Timed on its own
    after the step, beside the symmetric layer's figures from the step."""
    import torch
    from paper_2608_01653_amd import hatq, workloads
    L = wl.layers[li]
    x = ys[li - 1]
    n = x.shape[0]
    dev = x.device
    hb = L.hblock if L.form == "DH" else 1
    scale = torch.empty(n, dtype=torch.float32, device=dev)
    zero = torch.empty(n, dtype=torch.int32, device=dev)
    ws = torch.empty(int(hatq.load().hatq_fwht_quant_affine_ws_bytes(n)), dtype=torch.int8, device=dev)
    tapsum = hatq.hatq_weight_tapsums(layers[li], device=dev)

    def run(events=None):
        if events:
            events[0].record()
        hatq.hatq_fwht_quant_act_affine(x, hb, xq=xq[li], scale=scale, zero=zero, ws=ws)
        if events:
            events[1].record()
        hatq.hatq_conv_int8_affine(layers[li], xq[li], scale, zero, tapsum, hatq.HATQ_OUT_F32, y=ys[li])
        if events:
            events[2].record()

    for _ in range(args.warmup):
        run()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        run(ev[k])
    torch.cuda.synchronize()
    tq = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps * 1e3
    tc = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps * 1e3
    ops = workloads.conv_ops(wl, li)
    elems = x.numel()
    z = zero.cpu().tolist()
    log(f"affine layer {li + 1}: quant {tq:.1f} us, conv {tc:.1f} us")
    return {"layer": per_layer[li]["layer"],
            "act_quant_affine_us": round(tq, 2),
            "act_quant_affine_gbs_alg": round(elems * 5 / (tq * 1e-6) / 1e9, 1),
            "act_quant_affine_passes": 2,
            "conv_affine_us": round(tc, 2),
            "conv_affine_tops": round(ops / (tc * 1e-6) / 1e12, 1),
            "symmetric_act_quant_us": per_layer[li]["act_quant_us"],
            "symmetric_conv_us": per_layer[li]["conv_us"],
            "zero_points": [min(z), max(z)],
            "note": "dynamic per-sample affine activations (min/max pass + quantization), "
                    "zero-point correction in the conv epilogue"}


def measure_order_layer(args, wl, params, xq, sc, ys, per_layer, li=2):
    """Layer 3 (DH, 192 input channels) with the paper's transform order
    m(192) = 192 (one Kronecker block P_12 (x) H~_16 over all channels) in place
    of blocks of 64: the two-pass activation quantization of its fp32 input and
    the convolution, timed after the step beside the block-64 layer."""
    import torch
    from paper_2608_01653_amd import hatq, workloads
    L = wl.layers[li]
    m = 192
    if L.form != "DH" or L.cin % m:
        return None
    dev = ys[0].device
    w, b = params[li]
    layer = hatq.hatq_prepare_weights(hatq.desc(L.cin, L.cout, L.k, L.stride, L.pad, m, L.transposed, L.out_pad),
                                      "DH", torch.from_numpy(w).to(dev), torch.from_numpy(b).to(dev))
    x = ys[li - 1]
    n = x.shape[0]
    ws = torch.empty(int(hatq.load().hatq_fwht_quant_ws_bytes(n)), dtype=torch.int8, device=dev)

    def run(events=None):
        if events:
            events[0].record()
        hatq.hatq_fwht_quant_act(x, m, xq=xq[li], scale=sc[li], ws=ws)
        if events:
            events[1].record()
        hatq.hatq_conv_int8(layer, xq[li], sc[li], hatq.HATQ_OUT_F32, y=ys[li])
        if events:
            events[2].record()

    for _ in range(args.warmup):
        run()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        run(ev[k])
    torch.cuda.synchronize()
    tq = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps * 1e3
    tc = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps * 1e3
    elems = x.numel()
    log(f"order-{m} layer {li + 1}: quant {tq:.1f} us, conv {tc:.1f} us")
    return {"layer": per_layer[li]["layer"], "order": m, "construction": "P_12 (x) H~_16 (Paley-I q = 11)",
            "act_quant_us": round(tq, 2), "act_quant_passes": 2,
            "act_quant_gbs_alg": round(elems * 9 / (tq * 1e-6) / 1e9, 1),
            "conv_us": round(tc, 2),
            "conv_tops": round(workloads.conv_ops(wl, li) / (tc * 1e-6) / 1e12, 1),
            "block64_act_quant_us": per_layer[li]["act_quant_us"], "block64_conv_us": per_layer[li]["conv_us"],
            "note": "two-pass quantization (the fused next-operand absmax covers blocks up to 64); "
                    "algorithmic bytes 4 B read twice + 1 B written per element"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="analysis_stack4_rgb_b16_1024x1024")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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

    import numpy as np
    import torch
    from paper_2608_01653_amd import build, hatq, workloads

    if build.stale() and not os.path.exists(build.LIB):
        build.build()
    hatq.load()
    wl = workloads.ALL[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    x_np, params = wl.generate()
    log(f"inputs generated: {wl.name} {wl.input_shape}")
    shapes = wl.shapes()
    n = wl.input_shape[0]
    x0 = torch.from_numpy(x_np).to(dev)
    layers = []
    for L, (w, b) in zip(wl.layers, params):
        d = hatq.desc(L.cin, L.cout, L.k, L.stride, L.pad, L.hblock, L.transposed, L.out_pad)
        layers.append(hatq.hatq_prepare_weights(d, L.form, torch.from_numpy(w).to(dev),
                                                torch.from_numpy(b).to(dev)))
    # buffers, all allocated before timing
    xq, sc, amax, ys = [], [], [], []
    for (ishape, oshape) in shapes:
        xq.append(torch.empty(ishape, dtype=torch.int8, device=dev))
        sc.append(torch.empty(n, dtype=torch.float32, device=dev))
        amax.append(torch.empty(n, dtype=torch.float32, device=dev))
        ys.append(torch.empty(oshape, dtype=torch.float32, device=dev))
    ws = torch.empty(int(hatq.load().hatq_fwht_quant_ws_bytes(n)), dtype=torch.int8, device=dev)
    act_hb = [L.hblock if L.form == "DH" else 1 for L in wl.layers]
    nL = len(wl.layers)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * nL + 1)]
          for _ in range(args.steps)]

    # Transition i -> i+1 through the requantizing epilogue when layer i's conv
    # is cheap to run twice (the small-cin row-run path: its fp32 output is the
    # largest tensor of the stack): an absmax-only pass, then the codes of the
    # next operand.  The codes equal those of the F32-output-then-quantize path.
    requant = [i + 1 < nL and wl.layers[i].cin <= 4 for i in range(nL)]

    def step(events=None):
        x = x0
        for i in range(nL):
            if events:
                events[2 * i].record()
            # layer 1 has no producer: two-pass absmax; later layers use the
            # absmax the previous epilogue produced (or the codes it wrote)
            if not (i > 0 and requant[i - 1]):
                hatq.hatq_fwht_quant_act(x, act_hb[i], absmax=None if i == 0 else amax[i - 1],
                                         xq=xq[i], scale=sc[i], ws=ws)
            if events:
                events[2 * i + 1].record()
            nxt = i + 1 < nL
            if requant[i]:
                hatq.hatq_conv_int8(layers[i], xq[i], sc[i], hatq.HATQ_OUT_F32, next_hblock=act_hb[i + 1],
                                    next_absmax=amax[i], absmax_only=True)
                hatq.hatq_conv_int8_requant(layers[i], xq[i], sc[i], act_hb[i + 1], next_absmax=amax[i],
                                            next_scale=sc[i + 1], yq=xq[i + 1])
            else:
                hatq.hatq_conv_int8(layers[i], xq[i], sc[i], hatq.HATQ_OUT_F32,
                                    next_hblock=act_hb[i + 1] if nxt else 0,
                                    next_absmax=amax[i] if nxt else None, y=ys[i])
            x = ys[i]
        if events:
            events[2 * nL].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for k in range(args.steps):
        step(ev[k])
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    log(f"timed {args.steps} steps: {total_ms / args.steps:.3f} ms/step")
    ms_step = total_ms / args.steps

    def avg_ms(a, b):
        return sum(ev[k][a].elapsed_time(ev[k][b]) for k in range(args.steps)) / args.steps

    total_ops = sum(workloads.conv_ops(wl, i) for i in range(nL))
    img_pix = n * wl.input_shape[1] * wl.input_shape[2]
    per_layer = []
    for i, L in enumerate(wl.layers):
        (ishape, oshape) = shapes[i]
        tq = avg_ms(2 * i, 2 * i + 1)
        tc = avg_ms(2 * i + 1, 2 * i + 2)
        elems = int(np.prod(ishape))
        ops = workloads.conv_ops(wl, i)
        out_pix = oshape[0] * oshape[1] * oshape[2]
        conv_bytes = elems + layers[i].cout_pad * layers[i].k_stride + out_pix * L.cout * (1 if requant[i] else 4)
        per_layer.append({
            "layer": f"L{i + 1} {L.form} {L.cin}->{L.cout} k{L.k}s{L.stride}",
            "act_quant_us": round(tq * 1e3, 2),
            "act_quant_passes": 2 if i == 0 else 0 if requant[i - 1] else 1,
            "conv_passes": 2 if requant[i] else 1,
            "conv_output": "int8 codes of the next operand" if requant[i] else "fp32",
            "act_quant_gbs_alg": round(elems * 5 / (tq * 1e-3) / 1e9, 1),
            "conv_us": round(tc * 1e3, 2),
            "conv_tops": round(ops / (tc * 1e-3) / 1e12, 1),
            "conv_mfma_frac": round(ops / (tc * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4),
            "conv_gbs_alg": round(conv_bytes / (tc * 1e-3) / 1e9, 1),
            "mpix_per_s_image": round(img_pix / ((tq + tc) * 1e-3) / 1e6, 1),
            "mpix_per_s_output": round(out_pix / ((tq + tc) * 1e-3) / 1e6, 1),
        })

    # dominant kernel: the layer-2 convolution (INT8 MFMA bound)
    t_conv2 = avg_ms(3, 4) * 1e-3
    ops2 = workloads.conv_ops(wl, 1)
    ach = ops2 / t_conv2 / 1e12
    roof = {"kernel": "conv_halo5_kernel<192,Epi<0,64>> (layer 2, DH 192->192 k5s2)", "bound": "mfma",
            "achieved": round(ach, 1), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
            "frac": round(ach / PEAK_INT8_TOPS, 4), "traffic": traffic_bytes("conv_l2"),
            "traffic_detail": measured_traffic("conv_l2"),
            "avg_us": round(t_conv2 * 1e6, 2),
            "work": f"{ops2} ops per launch = 2 x {n}x256x256 outputs x 192 x 5x5x192"}
    # the activation pass of the first layer quantized from a stored fp32 output
    qi = next(i for i in range(1, nL) if not requant[i - 1])
    t_q = avg_ms(2 * qi, 2 * qi + 1) * 1e-3
    eq = int(np.prod(shapes[qi][0]))
    achq = eq * 5 / t_q / 1e9
    roof_q = {"kernel": f"quant_kernel<{act_hb[qi]}> (layer {qi + 1}, single read)", "bound": "hbm",
              "achieved": round(achq, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
              "frac": round(achq / PEAK_HBM_GBS, 4), "traffic": traffic_bytes(f"quant_l{qi + 1}"),
              "traffic_detail": measured_traffic(f"quant_l{qi + 1}"),
              "avg_us": round(t_q * 1e6, 2),
              "work": f"{eq * 5} bytes per launch = {eq} elements x (4 B fp32 in + 1 B int8 out)"}

    # the same two kernels launched back to back on their resident inputs (the
    # last step's buffers), with no producer kernel before them: in the step,
    # the quantization reads the fp32 output the layer-2 conv has just written
    # and competes with its write-back
    def back_to_back(f, reps=20):
        for _ in range(3):
            f()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            f()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3
    t_qi = back_to_back(lambda: hatq.hatq_fwht_quant_act(ys[qi - 1], act_hb[qi], absmax=amax[qi - 1],
                                                        xq=xq[qi], scale=sc[qi], ws=ws))
    roof_q["isolated"] = {"avg_us": round(t_qi * 1e6, 2), "achieved": round(eq * 5 / t_qi / 1e9, 1),
                          "frac": round(eq * 5 / t_qi / 1e9 / PEAK_HBM_GBS, 4),
                          "note": "20 launches back to back on the resident layer input after the timed steps"}
    t_ci = back_to_back(lambda: hatq.hatq_conv_int8(layers[1], xq[1], sc[1], hatq.HATQ_OUT_F32,
                                                   next_hblock=act_hb[2], next_absmax=amax[1], y=ys[1]))
    roof["isolated"] = {"avg_us": round(t_ci * 1e6, 2), "achieved": round(ops2 / t_ci / 1e12, 1),
                        "frac": round(ops2 / t_ci / 1e12 / PEAK_INT8_TOPS, 4),
                        "note": "20 launches back to back on the resident layer input after the timed steps"}

    integer_stack = measure_integer_stack(args, wl, layers, x0, xq, sc, ys, ws, act_hb, total_ops, img_pix)
    form_selection = measure_form_selection(args, wl, layers, x0, xq, sc, ys)
    affine = measure_affine_layer(args, wl, layers, xq, ys, per_layer)
    order_m = measure_order_layer(args, wl, params, xq, sc, ys, per_layer)

    out = {
        "metric": "Hadamard-INT8 conv TOPS + Mpixel/s per layer; % of INT8 MFMA / HBM peak",
        "value": round(total_ops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded uniform RGB input, Student-t weights)",
        "config": {"workload": wl.name, "input": list(wl.input_shape),
                   "layers": [f"{L.form} {L.cin}->{L.cout} k{L.k}s{L.stride} b{L.hblock}"
                              for L in wl.layers],
                   "form_mask": ",".join(L.form for L in wl.layers), "parallelism": "none"},
        "mpix_per_s": round(img_pix / (ms_step * 1e-3) / 1e6, 1),
        "layers": per_layer,
        "roofline": roof,
        "roofline_act_quant": roof_q,
        "integer_stack": integer_stack,
        "form_selection": form_selection,
        "affine_layer": affine,
        "paper_order_layer": order_m,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, x_np, params)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
