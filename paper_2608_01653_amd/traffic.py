"""HBM traffic per kernel launch from rocprofv3 counter runs of bench.py.

    python3 -m paper_2608_01653_amd.traffic FETCH_DIR WRITE_DIR CAL_FETCH_DIR CAL_WRITE_DIR [-o out.json]

Each directory holds the ``*_counter_collection.csv`` of one ``rocprofv3 --pmc``
pass (FETCH_SIZE or WRITE_SIZE, in KiB per dispatch).  The two calibration
passes profile ``bench.py --calibrate-copy`` (1 GiB device copies); the ratio of
the known copy size to what each counter reads scales the bench's counters to
bytes.  Launches are identified by their order within one step of the
four-layer stack: layer 1 runs the small-cin convolution twice
(``conv_rr32_kernel``: the absmax pass, then the requantizing pass that writes
layer 2's codes; ``conv_rowrun_kernel`` in the paired leg), so the first window
convolution with the F32 epilogue that also forms the next blocks-of-64 absmax
(``Epi<0, 64, 0>``; the integer stack's layer 2 uses another variant) after such
a launch is layer 2's convolution and the first ``quant_kernel<64>`` after it is
layer 3's quantization.  Layer 1's two passes are reported too.  The output JSON
carries a hash of the kernel sources; bench.py reports the traffic only while
the sources are unchanged.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import statistics
import sys

GIB_KIB = 1 << 20   # 1 GiB in KiB


def rows(d):
    out = []
    for p in glob.glob(os.path.join(d, "*_counter_collection.csv")):
        out += list(csv.DictReader(open(p)))
    out.sort(key=lambda r: int(r["Dispatch_Id"]))
    return out


def copy_factor(d):
    vals = [float(r["Counter_Value"]) for r in rows(d) if "copyBuffer" in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no copy dispatches in {d}")
    return GIB_KIB / statistics.median(vals)


def per_launch(d, factor):
    """KiB counter -> bytes, median over the steps, for layer 1's two passes, the
    layer-2 conv and the layer-3 quantization."""
    conv, quant, l1a, l1q = [], [], [], []
    want_q = want_c = False
    for r in rows(d):
        name = r["Kernel_Name"]
        v = float(r["Counter_Value"]) * factor * 1024
        if "conv_rr32_kernel" in name:
            # template arguments <TH, CIN, NS, PASS, MINB>: PASS 0 absmax, 1 codes
            (l1a if name.split("<")[1].split(",")[3].strip() == "0" else l1q).append(v)
            want_c = True
        elif "conv_rowrun_kernel" in name:
            want_c = True
        elif "conv_halo5_kernel<192" in name and "Epi<0, 64, 0>" in name and want_c:
            conv.append(v)
            want_c = False
            want_q = True
        elif "quant_kernel<64>" in name and want_q:
            quant.append(v)
            want_q = False
    med = lambda xs: statistics.median(xs) if xs else None
    return {"conv_l2": med(conv), "quant_l3": med(quant), "absmax_pass_l1": med(l1a), "codes_pass_l1": med(l1q)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("fetch")
    ap.add_argument("write")
    ap.add_argument("cal_fetch")
    ap.add_argument("cal_write")
    ap.add_argument("-o", "--out")
    a = ap.parse_args()
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench
    ff, fw = copy_factor(a.cal_fetch), copy_factor(a.cal_write)
    f, w = per_launch(a.fetch, ff), per_launch(a.write, fw)
    res = {"source_hash": bench.kernel_source_hash(),
           "calibration": {"fetch_factor": round(ff, 4), "write_factor": round(fw, 4),
                           "method": "1 GiB device copy (bench.py --calibrate-copy)"},
           "kernels": {k: {"fetch_bytes": f[k], "write_bytes": w[k],
                           "bytes": (f[k] or 0) + (w[k] or 0)} for k in f}}
    txt = json.dumps(res, indent=1)
    if a.out:
        open(a.out, "w").write(txt + "\n")
    print(txt)


if __name__ == "__main__":
    main()
