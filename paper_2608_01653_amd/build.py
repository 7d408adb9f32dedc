"""Build libhatq.so (the C-ABI library) for gfx950 with hipcc, in-tree.

Flags: -O3, gfx950 only, no fast-math, no FP contraction (the epilogue uses
explicit fma where the arithmetic contract says fma), fp32 denormals kept, and
packed-FP32 instructions disabled.

Every source compiles to an object of its own, in parallel; conv_i8.hip is
compiled once per part of its dispatch (HATQ_CONV_PART), since its kernel
instantiations take most of the build time. The objects are linked into one
shared library.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libhatq.so")
SOURCES = ["api.cpp", "act_quant.hip", "conv_i8.hip", "weights.hip"]
CONV_PARTS = 14         # HATQ_CONV_PART = 0 .. 13 in conv_i8.hip
OBJ_DIR = os.path.join(ROOT, "_build", "hatq")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"),
]


def sources():
    return [os.path.join(CSRC, s) for s in SOURCES]


def _units():
    """(source, extra flags, object) for every compilation."""
    units = []
    for src in sources():
        base = os.path.splitext(os.path.basename(src))[0]
        if base == "conv_i8":
            for k in range(CONV_PARTS):
                units.append((src, [f"-DHATQ_CONV_PART={k}"], os.path.join(OBJ_DIR, f"{base}.part{k}.o")))
        else:
            units.append((src, [], os.path.join(OBJ_DIR, base + ".o")))
    return units


# hipcc's host pass does not know the packed-fp32 feature and says so
_NOISE = "'-packed-fp32-ops' is not a recognized feature"


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if _NOISE not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, jobs: int = 0) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    cmds = [[HIPCC, *compile_flags, *extra, "-c", src, "-o", obj] for src, extra, obj in _units()]
    jobs = jobs or max(1, min(len(cmds), len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as pool:
        for cmd, err in zip(cmds, pool.map(_run, cmds)):
            if verbose:
                print(" ".join(cmd), flush=True)
                if err.strip():
                    print(err, file=sys.stderr)
    tmp = LIB + ".tmp"
    # -z defs: a symbol left unresolved (a part's entry point that another
    # compilation of conv_i8.hip does not define) fails the link, not the load
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,-z,defs", *[o for _, _, o in _units()],
          "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    deps = sources() + [os.path.join(CSRC, f) for f in os.listdir(CSRC)] + \
        [os.path.join(ROOT, "include", "hatq.h")]
    return any(os.path.getmtime(p) > t for p in deps)


if __name__ == "__main__":
    print(build(verbose=True))
