"""Summarize rocprofv3 output per kernel launch shape.

    python3 -m paper_2608_01653_amd.profsum <results.db> [--title T] [--cmd C]
    python3 -m paper_2608_01653_amd.profsum --counters DIR [DIR ...] [--match S ...] [--title T] [--cmd C]

The first form reads a kernel-trace database (rocpd SQLite), groups dispatches
by (kernel name, grid size), so launches of one kernel on different layers are
reported separately, and prints a Markdown table of count / average / min / max
duration in microseconds.  The second reads the ``*_counter_collection.csv`` of
one or more ``rocprofv3 --pmc`` passes and prints, per (kernel, grid) whose name
contains one of the --match strings, the median of each counter over its
dispatches.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import re
import sqlite3
import statistics
from collections import defaultdict


def short(name: str) -> str:
    name = re.sub(r"\(anonymous namespace\)::", "", name)
    name = re.sub(r"^void ", "", name)
    name = re.sub(r"\(.*\)$", "", name)
    return name.replace("hatq::", "")


def summarize(db: str):
    c = sqlite3.connect(db)
    rows = c.execute("select name, grid_x, grid_y, grid_z, workgroup_x, duration from kernels").fetchall()
    groups = defaultdict(list)
    for name, gx, gy, gz, wx, dur in rows:
        groups[(short(name), gx, gy, gz, wx)].append(dur / 1e3)
    out = []
    for (name, gx, gy, gz, wx), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append((name, f"{gx}x{gy}x{gz}/{wx}", len(d), statistics.mean(d), min(d), max(d), sum(d)))
    return out


XCDS = 8   # GRBM_COUNT / GRBM_GUI_ACTIVE sum one count per XCD per clock


def counters(dirs, match):
    """{(kernel, grid): {counter: (median value per dispatch, dispatches)}} over the
    passes in dirs, with the median dispatch duration ("dur_us", from the
    dispatch timestamps of the counter runs) and, where GRBM_GUI_ACTIVE was
    collected, the mean shader clock over the dispatch ("clock_GHz")."""
    per = defaultdict(lambda: defaultdict(list))
    for d in dirs:
        for p in glob.glob(os.path.join(d, "*_counter_collection.csv")):
            seen = set()
            for r in csv.DictReader(open(p)):
                name = short(r["Kernel_Name"])
                if match and not any(m in name for m in match):
                    continue
                key = (name, int(r["Grid_Size"]))
                dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
                per[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
                if (p, r["Dispatch_Id"]) not in seen:
                    seen.add((p, r["Dispatch_Id"]))
                    per[key]["dur_us"].append(dur)
                if r["Counter_Name"] == "GRBM_GUI_ACTIVE" and dur > 0:
                    per[key]["clock_GHz"].append(float(r["Counter_Value"]) / XCDS / (dur * 1e3))
    return {k: {c: (statistics.median(v), len(v)) for c, v in cs.items()} for k, cs in per.items()}


def main_counters(a):
    res = counters(a.counters, a.match)
    print(f"# {a.title}\n")
    if a.cmd:
        print(f"Commands: `{a.cmd}`\n")
    names = sorted({c for cs in res.values() for c in cs})
    print("| kernel | grid (threads) | " + " | ".join(names) + " |")
    print("|---|---|" + "---|" * len(names))
    for (name, grid), cs in sorted(res.items()):
        vals = [f"{cs[c][0]:.4g}" if c in cs else "" for c in names]
        print(f"| `{name}` | {grid} | " + " | ".join(vals) + " |")
    print("\n(medians per dispatch; dispatches per kernel: " +
          ", ".join(f"`{n}` {max(v[1] for v in cs.values())}" for (n, _), cs in sorted(res.items())) + ")")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="?")
    ap.add_argument("--counters", nargs="+")
    ap.add_argument("--match", nargs="*", default=[])
    ap.add_argument("--title", default="rocprofv3 kernel trace")
    ap.add_argument("--cmd", default="")
    a = ap.parse_args()
    if a.counters:
        main_counters(a)
        return
    rows = summarize(a.db)
    total = sum(r[6] for r in rows)
    print(f"# {a.title}\n")
    if a.cmd:
        print(f"Command: `{a.cmd}`\n")
    print("| kernel | grid (threads) / block | calls | avg us | min us | max us | % time |")
    print("|---|---|---|---|---|---|---|")
    for name, g, n, avg, mn, mx, tot in rows:
        print(f"| `{name}` | {g} | {n} | {avg:.1f} | {mn:.1f} | {mx:.1f} | {100 * tot / total:.1f} |")


if __name__ == "__main__":
    main()
