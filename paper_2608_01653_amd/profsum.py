"""Summarize a rocprofv3 kernel-trace database (rocpd SQLite) per kernel launch shape.

    python3 -m paper_2608_01653_amd.profsum <results.db> [--title T] [--cmd C]

Groups dispatches by (kernel name, grid size), so launches of one kernel on
different layers are reported separately, and prints a Markdown table of
count / average / min / max duration in microseconds.
"""
from __future__ import annotations

import argparse
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("db")
    ap.add_argument("--title", default="rocprofv3 kernel trace")
    ap.add_argument("--cmd", default="")
    a = ap.parse_args()
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
