"""Summarise a rocprofv3 kernel trace (CSV) per kernel and launch shape.

Usage: python -m paper_1712_04432_amd.profile_summary <..._kernel_trace.csv> [--title TEXT]

rocprofv3's own --stats groups launches by kernel symbol only; the weight-gradient
kernel of every layer is one symbol, so this groups by (symbol, grid size) as well and
prints a markdown table with the launch count and the average/min/max duration.
"""
from __future__ import annotations

import argparse
import collections
import csv
import re
import statistics


def short_name(name: str) -> str:
    name = re.sub(r"\(anonymous namespace\)::", "", name)
    name = re.sub(r"^void ", "", name)
    name = re.sub(r"\(.*\)$", "", name)
    return name.replace("imbd::", "").replace("unsigned short", "bf16")


def summarize(path: str):
    rows = list(csv.DictReader(open(path)))
    groups = collections.defaultdict(list)
    for r in rows:
        wg = int(r["Workgroup_Size_X"]) * int(r.get("Workgroup_Size_Y", 1) or 1) * int(r.get("Workgroup_Size_Z", 1) or 1)
        items = int(r["Grid_Size_X"]) * int(r.get("Grid_Size_Y", 1) or 1) * int(r.get("Grid_Size_Z", 1) or 1)
        grid = items // max(wg, 1)
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0
        groups[(short_name(r["Kernel_Name"]), grid, wg)].append(dur)
    total = sum(sum(v) for v in groups.values())
    out = []
    for (name, grid, wg), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append({"kernel": name, "workgroups": grid, "wg_size": wg, "launches": len(v),
                    "avg_us": statistics.mean(v), "median_us": statistics.median(v), "min_us": min(v),
                    "max_us": max(v), "share": sum(v) / total if total else 0.0})
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace")
    ap.add_argument("--title", default="")
    ap.add_argument("--top", type=int, default=30)
    a = ap.parse_args()
    rows = summarize(a.trace)
    if a.title:
        print(a.title)
        print()
    print("| kernel | workgroups x size | launches | avg us | median us | min us | max us | share |")
    print("|---|---|---|---|---|---|---|---|")
    for r in rows[:a.top]:
        print(f"| `{r['kernel']}` | {r['workgroups']} x {r['wg_size']} | {r['launches']} | {r['avg_us']:.2f} | "
              f"{r['median_us']:.2f} | {r['min_us']:.2f} | {r['max_us']:.2f} | {100 * r['share']:.1f}% |")


if __name__ == "__main__":
    main()
