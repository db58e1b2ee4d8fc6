"""Summarise a rocprofv3 kernel trace (CSV) per kernel and launch shape.

Usage: python -m paper_1712_04432_amd.profile_summary <..._kernel_trace.csv> [--title TEXT]
       python -m paper_1712_04432_amd.profile_summary <run_counter_collection.csv> --counter NAME --kernel SUBSTR
       python -m paper_1712_04432_amd.profile_summary <run_counter_collection.csv> --mfma

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


def summarize(path: str, per_step_ref: str = ""):
    """Group launches by (kernel, grid, workgroup size). With per_step_ref (a kernel that
    runs once per step), a group with n launches per step is split further by the
    launch's position within the step, so that e.g. the layers of one kernel separate."""
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    groups = collections.defaultdict(list)
    for r in rows:
        wg = int(r["Workgroup_Size_X"]) * int(r.get("Workgroup_Size_Y", 1) or 1) * int(r.get("Workgroup_Size_Z", 1) or 1)
        items = int(r["Grid_Size_X"]) * int(r.get("Grid_Size_Y", 1) or 1) * int(r.get("Grid_Size_Z", 1) or 1)
        grid = items // max(wg, 1)
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0
        groups[(short_name(r["Kernel_Name"]), grid, wg)].append(dur)
    if per_step_ref:
        steps = sum(len(v) for k, v in groups.items() if per_step_ref in k[0])
        split = collections.defaultdict(list)
        for (name, grid, wg), v in groups.items():
            per = len(v) // steps if steps and len(v) % steps == 0 and len(v) >= steps else 1
            for i, d in enumerate(v):
                split[(name if per == 1 else f"{name} [{i % per + 1}/{per}]", grid, wg)].append(d)
        groups = split
    total = sum(sum(v) for v in groups.values())
    out = []
    for (name, grid, wg), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append({"kernel": name, "workgroups": grid, "wg_size": wg, "launches": len(v),
                    "avg_us": statistics.mean(v), "median_us": statistics.median(v), "min_us": min(v),
                    "max_us": max(v), "share": sum(v) / total if total else 0.0})
    return out


def counter_per_dispatch(path: str, kernel: str, counter: str):
    """Per-dispatch totals of one counter (summed over the instances rocprofv3 reports)
    for the dispatches whose kernel name contains `kernel`, in dispatch order."""
    tot = collections.OrderedDict()
    for r in csv.DictReader(open(path)):
        if kernel in r["Kernel_Name"] and r["Counter_Name"] == counter:
            d = int(r["Dispatch_Id"])
            tot[d] = tot.get(d, 0.0) + float(r["Counter_Value"])
    return [tot[d] for d in sorted(tot)]


def mfma_utilisation(path: str, simds: int = 1024, xcds: int = 8):
    """Per (kernel, grid) of a --pmc run with SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE:
    the matrix-pipe utilisation MFMA_BUSY / (cycles x SIMDs), MFMA_BUSY counting the busy
    cycles of every SIMD's matrix pipe (16 per 16x16x32 bf16 MFMA). Two cycle counts:
    GRBM_GUI_ACTIVE per XCD (it is summed over the XCDs; the measured clock, but its
    window also covers the dispatch's launch and drain, which inflates it for launches of
    a few microseconds), and the dispatch's duration at the 2.4 GHz peak clock (the share
    of the dense peak). Medians over the dispatches of each group."""
    disp = collections.OrderedDict()
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        e = disp.setdefault(d, {"name": short_name(r["Kernel_Name"]), "grid": int(r["Grid_Size"]),
                                "wg": int(r["Workgroup_Size"]),
                                "dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    groups = collections.defaultdict(list)
    for e in disp.values():
        if e.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) > 0 and e.get("GRBM_GUI_ACTIVE", 0.0) > 0:
            cyc = e["GRBM_GUI_ACTIVE"] / xcds
            groups[(e["name"], e["grid"] // max(e["wg"], 1), e["wg"])].append(
                (e["dur"], cyc / e["dur"] / 1e3, e["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * simds),
                 e["SQ_VALU_MFMA_BUSY_CYCLES"] / (e["dur"] * 2.4e3 * simds)))
    out = []
    for (name, grid, wg), v in groups.items():
        out.append({"kernel": name, "workgroups": grid, "wg_size": wg, "dispatches": len(v),
                    "dur_us": statistics.median(x[0] for x in v), "clock_ghz": statistics.median(x[1] for x in v),
                    "mfma_util": statistics.median(x[2] for x in v),
                    "mfma_peak": statistics.median(x[3] for x in v)})
    return sorted(out, key=lambda r: -r["dur_us"] * r["dispatches"])


def counter_table(path: str, per_step_ref: str = ""):
    """Per (kernel, grid, position in the step) group of a --pmc run: the median over its
    dispatches of every counter collected (each summed over the instances rocprofv3
    reports for a dispatch) and of the dispatch's duration."""
    disp = collections.OrderedDict()
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        e = disp.setdefault(d, {"name": short_name(r["Kernel_Name"]), "grid": int(r["Grid_Size"]) // max(int(r["Workgroup_Size"]), 1),
                                "wg": int(r["Workgroup_Size"]),
                                "dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0, "c": {}})
        e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    seq = list(disp.values())
    steps = sum(1 for e in seq if per_step_ref and per_step_ref in e["name"])
    groups = collections.defaultdict(list)
    for e in seq:
        groups[(e["name"], e["grid"], e["wg"])].append(e)
    out = []
    for (name, grid, wg), v in groups.items():
        per = len(v) // steps if steps and len(v) % steps == 0 and len(v) >= steps else 1
        for k in range(per):
            sub = v[k::per]
            label = name if per == 1 else f"{name} [{k + 1}/{per}]"
            names = sorted({c for e in sub for c in e["c"]})
            out.append({"kernel": label, "workgroups": grid, "wg_size": wg, "dispatches": len(sub),
                        "dur_us": statistics.median(e["dur"] for e in sub),
                        "counters": {c: statistics.median(e["c"].get(c, 0.0) for e in sub) for c in names}})
    return sorted(out, key=lambda r: -r["dur_us"] * r["dispatches"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace")
    ap.add_argument("--title", default="")
    ap.add_argument("--top", type=int, default=30)
    ap.add_argument("--counter", default="", help="summarise this counter of a --pmc run instead")
    ap.add_argument("--kernel", default="", help="kernel-name substring for --counter")
    ap.add_argument("--per-step-ref", default="", help="kernel launched once per step (splits layers)")
    ap.add_argument("--period", type=int, default=1,
                    help="dispatches of the kernel per step; one median per position in the step")
    ap.add_argument("--mfma", action="store_true",
                    help="matrix-pipe utilisation per kernel of a --pmc run with SQ_VALU_MFMA_BUSY_CYCLES "
                         "and GRBM_GUI_ACTIVE")
    ap.add_argument("--counters", action="store_true",
                    help="every counter of a --pmc run, median per dispatch, per kernel and grid")
    a = ap.parse_args()
    if a.counters:
        rows = counter_table(a.trace, a.per_step_ref)[:a.top]
        names = sorted({c for r in rows for c in r["counters"]})
        print("| kernel | workgroups x size | dispatches | median us | " + " | ".join(names) + " |")
        print("|---|---|---|---|" + "---|" * len(names))
        for r in rows:
            print(f"| `{r['kernel']}` | {r['workgroups']} x {r['wg_size']} | {r['dispatches']} | {r['dur_us']:.2f} | "
                  + " | ".join(f"{r['counters'].get(c, 0.0):.4g}" for c in names) + " |")
        return
    if a.mfma:
        print("| kernel | workgroups x size | dispatches | median us | GUI clock GHz | MFMA busy of GUI cycles | "
              "MFMA busy at 2.4 GHz |")
        print("|---|---|---|---|---|---|---|")
        for r in mfma_utilisation(a.trace)[:a.top]:
            print(f"| `{r['kernel']}` | {r['workgroups']} x {r['wg_size']} | {r['dispatches']} | {r['dur_us']:.2f} | "
                  f"{r['clock_ghz']:.2f} | {100 * r['mfma_util']:.1f}% | {100 * r['mfma_peak']:.1f}% |")
        return
    if a.counter:
        v = counter_per_dispatch(a.trace, a.kernel, a.counter)
        print(f"{a.counter} per dispatch of '{a.kernel}' ({len(v)} dispatches)")
        for k in range(a.period):
            s = v[k::a.period]
            if s:
                print(f"  position {k}: median {statistics.median(s):.1f}  min {min(s):.1f}  max {max(s):.1f}  (n={len(s)})")
        return
    rows = summarize(a.trace, a.per_step_ref)
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
