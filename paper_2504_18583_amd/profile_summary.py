"""Text summaries of rocprofv3 CSV output (kernel traces and PMC counters).

    python -m paper_2504_18583_amd.profile_summary trace <dir>/run_kernel_trace.csv [--last N]
    python -m paper_2504_18583_amd.profile_summary pmc <dir>/run_counter_collection.csv \
        --kernel NAME_SUBSTRING [--workgroups WG] [--skip N] [--at-max COUNTER]
    python -m paper_2504_18583_amd.profile_summary window <dir>/run_counter_collection.csv \
        --after NAME_SUBSTRING

``trace`` groups dispatches by kernel (template arguments included) and
workgroup count -- the same template runs for the target and the draft with
different grids -- and prints calls and mean / min / max duration.  ``pmc``
averages each counter over the dispatches of one kernel and grid (with
``--at-max``, only over the dispatches whose value of that counter is the
largest seen: e.g. the full-size passes of a GEMM whose shorter prefill passes
share its grid).
``window`` sums each counter over every dispatch after the last dispatch of a
marker kernel, in total and per kernel (a program's measured region).
"""
from __future__ import annotations

import argparse
import csv
import re
import statistics
import sys
from collections import defaultdict


def _short(name: str) -> str:
    m = re.search(r"(k_\w+)(<[^(]*>)?", name)
    return m.group(0) if m else name[:48]


def trace(path: str, last: int) -> str:
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    if last > 0:
        rows = rows[-last:]
    groups = defaultdict(list)
    for r in rows:
        wgs = (int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"])) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
        groups[(_short(r["Kernel_Name"]), wgs, int(r["Workgroup_Size_X"]))].append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    span = (int(rows[-1]["End_Timestamp"]) - int(rows[0]["Start_Timestamp"])) / 1e3
    busy = sum(sum(v) for v in groups.values())
    out = [f"dispatches {len(rows)}, busy {busy:.1f} us over a span of {span:.1f} us",
           f"{'kernel':34s} {'WGs':>6s} {'thr':>5s} {'calls':>6s} {'mean_us':>9s} {'min_us':>8s} "
           f"{'max_us':>8s} {'total_us':>10s}"]
    for (name, wgs, thr), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"{name:34s} {wgs:6d} {thr:5d} {len(v):6d} {statistics.mean(v):9.2f} {min(v):8.2f} "
                   f"{max(v):8.2f} {sum(v):10.1f}")
    return "\n".join(out)


def pmc(path: str, kernel: str, workgroups: int, skip: int, at_max: str = "") -> str:
    rows = list(csv.DictReader(open(path)))
    key = "Dispatch_Id" if rows and "Dispatch_Id" in rows[0] else "Correlation_Id"
    disp = {}
    for r in rows:
        if kernel not in r["Kernel_Name"]:
            continue
        wgs = int(r["Grid_Size"]) // int(r["Workgroup_Size"])
        if workgroups and wgs != workgroups:
            continue
        disp.setdefault(int(r[key]), {})[r["Counter_Name"]] = float(r["Counter_Value"])
    order = [disp[k] for k in sorted(disp)]
    order = order[skip:] if len(order) > skip else order
    if at_max:
        top = max((d.get(at_max, float("-inf")) for d in order), default=0.0)
        order = [d for d in order if d.get(at_max) == top]
    vals = defaultdict(list)
    for d in order:
        for name, v in d.items():
            vals[name].append(v)
    sel = f", dispatches at the largest {at_max}" if at_max else ""
    out = [f"kernel ~ {kernel!r}, workgroups {workgroups or 'any'}{sel}"]
    for name, v in sorted(vals.items()):
        out.append(f"{name}: dispatches {len(v)}, mean {statistics.mean(v):.1f}, "
                   f"min {min(v):.1f}, max {max(v):.1f}")
    return "\n".join(out)


def window(path: str, after: str) -> str:
    rows = list(csv.DictReader(open(path)))
    if not rows:
        return "no dispatches"
    key = "Dispatch_Id" if "Dispatch_Id" in rows[0] else "Correlation_Id"
    disp = {}
    for r in rows:
        d = disp.setdefault(int(r[key]), {"name": r["Kernel_Name"], "c": defaultdict(float)})
        d["c"][r["Counter_Name"]] += float(r["Counter_Value"])
    order = sorted(disp)
    marks = [i for i, k in enumerate(order) if after in disp[k]["name"]]
    if not marks:
        return f"no dispatch of {after!r}"
    sel = [disp[k] for k in order[marks[-1] + 1:]]
    tot = defaultdict(float)
    per = defaultdict(lambda: [0, defaultdict(float)])
    for d in sel:
        e = per[_short(d["name"])]
        e[0] += 1
        for c, v in d["c"].items():
            tot[c] += v
            e[1][c] += v
    out = [f"dispatches after the last {after!r}: {len(sel)}"]
    for c, v in sorted(tot.items()):
        out.append(f"{c}: total {v:.1f}")
    names = sorted(tot)
    out.append(f"{'kernel':34s} {'calls':>6s} " + " ".join(f"{c:>16s}" for c in names))
    for k, (n, cs) in sorted(per.items(), key=lambda kv: -sum(kv[1][1].values())):
        out.append(f"{k:34s} {n:6d} " + " ".join(f"{cs[c]:16.1f}" for c in names))
    return "\n".join(out)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    t = sub.add_parser("trace")
    t.add_argument("csv")
    t.add_argument("--last", type=int, default=0)
    p = sub.add_parser("pmc")
    p.add_argument("csv")
    p.add_argument("--kernel", required=True)
    p.add_argument("--workgroups", type=int, default=0)
    p.add_argument("--skip", type=int, default=0)
    p.add_argument("--at-max", default="")
    w = sub.add_parser("window")
    w.add_argument("csv")
    w.add_argument("--after", required=True)
    a = ap.parse_args(argv)
    if a.mode == "trace":
        print(trace(a.csv, a.last))
    elif a.mode == "pmc":
        print(pmc(a.csv, a.kernel, a.workgroups, a.skip, a.at_max))
    else:
        print(window(a.csv, a.after))
    return 0


if __name__ == "__main__":
    sys.exit(main())
