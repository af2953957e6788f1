"""Text summaries of rocprofv3 CSV output (kernel traces and PMC counters).

    python -m paper_2504_18583_amd.profile_summary trace <dir>/run_kernel_trace.csv [--last N]
    python -m paper_2504_18583_amd.profile_summary pmc <dir>/run_counter_collection.csv \
        --kernel NAME_SUBSTRING [--workgroups WG] [--skip N]

``trace`` groups dispatches by kernel (template arguments included) and
workgroup count -- the same template runs for the target and the draft with
different grids -- and prints calls and mean / min / max duration.  ``pmc``
averages each counter over the dispatches of one kernel and grid.
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


def pmc(path: str, kernel: str, workgroups: int, skip: int) -> str:
    rows = list(csv.DictReader(open(path)))
    vals = defaultdict(list)
    for r in rows:
        if kernel not in r["Kernel_Name"]:
            continue
        wgs = int(r["Grid_Size"]) // int(r["Workgroup_Size"])
        if workgroups and wgs != workgroups:
            continue
        vals[r["Counter_Name"]].append(float(r["Counter_Value"]))
    out = [f"kernel ~ {kernel!r}, workgroups {workgroups or 'any'}"]
    for name, v in sorted(vals.items()):
        v = v[skip:] if len(v) > skip else v
        out.append(f"{name}: dispatches {len(v)}, mean {statistics.mean(v):.1f}, "
                   f"min {min(v):.1f}, max {max(v):.1f}")
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
    a = ap.parse_args(argv)
    print(trace(a.csv, a.last) if a.mode == "trace" else pmc(a.csv, a.kernel, a.workgroups, a.skip))
    return 0


if __name__ == "__main__":
    sys.exit(main())
