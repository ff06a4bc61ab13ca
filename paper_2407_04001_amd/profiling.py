"""Summaries of rocprofv3 CSV output (kernel statistics and PMC counters).

    python -m paper_2407_04001_amd.profiling stats <kernel_stats.csv>
    python -m paper_2407_04001_amd.profiling counters <counter_collection.csv> [kernel-substring]

Counter values of one dispatch are summed over their instances (SEs, XCDs).
"""
from __future__ import annotations

import collections
import csv
import sys


def kernel_stats(path: str, top: int = 20):
    rows = list(csv.DictReader(open(path)))
    out = []
    for r in rows[:top]:
        out.append({"name": r["Name"].split("(")[0], "calls": int(r["Calls"]),
                    "total_us": float(r["TotalDurationNs"]) / 1e3,
                    "avg_us": float(r["AverageNs"]) / 1e3, "pct": float(r["Percentage"])})
    return out


def counters_by_dispatch(path: str):
    disp = collections.defaultdict(dict)
    meta = {}
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        disp[d][r["Counter_Name"]] = disp[d].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        meta[d] = (r["Kernel_Name"].split("(")[0], int(r["Grid_Size"]))
    return disp, meta


def counter_totals(path: str, kernel_substring: str):
    """Sum of each counter over the dispatches whose name contains the substring."""
    disp, meta = counters_by_dispatch(path)
    tot = collections.Counter()
    n = 0
    for d, c in disp.items():
        if kernel_substring in meta[d][0]:
            n += 1
            for k, v in c.items():
                tot[k] += v
    return dict(tot), n


def _main(argv):
    if len(argv) >= 2 and argv[0] == "stats":
        for r in kernel_stats(argv[1]):
            print(f"{r['name'][:60]:60s} {r['calls']:6d} {r['total_us']:12.1f} {r['avg_us']:10.2f} {r['pct']:6.2f}")
    elif len(argv) >= 2 and argv[0] == "counters":
        tot, n = counter_totals(argv[1], argv[2] if len(argv) > 2 else "")
        print(n, "dispatches")
        for k, v in sorted(tot.items()):
            print(f"{k:32s} {v:.6g}")
    else:
        print(__doc__)


if __name__ == "__main__":
    _main(sys.argv[1:])
