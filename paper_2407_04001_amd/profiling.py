"""Summaries of rocprofv3 CSV output (kernel statistics and PMC counters).

    python -m paper_2407_04001_amd.profiling stats <kernel_stats.csv>
    python -m paper_2407_04001_amd.profiling counters <counter_collection.csv> [kernel-substring]
    python -m paper_2407_04001_amd.profiling report <prof_dir> <workload> <cells> <commands.json>

Counter values of one dispatch are summed over their instances (SEs, XCDs).
"""
from __future__ import annotations

import collections
import csv
import hashlib
import json
import os
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




# ------------------------------------------------------------------ report
def _searches(rows):
    """Split dispatch rows (sorted by start) into searches; each search begins
    with the cost-table kernel."""
    out, cur = [], None
    for r in rows:
        if r["name"].startswith("k_cost_tables"):
            cur = []
            out.append(cur)
        if cur is not None:
            cur.append(r)
    return out


def _template_args(name):
    if "<" not in name:
        return []
    inner = name[name.index("<") + 1:name.rindex(">")]
    return [x.strip() for x in inner.split(",")]


def is_column_fill(name):
    """The dominant kernel: the row fill with a column chunk per lane (TZ > 1)."""
    if not name.startswith("void k_fill_rows<"):
        return False
    args = _template_args(name)
    return len(args) >= 2 and int(args[1]) > 1


def trace_rows(path):
    rows = []
    for r in csv.DictReader(open(path)):
        rows.append({"name": r["Kernel_Name"].split("(")[0], "start": int(r["Start_Timestamp"]),
                     "end": int(r["End_Timestamp"]), "grid": int(r["Grid_Size_X"])})
    rows.sort(key=lambda r: r["start"])
    return rows


def counter_rows(path):
    disp, meta = counters_by_dispatch(path)
    rows = [{"name": meta[d][0], "dispatch": d, "grid": meta[d][1], **disp[d]} for d in sorted(disp)]
    return rows


def _find_csv(d, suffix):
    for root, _, files in os.walk(d):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    raise FileNotFoundError(f"no *{suffix} under {d}")


def report(trace_dir, fetch_dir, write_dir, cfetch_dir, cwrite_dir, valu_dir, workload, cells, src_hash,
           commands):
    """Kernel-time table, copy-calibrated HBM traffic and VALU issue of the
    strategy search, as markdown plus the per-launch traffic record that the
    benchmark reads."""
    # kernel time: every search but the first (warm-up)
    tr = _searches(trace_rows(_find_csv(trace_dir, "kernel_trace.csv")))[1:]
    ns = len(tr)
    agg = collections.OrderedDict()
    span = busy = 0
    for s in tr:
        span += s[-1]["end"] - s[0]["start"]
        for r in s:
            a = agg.setdefault(r["name"], [0, 0])
            a[0] += 1
            a[1] += r["end"] - r["start"]
            busy += r["end"] - r["start"]
    tot = sum(v[1] for v in agg.values())
    col_launch = sum(v[0] for k, v in agg.items() if is_column_fill(k)) / ns
    col_us = sum(v[1] for k, v in agg.items() if is_column_fill(k)) / ns / 1e3

    # calibration: plain 1 GiB device copies (the fill kernel of the source
    # tensor writes 1 GiB and reads nothing)
    def cal(d, counter, copies=3, fill_writes=True):
        rows = counter_rows(_find_csv(d, "counter_collection.csv"))
        total = sum(r.get(counter, 0.0) for r in rows) * 1024.0
        copied = copies * (1 << 30)
        if counter == "WRITE_SIZE" and fill_writes:
            copied += 1 << 30
        return total / copied
    kf, kw = cal(cfetch_dir, "FETCH_SIZE"), cal(cwrite_dir, "WRITE_SIZE")

    def per_search(d, counter, scale):
        rows = counter_rows(_find_csv(d, "counter_collection.csv"))
        s = _searches(rows)[-1]   # the second (timed) search of the run
        col = sum(r.get(counter, 0.0) for r in s if is_column_fill(r["name"])) * 1024.0 / scale
        allk = sum(r.get(counter, 0.0) for r in s) * 1024.0 / scale
        n = sum(1 for r in s if is_column_fill(r["name"]))
        return col, allk, n
    f_col, f_all, n_col = per_search(fetch_dir, "FETCH_SIZE", kf)
    w_col, w_all, _ = per_search(write_dir, "WRITE_SIZE", kw)

    vrows = _searches(counter_rows(_find_csv(valu_dir, "counter_collection.csv")))[-1]

    L = []
    L.append(f"# Kernel profile: {workload} strategy search on one MI355X\n")
    L.append(f"{cells:.3e} DP cell updates per search. Summary written by "
             "`python -m paper_2407_04001_amd.profiling report` from the rocprofv3 output of the commands below "
             f"(kernel sources sha256 `{src_hash[:16]}…`).\n")
    L.append("## Kernel time (rocprofv3 kernel trace)\n")
    L.append("Command (from the repository root, after `cd /tmp && export TMPDIR=/tmp`):\n")
    L.append(f"    {commands['trace']}\n")
    L.append(f"{ns} timed searches (the warm-up search is dropped). Per search: {span / ns / 1e3:.1f} us from the first "
             f"kernel start to the last kernel end, {busy / ns / 1e3:.1f} us inside kernels, "
             f"{sum(v[0] for v in agg.values()) / ns:.0f} launches.\n")
    L.append("| kernel | launches / search | time / search (us) | avg per launch (us) | share |")
    L.append("|---|---|---|---|---|")
    for k, (c, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        L.append(f"| `{k}` | {c / ns:.0f} | {t / ns / 1e3:.1f} | {t / c / 1e3:.2f} | {100 * t / tot:.1f}% |")
    L.append("")
    L.append(f"Dominant kernel: `k_fill_rows` with a column chunk per lane (TZ > 1): {col_launch:.0f} launches, "
             f"{col_us:.1f} us per search, {col_us / col_launch:.1f} us average per launch.\n")
    L.append("## HBM traffic (rocprofv3 PMC, copy-calibrated)\n")
    L.append("Commands:\n")
    for k in ("fetch", "write", "cfetch", "cwrite"):
        L.append(f"    {commands[k]}")
    L.append("")
    L.append(f"Calibration (counter bytes / bytes moved by three plain 1 GiB device copies; the write counter also "
             f"sees the 1 GiB fill of the source): FETCH_SIZE {kf:.4f}, WRITE_SIZE {kw:.4f}.\n")
    L.append(f"Second search of the run: column-form `k_fill_rows` ({n_col} launches) read {f_col / 1e6:.1f} MB and "
             f"wrote {w_col / 1e6:.1f} MB, {(f_col + w_col) / n_col / 1e6:.3f} MB per launch; all kernels of the "
             f"search read {f_all / 1e6:.1f} MB and wrote {w_all / 1e6:.1f} MB "
             f"({(f_all + w_all) / (busy / ns / 1e9) / 1e9:.0f} GB/s over the time inside kernels, "
             f"against 8000 GB/s peak).\n")
    L.append("## VALU issue (rocprofv3 PMC)\n")
    L.append(f"    {commands['valu']}\n")
    L.append("VALU busy = SQ_ACTIVE_INST_VALU x 4 cycles / (1024 SIMDs x GRBM_GUI_ACTIVE per XCD); "
             "cells = SQ_INSTS_VALU_ADD_F64 x 64 lanes for the fill kernels (one fp64 add per cell).\n")
    L.append("| launch | grid threads | VALU busy | v_add_f64 | VALU instructions | VALU / add |")
    L.append("|---|---|---|---|---|---|")
    tot_add = tot_valu = tot_act = tot_gui = 0.0
    for r in vrows:
        if not is_column_fill(r["name"]):
            continue
        gui = r.get("GRBM_GUI_ACTIVE", 0.0) / 8
        act = r.get("SQ_ACTIVE_INST_VALU", 0.0)
        add = r.get("SQ_INSTS_VALU_ADD_F64", 0.0)
        valu = r.get("SQ_INSTS_VALU", 0.0)
        tot_add += add
        tot_valu += valu
        tot_act += act
        tot_gui += gui
        if add * 64 >= 1e9:
            L.append(f"| `{r['name'][5:]}` | {r['grid']} | {act * 4 / (1024 * gui):.2f} | {add:.3e} | {valu:.3e} | "
                     f"{valu / add:.2f} |")
    if tot_gui:
        L.append(f"| all column-form launches of one search | | {tot_act * 4 / (1024 * tot_gui):.2f} | {tot_add:.3e} | "
                 f"{tot_valu:.3e} | {tot_valu / tot_add:.2f} |")
    L.append("")
    rec = {"kernel": "k_fill_rows (column form, TZ > 1)", "workload": workload, "kernel_sources_sha256": src_hash,
           "bytes_per_launch": (f_col + w_col) / n_col, "fetch_bytes_per_search": f_col,
           "write_bytes_per_search": w_col, "launches_per_search": n_col,
           "copy_calibration": {"FETCH_SIZE": kf, "WRITE_SIZE": kw},
           "commands": [commands[k] for k in ("fetch", "write", "cfetch", "cwrite")]}
    return "\n".join(L) + "\n", rec


KERNEL_SOURCES = ("device.hip", "kernels.h", "internal.h", "launch_plan.cpp", "host.cpp")


def kernel_source_digest(root: str) -> str:
    """sha256 over the device code and the host code that plans its launches,
    in a fixed order: a counter record is valid for the kernels only while this
    digest matches."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(root, "paper_2407_04001_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def write_report(prof_dir: str, root: str, workload: str, cells: float, commands: dict):
    """Write profiles/k_fill_rows_<workload>.md and the traffic record from the
    six rocprofv3 output directories under prof_dir (kt, fetch, write,
    cfetch, cwrite, valu)."""
    digest = kernel_source_digest(root)
    sub = {k: os.path.join(prof_dir, k) for k in ("kt", "fetch", "write", "cfetch", "cwrite", "valu")}
    md, rec = report(sub["kt"], sub["fetch"], sub["write"], sub["cfetch"], sub["cwrite"], sub["valu"],
                     workload, cells, digest, commands)
    with open(os.path.join(root, "profiles", f"k_fill_rows_{workload}.md"), "w") as f:
        f.write(md)
    with open(os.path.join(root, "profiles", "k_fill_rows_hbm_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    return md, rec


def _main(argv):
    if len(argv) >= 2 and argv[0] == "stats":
        for r in kernel_stats(argv[1]):
            print(f"{r['name'][:60]:60s} {r['calls']:6d} {r['total_us']:12.1f} {r['avg_us']:10.2f} {r['pct']:6.2f}")
    elif len(argv) >= 2 and argv[0] == "counters":
        tot, n = counter_totals(argv[1], argv[2] if len(argv) > 2 else "")
        print(n, "dispatches")
        for k, v in sorted(tot.items()):
            print(f"{k:32s} {v:.6g}")
    elif len(argv) >= 2 and argv[0] == "report":
        # report <prof_dir> <workload> <cells> <commands.json>
        root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
        commands = json.load(open(argv[4]))
        md, _ = write_report(argv[1], root, argv[2], float(argv[3]), commands)
        print(md)
    else:
        print(__doc__)


if __name__ == "__main__":
    _main(sys.argv[1:])
