"""Benchmark of the PaSE strategy search on one MI355X.

One step = the whole search for one graph: pase_enumerate_configs(p) (config
enumeration, GenerateSeq, plans) + pase_find_best_strategy (cost tables,
per-vertex DP fill, back-substitution).  Default workload: the Transformer
encoder-decoder graph at p = 64 modeled devices (6.99e10 DP cell updates).

Prints one JSON line: DP cell-updates/s of whole steps (`value`), the step
wall time, the roofline of the dominant kernel (the row/column-chunk fill,
fp64 add + min per cell, timed with HIP events on the search stream), the
parity of the result with the CPU oracle's stored answer, and the oracle's
own time for the same search on the host cores (and single-threaded on a
prefix of the vertex sequence).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DP cell-updates/sec and FindBestStrategy wall time (Transformer, p=64)"
# VALU: 256 CUs x 64 lanes x 2.4 GHz lane-ops/s (one fp64 add or min, or one
# int32 op, per lane-cycle)
FP64_OPS_PEAK_T = 256 * 64 * 2.4e9 / 1e12
OPS_PER_CELL = 2          # fp64 keys: one add and one min (the min-plus multiply-accumulate)
OPS_PER_CELL_U64 = 5      # uint64 keys: add + carry, 64-bit compare, two selects (int32 lane-ops)


def cpu_threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp and omp.isdigit():
        n = min(n, int(omp))
    return max(1, n)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_baseline(g, p, max_cells, single_cells, all_integers=False, bf=False, volume=False, grad=False,
                    halo=False):
    """The oracle on the host cores (OpenMP over table entries): the whole
    search when it has at most `max_cells` cells (else the prefix of the vertex
    order that reaches that many), and single-threaded on the longest prefix
    of the vertex order with at most `single_cells` cells (at least one
    vertex)."""
    from oracle.oracle import Oracle
    threads = cpu_threads()
    o = Oracle(g)
    o.configs(p, all_integers=all_integers, volume=volume, grad_sync=grad, halo=halo)

    def run(cells, nthreads):
        if bf:
            o.solve_bf(max_cells=cells, threads=nthreads)
        else:
            o.solve(max_cells=cells, threads=nthreads)
        return o.cells_done() / o.seconds(), o.cells_done(), o.seconds()

    # the sequence and table sizes (the first vertex only), then the prefix
    run(1, 1)
    cum, budget = 0, 0
    for i, v in enumerate(o.sequence()):
        cum += o.table_size(i) * int(o.K[v])
        if i > 0 and cum > single_cells:
            break
        budget = cum
    one, one_cells, one_s = run(max(1, budget), 1)
    total = o.cells()
    run(0 if total <= max_cells else int(max_cells), threads)
    done = o.cells_done()
    n_done = 0
    cum = 0
    seq = o.sequence()
    for i in range(len(seq)):
        cum += o.table_size(i) * int(o.K[seq[i]])
        n_done += 1
        if cum >= done:
            break
    order = "breadth-first" if bf else "GenerateSeq"
    whole = done == total
    sample = (f"the whole search: all {len(seq)} vertices of the {order} order" if whole else
              f"first {n_done} of {len(seq)} vertices of the same {order} order")
    return {"value": done / o.seconds(), "unit": "cell-updates/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample} ({done:.3e} of {total:.3e} cells, {o.seconds():.1f} s, "
                      f"OpenMP over table entries)",
            "whole_search": whole, "seconds": round(o.seconds(), 2),
            "single_thread": {"value": one, "cells": one_cells, "seconds": round(one_s, 2),
                              "sample": f"the longest prefix of the {order} order with at most "
                                        f"{single_cells:.1e} cells"},
            "cpu_model": cpu_model()}


def copy_calibration(mib):
    """A plain device-to-device copy of known size: under rocprofv3 --pmc its
    FETCH_SIZE / WRITE_SIZE readings give the scale of those counters."""
    import torch
    n = mib * 1024 * 1024
    a = torch.ones(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "copies": 3}), flush=True)


def traffic_from_profile():
    """HBM bytes per launch of the row kernel from the committed counter
    summary, if it was taken on the current kernel sources; else None."""
    from paper_2407_04001_amd.profiling import kernel_source_digest
    path = os.path.join(ROOT, "profiles", "k_fill_rows_hbm_traffic.json")
    try:
        with open(path) as f:
            prof = json.load(f)
        digest = kernel_source_digest(ROOT)
    except OSError:
        return None
    if prof.get("kernel_sources_sha256") != digest:
        return None
    return prof.get("bytes_per_launch")


SCHEDULES = {0: "level", 1: "sequential", 4: "bulk lane", 5: "split chains"}
WORKLOADS = ["w0_fc_chain", "w1_residual_cnn", "w2_inception", "w3_lstm_grid", "w4_transformer"]


def run_workload(name, seed, steps, warmup, cpu_cells, cpu_single_cells, no_cpu, p=None, all_integers=False,
                 bf=False, volume=False, grad=False, schedule=None, no_roofline=False, halo=False, fused_min=None,
                 hoist_elems=None, bulk_us=None):
    """Time `steps` whole searches of one workload (at its own power-of-two p,
    or at `p` with every integer split when `all_integers`; over the
    breadth-first order, i.e. recurrence (2), when `bf`; with volume-intersection
    transfer costs when `volume`; with the weight-gradient term when `grad`);
    returns the report
    dict (the oracle timed on the same graph: the whole search when it has at
    most `cpu_cells` cells, else a prefix of the vertex order; single-threaded
    on a prefix of about `cpu_single_cells` cells).  A search the
    library refuses as too large gives a line with value null and the reason."""
    import torch
    from paper_2407_04001_amd import (OPT_BULK_US, OPT_FUSED_MIN, OPT_GRAD_SYNC, OPT_HALO, OPT_HOIST_ELEMS, OPT_ORDER,
                                      OPT_PROFILE, OPT_SCHEDULE, OPT_TRANSFER, Graph, PaseError)
    from workloads import workload

    g = workload(name, seed)
    p = p or g["p"]
    pg = Graph(g)
    pg.set_option(OPT_ORDER, int(bf))
    pg.set_option(OPT_TRANSFER, int(volume))
    pg.set_option(OPT_GRAD_SYNC, int(grad))
    pg.set_option(OPT_HALO, int(halo))
    if schedule is not None:
        pg.set_option(OPT_SCHEDULE, schedule)
    if fused_min is not None:
        pg.set_option(OPT_FUSED_MIN, fused_min)
    if hoist_elems is not None:
        pg.set_option(OPT_HOIST_ELEMS, hoist_elems)
    if bulk_us is not None:
        pg.set_option(OPT_BULK_US, bulk_us)
    wl = g["name"] if p == g["p"] else f"{g['name']} at p={p}"
    if all_integers:
        wl += ", every integer split"
    if bf:
        wl += ", breadth-first order (eq. 2)"
    if volume:
        wl += ", volume-intersection transfer costs"
    if grad:
        wl += ", weight-gradient all-reduce"
    if halo:
        wl += ", halo exchange"
    headline = (name == "w4_transformer" and p == g["p"] and not all_integers and not bf and not volume
                and not grad and not halo)
    metric = METRIC if headline else f"DP cell-updates/sec and FindBestStrategy wall time ({wl})"
    config = {"workload": g["name"], "p": p,
              "config_set": "every integer split" if all_integers else "powers of two",
              "order": "breadth-first" if bf else "GenerateSeq",
              "transfer": "volume intersection" if volume else "split match",
              "grad_sync": grad, "halo": halo,
              "vertices": len(g["vertices"]), "edges": len(g["edges"]), "seed": seed}
    try:
        pg.enumerate_configs(p, all_integers=all_integers)
    except PaseError as e:
        return {"metric": metric, "value": None, "unit": "cell-updates/s", "n_gpus": 1, "steps": 0,
                "warmup": 0, "higher_is_better": True, "data": "synthetic", "config": config,
                "refused": str(e)}
    stream = torch.cuda.current_stream()

    def step():
        pg.enumerate_configs(p)
        return pg.find_best_strategy(stream)

    # timed steps: no timing events at all (each event attached to a launch or
    # recorded between launches costs the stream ~4.4 us of serialization)
    pg.set_option(OPT_PROFILE, 0)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    walls, step_ms = [], []
    phase_keys = ("seq_ms", "plan_ms", "setup_ms")
    phases = dict.fromkeys(phase_keys, 0.0)
    t0 = time.perf_counter()
    for _ in range(steps):
        ts = time.perf_counter()
        mc, strat = step()
        step_ms.append((time.perf_counter() - ts) * 1e3)
        st = pg.stats()
        walls.append(st["wall_ms"])
        for k in phase_keys:
            phases[k] += st[k] / steps
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # profiled steps, right after the timed ones: the same searches with HIP
    # events (on the search stream) attached to every launch of the dominant
    # kernel -- the row kernel with a column chunk per lane -- and recorded at
    # the phase boundaries; they give the roofline and the device phases
    rows_ms, rows_launches, prof_ms = 0.0, 0, []
    if no_roofline:
        prof_steps = 0
    else:
        prof_steps = steps
        pg.set_option(OPT_PROFILE, 2)
        step()
        torch.cuda.synchronize()
    dev_keys = ("cost_tables_ms", "fill_span_ms", "backtrack_ms")
    dev_phases = dict.fromkeys(dev_keys, 0.0)
    for _ in range(prof_steps):
        ts = time.perf_counter()
        pmc, pstrat = step()
        prof_ms.append((time.perf_counter() - ts) * 1e3)
        assert (pmc, pstrat) == (mc, strat)
        pst = pg.stats()
        rows_ms += pst["rows_fill_ms"]
        rows_launches += pst["rows_launches"]
        for k in dev_keys:
            dev_phases[k] += pst[k] / prof_steps
    torch.cuda.synchronize()
    phases.update(dev_phases)

    cells = st["cells"]
    col_cells = st["rows_cells"] - st["stream_cells"]
    ops = OPS_PER_CELL if st["key_type"] == 0 else OPS_PER_CELL_U64
    achieved = ops * col_cells * prof_steps / (rows_ms / 1e3) / 1e12 if rows_ms else 0.0
    t_roof_ms = ops * cells / (FP64_OPS_PEAK_T * 1e12) * 1e3
    parity = None
    # the oracle's stored answer for exactly this variant, if one was written
    gold_name = None
    if halo and not (bf or volume or all_integers):
        gold_name = f"{name}_seed{seed}_{'grad_' if grad else ''}halo.json"
    elif sum((bf, volume, grad, all_integers)) <= 1:
        if bf:
            gold_name = f"{name}_seed{seed}_p{p}_bf.json"
        elif volume:
            gold_name = f"{name}_seed{seed}_volume.json"
        elif grad:
            gold_name = f"{name}_seed{seed}_grad.json"
        elif all_integers:
            gold_name = f"{name}_seed{seed}_p{p}_all.json"
        else:
            gold_name = f"{name}_seed{seed}.json"
    gold_path = os.path.join(ROOT, "tests", "golden", gold_name) if gold_name else None
    if gold_path and os.path.exists(gold_path):
        with open(gold_path) as f:
            gold = json.load(f)
        if gold.get("p", g["p"]) == p:
            parity = (mc == int(gold["min_cost"]) and strat == gold["strategy"])
    out = {
        "metric": metric, "value": cells * steps / elapsed, "unit": "cell-updates/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup,
        "ms_per_step": elapsed * 1e3 / steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if st["key_type"] == 0 else "u64", "data": "synthetic",
        "config": dict(config, cells=cells, schedule=SCHEDULES.get(st["schedule"], st["schedule"])),
        "find_best_strategy_ms": sum(walls) / len(walls),
        # mean per step: host GenerateSeq / plans (enumerate) and launch setup
        # of the timed steps; device phases of the profiled steps (events on
        # the search stream)
        "phases_ms": {k[:-3]: round(v, 4) for k, v in phases.items()},
        "profiled_ms_per_step": sorted(prof_ms)[len(prof_ms) // 2] if prof_ms else None,
        "median_ms_per_step": sorted(step_ms)[len(step_ms) // 2],
        # the whole search against the ALU roofline: every cell costs `ops` VALU
        # lane-ops (t_roof), against the fill-kernel time and the step
        "search_roofline": {"t_roof_ms": t_roof_ms, "ops_per_cell": ops,
                            "frac_of_step": t_roof_ms / (elapsed * 1e3 / steps)},
        "min_cost": mc, "parity_with_oracle": parity,
        "roofline": {"bound": "alu", "kernel": "k_fill_rows",
                     "achieved": achieved, "peak": FP64_OPS_PEAK_T,
                     "unit": "T fp64-op/s" if st["key_type"] == 0 else "T int32-op/s",
                     "frac": achieved / FP64_OPS_PEAK_T,
                     "traffic": traffic_from_profile() if headline else None,
                     "launches_per_step": rows_launches // steps,
                     "avg_launch_us": rows_ms * 1e3 / max(rows_launches, 1),
                     "cells_per_step": col_cells,
                     "timed_in": f"{steps} profiled steps after the timed ones (HIP events on the search "
                                 "stream around every launch of the kernel)"},
    }
    if not no_cpu:
        out["cpu_baseline"] = oracle_baseline(g, p, int(cpu_cells), int(cpu_single_cells), all_integers, bf,
                                              volume, grad, halo)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="w4_transformer")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-cells", type=float, default=1e11,
                    help="oracle on all host cores: the whole search up to this many cells, else a prefix")
    ap.add_argument("--cpu-single-cells", type=float, default=3e9,
                    help="single-threaded oracle sample (cells, a prefix of the vertex order)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (HBM counter calibration)")
    ap.add_argument("--all-workloads", action="store_true",
                    help="one JSON line per synthetic workload (W0..W4) instead of the W4 line")
    ap.add_argument("--p", type=int, default=0, help="modeled devices (default: the workload's own)")
    ap.add_argument("--all-integers", action="store_true",
                    help="every integer split factor (Sec. II's full C(v)) instead of powers of two")
    ap.add_argument("--order", choices=("genseq", "bf"), default="genseq",
                    help="vertex order: GenerateSeq (default) or breadth-first (recurrence 2)")
    ap.add_argument("--transfer", choices=("match", "volume"), default="match",
                    help="transfer cost model: split match (default) or volume intersection")
    ap.add_argument("--grad-sync", action="store_true",
                    help="add the weight-gradient all-reduce to the layer costs")
    ap.add_argument("--halo", action="store_true", help="add the halo exchange of convolutions to the layer costs")
    ap.add_argument("--no-roofline", action="store_true",
                    help="skip the profiled steps (no HIP events at all; for traces of the timed steps)")
    ap.add_argument("--schedule", type=int, default=None, choices=(0, 1, 4, 5),
                    help="launch schedule (PASE_OPT_SCHEDULE; default: the library's)")
    ap.add_argument("--fused-min", type=int, default=None, choices=(0, 1),
                    help="fused minima (PASE_OPT_FUSED_MIN; default: the library's, on)")
    ap.add_argument("--bulk-us", type=int, default=None,
                    help="bulk lane threshold in planned microseconds (PASE_OPT_BULK_US; default: the library's)")
    ap.add_argument("--hoist-elems", type=int, default=None,
                    help="prep hoisting threshold (PASE_OPT_HOIST_ELEMS; 0 = off; default: the library's)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the strategy search runs on a single device "
              "(see the sharding notes in DESIGN.md); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    names = WORKLOADS if args.all_workloads else [args.workload]
    for name in names:
        out = run_workload(name, args.seed, args.steps, args.warmup, args.cpu_cells, args.cpu_single_cells,
                           args.no_cpu,
                           args.p or None, args.all_integers, args.order == "bf",
                           args.transfer == "volume", args.grad_sync, args.schedule, args.no_roofline, args.halo,
                           args.fused_min, args.hoist_elems, args.bulk_us)
        print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
