"""Write the expected results of the five synthetic workloads from the CPU oracle.

Only ``oracle/`` (and the input generators in ``workloads/``) are called; no
value here comes from the HIP library.  For each workload instance the file
holds the GenerateSeq order, every dependent set, the minimum cost, the
strategy, the cell count, per-vertex fingerprints of the cost and argmin
tables (canonical order, SplitMix64-based, see ``pase.h``) and a seeded sample
of table entries.

    python tests/golden/make_golden.py [--only NAME] [--threads N] [--all-integers-only] [--bf-only] [--volume-only] [--grad-only] [--halo-only]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle.oracle import Oracle, build  # noqa: E402
from workloads import workload  # noqa: E402

# Instances: the workload and seed; p (None = the workload's own power-of-two
# p); `all_integers` enumerates Sec. II's full C(v); `bf` solves the
# breadth-first recurrence (2) instead of GenerateSeq + recurrence (4);
# `volume` prices transfers with the volume-intersection model; `grad` adds the
# weight-gradient all-reduce to the layer costs; `halo` the halo exchange of
# convolutions.
def _inst(name, seed=0, p=None, all_integers=False, bf=False, volume=False, grad=False, halo=False):
    return {"name": name, "seed": seed, "p": p, "all_integers": all_integers, "bf": bf, "volume": volume,
            "grad": grad, "halo": halo}


INSTANCES = [_inst("w0_fc_chain"), _inst("w1_residual_cnn"), _inst("w1_residual_cnn", 1),
             _inst("w1_residual_cnn", 2), _inst("w2_inception"), _inst("w2_inception", 1),
             _inst("w2_inception", 2), _inst("w3_lstm_grid"), _inst("w4_transformer"),
             _inst("w0_fc_chain", p=12, all_integers=True), _inst("w2_inception", p=12, all_integers=True),
             _inst("w4_transformer", p=12, all_integers=True),
             _inst("w1_residual_cnn", p=64, bf=True),
             _inst("w1_residual_cnn", volume=True), _inst("w2_inception", volume=True),
             _inst("w3_lstm_grid", volume=True), _inst("w4_transformer", volume=True),
             _inst("w1_residual_cnn", grad=True), _inst("w2_inception", grad=True),
             _inst("w3_lstm_grid", grad=True), _inst("w4_transformer", grad=True),
             _inst("w1_residual_cnn", halo=True), _inst("w2_inception", halo=True),
             _inst("w1_residual_cnn", grad=True, halo=True), _inst("w2_inception", grad=True, halo=True)]


def file_name(name: str, seed: int, p=None, all_integers: bool = False, bf: bool = False,
              volume: bool = False, grad: bool = False, halo: bool = False) -> str:
    if halo:
        return f"{name}_seed{seed}_{'grad_' if grad else ''}halo.json"
    if bf:
        return f"{name}_seed{seed}_p{p}_bf.json"
    if volume:
        return f"{name}_seed{seed}_volume.json"
    if grad:
        return f"{name}_seed{seed}_grad.json"
    return f"{name}_seed{seed}_p{p}_all.json" if all_integers else f"{name}_seed{seed}.json"


SAMPLES_PER_TABLE = 24


def golden(name: str, seed: int, threads: int, p=None, all_integers: bool = False, bf: bool = False,
           volume: bool = False, grad: bool = False, halo: bool = False) -> dict:
    g = workload(name, seed)
    p = p or g["p"]
    o = Oracle(g)
    K = o.configs(p, all_integers=all_integers, volume=volume, grad_sync=grad, halo=halo)
    t0 = time.time()
    if bf:
        o.solve_bf(threads=threads)
    else:
        o.solve(rule=0, threads=threads)
    wall = time.time() - t0
    seq = o.sequence()
    mc, strat = o.result()
    rng = np.random.default_rng(1234 + seed)
    tables = []
    for i in range(len(seq)):
        n = o.table_size(i)
        fpT, fpA = o.fingerprint(i)
        idx = sorted({0, n - 1} | set(int(x) for x in rng.integers(0, n, size=SAMPLES_PER_TABLE)))
        samples = []
        for k in idx:
            t, a = o.entry(i, k)
            samples.append([k, str(t), a])
        tables.append({"vertex": seq[i], "dep": o.dependent_set(i), "entries": n,
                       "fp_cost": str(fpT), "fp_arg": str(fpA), "samples": samples})
    return {"workload": name, "seed": seed, "p": p, "all_integers": all_integers,
            "order": "breadth-first" if bf else "GenerateSeq",
            "transfer": "volume intersection" if volume else "split match",
            "grad_sync": grad, "halo": halo,
            "num_configs": [int(k) for k in K],
            "sequence": seq, "min_cost": str(mc), "strategy": strat, "cells": o.cells(),
            "tables": tables, "oracle_seconds": round(wall, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", default=None)
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--all-integers-only", action="store_true",
                    help="only the instances with every integer split")
    ap.add_argument("--bf-only", action="store_true", help="only the breadth-first instances")
    ap.add_argument("--volume-only", action="store_true", help="only the volume-model instances")
    ap.add_argument("--grad-only", action="store_true", help="only the gradient-term instances")
    ap.add_argument("--halo-only", action="store_true", help="only the halo-term instances")
    args = ap.parse_args()
    build(force=False)
    for inst in INSTANCES:
        name, seed = inst["name"], inst["seed"]
        if args.only and args.only != name:
            continue
        if args.all_integers_only and not inst["all_integers"]:
            continue
        if args.bf_only and not inst["bf"]:
            continue
        if args.volume_only and not inst["volume"]:
            continue
        if args.grad_only and (not inst["grad"] or inst["halo"]):
            continue
        if args.halo_only and not inst["halo"]:
            continue
        t = time.time()
        out = golden(name, seed, args.threads, inst["p"], inst["all_integers"], inst["bf"], inst["volume"],
                     inst["grad"], inst["halo"])
        keys = ("seed", "p", "all_integers", "bf", "volume", "grad", "halo")
        path = os.path.join(HERE, file_name(name=name, **{k: inst[k] for k in keys}))
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        print(f"{name} seed {seed}: min_cost {out['min_cost']} cells {out['cells']:.3e} "
              f"({time.time() - t:.1f} s)", flush=True)


if __name__ == "__main__":
    main()
