"""Write the expected results of the five synthetic workloads from the CPU oracle.

Only ``oracle/`` (and the input generators in ``workloads/``) are called; no
value here comes from the HIP library.  For each workload instance the file
holds the GenerateSeq order, every dependent set, the minimum cost, the
strategy, the cell count, per-vertex fingerprints of the cost and argmin
tables (canonical order, SplitMix64-based, see ``pase.h``) and a seeded sample
of table entries.

    python tests/golden/make_golden.py [--only NAME] [--threads N]
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

INSTANCES = [("w0_fc_chain", 0), ("w1_residual_cnn", 0), ("w1_residual_cnn", 1),
             ("w1_residual_cnn", 2), ("w2_inception", 0), ("w2_inception", 1),
             ("w2_inception", 2), ("w3_lstm_grid", 0), ("w4_transformer", 0)]
SAMPLES_PER_TABLE = 24


def golden(name: str, seed: int, threads: int) -> dict:
    g = workload(name, seed)
    o = Oracle(g)
    K = o.configs(g["p"])
    t0 = time.time()
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
    return {"workload": name, "seed": seed, "p": g["p"], "num_configs": [int(k) for k in K],
            "sequence": seq, "min_cost": str(mc), "strategy": strat, "cells": o.cells(),
            "tables": tables, "oracle_seconds": round(wall, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", default=None)
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    build(force=False)
    for name, seed in INSTANCES:
        if args.only and args.only != name:
            continue
        t = time.time()
        out = golden(name, seed, args.threads)
        path = os.path.join(HERE, f"{name}_seed{seed}.json")
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        print(f"{name} seed {seed}: min_cost {out['min_cost']} cells {out['cells']:.3e} "
              f"({time.time() - t:.1f} s)", flush=True)


if __name__ == "__main__":
    main()
