"""Write the oracle's reference digests for the five full-size workloads.

Calls only the CPU oracle (``oracle/``) and the input generators
(``sim_inputs``); nothing here touches the GPU library.  Output:
``tests/golden/<config>.json`` with, per scenario, the status, makespan,
processed-cycle count and SHA-256 digests of the completion array (u32
little-endian), tx_lines and busy_cycles (u64 little-endian), plus for
single-scenario workloads a seeded sample of completion values.

Usage: python tests/golden/make_golden.py C1 C2 C3 C4 C5 [--jobs 8]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from multiprocessing import Pool

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import sim_inputs as si  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLE_SEED = 20261202
N_SAMPLE = 4096


def digest(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def _one(args):
    name, s = args
    w = si.config(name)
    r = oracle.simulate_workload(w, s)
    return (s, r.status, r.makespan, r.processed_cycles, r.line_hops, r.seconds,
            digest(r.completion.astype("<u4")), digest(r.tx_lines.astype("<u8")),
            digest(r.busy_cycles.astype("<u8")),
            r.completion if w.n_scenarios == 1 else None)


def make(name: str, jobs: int) -> dict:
    w = si.config(name)
    S = w.n_scenarios
    t0 = time.time()
    if S == 1:
        res = [_one((name, 0))]
    else:
        with Pool(jobs) as pool:
            res = pool.map(_one, [(name, s) for s in range(S)], chunksize=8)
    res.sort(key=lambda r: r[0])
    out = {
        "config": name, "workload": w.name, "n_scenarios": S,
        "n_links": w.n_links, "line_hops_per_scenario": res[0][4],
        "status": [r[1] for r in res], "makespan": [r[2] for r in res],
        "processed_cycles": [r[3] for r in res],
        "completion_sha256": [r[6] for r in res],
        "tx_lines_sha256": [r[7] for r in res],
        "busy_cycles_sha256": [r[8] for r in res],
        "oracle_seconds_total": sum(r[5] for r in res),
        "generated_by": "tests/golden/make_golden.py (CPU oracle only)",
    }
    if S == 1:
        comp = res[0][9]
        rng = np.random.default_rng(SAMPLE_SEED)
        idx = np.unique(np.concatenate([
            np.array([0, len(comp) - 1]), rng.integers(0, len(comp), size=N_SAMPLE)]))
        out["sample_idx"] = idx.tolist()
        out["sample_completion"] = comp[idx].astype(np.int64).tolist()
    print(f"{name}: S={S} makespan[0]={res[0][2]} wall={time.time() - t0:.1f}s", flush=True)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("configs", nargs="+")
    ap.add_argument("--jobs", type=int, default=8)
    a = ap.parse_args()
    oracle.build(force=False)
    for name in a.configs:
        out = make(name, a.jobs)
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(out, f, separators=(",", ":"))
            f.write("\n")


if __name__ == "__main__":
    main()
