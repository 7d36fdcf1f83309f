"""Benchmark: simulated line-hop events per second on one MI355X.

One step = one full simulation (``sim_run``) of the workload's whole batch:
every line of every scenario advanced hop by hop to completion, inputs and
state resident in HBM.  The default workload is the batched design sweep
(4096 scenarios of a 4x4 torus, ring all-reduce of 4 MiB per endpoint,
seeded bandwidth/latency/depth per scenario), the largest workload by
line-hop events; ``--workload C1..C4`` selects the others, a ``_chunk``
suffix (C1, C2, C5) the same workload with per-chunk step dependencies, and
C5_rhd / C5_dbt / C5_ag the batched sweep with another collective; NOC2_ag
is the GPU-as-NoC memcpy sweep.

Prints one JSON line with the metric, a roofline entry for the engine
kernel (algorithmic bytes per launch / measured launch time vs the 8 TB/s
HBM peak) and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
from paper_2606_10440_amd import build as _build  # noqa: E402  (compile flags, for the profile digests)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, 8 TB/s
COMPLETION_BYTES = 4            # u32 completion cycle written per line
HOP_BYTES_HBM = 20              # HBM-resident queue state: per line-hop, 8 B FIFO entry read,
                                # 8 B written into the next FIFO, 4 B path lookup
TXN_BYTES_HBM = 12              # and per line: stream/predecessor read, completion write, release read
KERNEL_NAME = "engine_"         # substring of the engine kernels' symbols
# workloads whose engines keep the queue state in device memory (L2/HBM) rather
# than in LDS and registers: their roofline counts the HBM-resident bytes
HBM_STATE = ("C3", "C4", "C4_credit", "NOC2_ag")

DESCR = {
    "C1": "4-endpoint full mesh, direct all-reduce 64 KiB, b=1 L=10 cap=16, lowest-id",
    "C2": "8-endpoint full mesh, ring all-reduce 16 MiB, b=1 L=50 cap=64, lowest-id",
    "C3": "8 full-mesh domains of 8 + 8-leaf/4-spine fabric, hierarchical all-reduce 64 MiB, round-robin",
    "C4": "k=16 fat-tree (1024 hosts, 320 switches), all-to-all 64 KiB per pair, L in [100,300], cap 32",
    "C5": "4096 scenarios x 4x4 torus, ring all-reduce 4 MiB, seeded b in {1,2,4}, L in [20,200], depth in {16,32,64}",
}
for _k in ("C1", "C2", "C5"):
    DESCR[_k + "_chunk"] = DESCR[_k] + "; per-chunk (put + signal) step dependencies"
for _k, _c in (("rhd", "recursive halving-doubling all-reduce"), ("dbt", "double binary tree all-reduce"),
               ("ag", "ring all-gather")):
    DESCR["C5_" + _k] = DESCR["C5"].replace("ring all-reduce", _c)
DESCR["C5_credit"] = DESCR["C5"] + "; credit delay = link latency"
DESCR["C4_credit"] = DESCR["C4"] + "; credit delay = link latency"
DESCR["NOC2_ag"] = ("1024 scenarios x 2 generic GPUs as NoCs (448 nodes each) + 32 scale-up switches, "
                    "put-based all-gather 2 MiB out per GPU as memcpy programs (32 WGs/GPU, unroll 4, "
                    "64 outstanding), channel latency in {1,2,4,8}, scale-up cable latency in {40,67,134}")


def algorithmic_bytes(T: int, S: int, m: int) -> int:
    """Bytes the method must move per launch when the scenario state stays on
    chip (LDS and registers): one u32 completion per line plus the per-link
    u64 counters and per-scenario makespan."""
    return S * (T * COMPLETION_BYTES + m * 16 + 4)


def algorithmic_bytes_hbm_state(T: int, S: int, m: int, line_hops: int) -> int:
    """Bytes per launch when the queue state lives in device memory: 20 B per
    line-hop (FIFO entry read and written on, path lookup) and 12 B per line
    (stream or predecessor read, completion write, release read), plus the
    per-link counters and makespans."""
    return S * (line_hops * HOP_BYTES_HBM + T * TXN_BYTES_HBM + m * 16 + 4)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def load_latency_profile(workload: str):
    """Per-simulated-cycle SQ counters of the critical wave from the committed
    profile summary, if one exists for the current engine source."""
    path = os.path.join(ROOT, "profiles", f"engine_{workload}_sq_per_cycle.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("engine_source_hash") != engine_source_hash(c.get("kernel", KERNEL_NAME)):
        return None
    return c.get("per_simulated_cycle")


def engine_source_hash(kernel: str = "") -> str:
    """Digest of the device sources a kernel is built from: its engine's
    .hip file (named after the kernel symbol, e.g. engine_wave) and the
    headers it includes, transitively, with the flags each is compiled
    with.  With no kernel name, every engine
    source.  Counters taken on other sources are not reported."""
    csrc = os.path.join(ROOT, "paper_2606_10440_amd", "csrc")
    m = re.search(r"(engine_[a-z0-9]+)", kernel or "")
    names = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    if m and m.group(1) + ".hip" in names:
        todo, names = [m.group(1) + ".hip"], set()
        while todo:
            f = todo.pop()
            if f in names or not os.path.exists(os.path.join(csrc, f)):
                continue
            names.add(f)
            with open(os.path.join(csrc, f)) as fh:
                todo += re.findall(r'^#include "([^"]+)"', fh.read(), re.M)
        names = sorted(names)
    h = hashlib.sha256()
    for f in names:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
        # the flags it is compiled with
        h.update(" ".join(_build.FLAGS[:4] + _build.EXTRA.get(f, [])).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, launch_s: float):
    """HBM traffic per launch and kernel symbol from the committed rocprofv3
    counter summary; the traffic only if it was taken on the current engine
    source."""
    path = os.path.join(ROOT, "profiles", f"engine_{workload}_hbm_counters.json")
    if not os.path.exists(path):
        return None, KERNEL_NAME
    with open(path) as f:
        c = json.load(f)
    kernel = c.get("kernel", KERNEL_NAME)
    if c.get("engine_source_hash") != engine_source_hash(kernel):
        return None, kernel
    return c.get("traffic_bytes_per_launch"), kernel


def cpu_baseline(w, sample_seconds: float):
    """Time the CPU oracle (single thread) on a bounded sample of the same
    workload: whole scenarios until about sample_seconds of event-loop time
    has accumulated or, for a workload of one scenario, a prefix of its
    simulated cycles (the oracle stops at a cycle guard; the line-hops done
    are its link admissions so far), sized from a first short prefix."""
    import oracle
    oracle.build(force=False)
    if w.n_scenarios == 1:
        mc, r = 20000, None
        for _ in range(2):
            r = oracle.simulate_workload(w, 0, max_cycles=mc)
            if r.status != 8 or r.seconds >= sample_seconds / 2:  # 8: stopped at the cycle guard
                break
            mc = int(mc * sample_seconds / max(r.seconds, 1e-3))
        hops = int(r.tx_lines.sum())
        what = "the whole scenario" if r.status == 0 else f"its first {r.processed_cycles} processed cycles"
        return {"value": hops / r.seconds, "unit": "line-hop events/s", "cores": 1, "kind": "oracle",
                "cpu_model": cpu_model(),
                "sample": f"1 of 1 scenario, {what}, event loop only ({hops} line-hops in {r.seconds:.1f} s)"}
    total_hops = 0
    total_s = 0.0
    n = 0
    for s in range(w.n_scenarios):
        r = oracle.simulate_workload(w, s)
        total_hops += r.line_hops
        total_s += r.seconds
        n += 1
        if total_s >= sample_seconds:
            break
    return {"value": total_hops / total_s, "unit": "line-hop events/s", "cores": 1, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{n} of {w.n_scenarios} scenario(s), full size, event loop only "
                      f"({total_hops} line-hops in {total_s:.1f} s)"}


def _oracle_worker(args):
    """One host process of the all-core baseline: whole scenarios wid,
    wid + n, ... until budget seconds of event-loop time."""
    name, wid, n, budget = args
    import oracle
    import sim_inputs as si
    w = si.config(name)
    hops, secs, k = 0, 0.0, 0
    for sc in range(wid, w.n_scenarios, n):
        r = oracle.simulate_workload(w, sc)
        hops += r.line_hops
        secs += r.seconds
        k += 1
        if secs >= budget:
            break
    return hops, secs, k


def cpu_baseline_all_cores(name: str, n_scenarios: int, budget: float):
    """The same oracle, one process per host core (at most 16, the GPU
    box's share), each on its own whole scenarios of a batched workload:
    the sum of the processes' rates."""
    import multiprocessing as mp
    import oracle
    oracle.build(force=False)
    n = max(1, min(16, len(os.sched_getaffinity(0)), n_scenarios))
    with mp.get_context("spawn").Pool(n) as pool:
        res = pool.map(_oracle_worker, [(name, i, n, budget) for i in range(n)])
    rate = sum(h / sec for h, sec, _ in res if sec > 0)
    return {"value": rate, "unit": "line-hop events/s", "cores": n, "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{sum(k for _, _, k in res)} of {n_scenarios} scenarios, full size, "
                      f"{n} processes, about {budget:.0f} s of event loop each"}


def copy_calibration():
    """A plain device copy of known size, for scaling the HBM counters."""
    import torch
    n = 1 << 28  # 1 GiB of int32
    a = torch.ones(n, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))


def sweep_allgather(points, n_wg=32, seconds_cap=120.0):
    """The scalability measurement of the paper's Sec. 5.4: a put-based
    all-gather with n_wg workgroups per GPU on G generic GPUs, for several
    output buffer sizes per GPU.  Per point one JSON line: host setup time
    (expansion and tables, not simulated time), the launch's wall time
    (device events around sim_run), the makespan in cycles and in simulated
    nanoseconds (one cycle = one line on one memory channel), and simulated
    nanoseconds per wall-clock second.  A GPU count's larger sizes are
    skipped once a launch took longer than seconds_cap."""
    import torch
    from sim_inputs import noc
    from paper_2606_10440_amd import sim
    stop = set()
    for G, mib in points:
        if G in stop:
            continue
        chunk = int(mib * 2 ** 20 / 128) // G
        chunk = max(n_wg, chunk // n_wg * n_wg)
        t0 = time.time()
        w, lay = noc.gpu_noc(G)
        wm = noc.memcpy_workload(w, noc.allgather_ops(lay, chunk * G, n_wg=n_wg), name=f"ag_{G}gpu")
        s = sim.Simulator.from_workload(wm)
        T, m, S, line_hops = s.sizes()
        outs = s.alloc_outputs()
        torch.cuda.synchronize()
        setup = time.time() - t0
        stream = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        s.enqueue(outs, stream=stream)
        e1.record(stream)
        stream.synchronize()
        run_s = e0.elapsed_time(e1) / 1e3
        rc, st, cyc = sim.sim_status_after_sync(s.ctx, S)
        mk = int(outs[3][0])
        sim_ns = mk * noc.CYCLE_NS
        print(json.dumps({"sweep": "allgather", "gpus": G, "endpoints": G * 448, "out_mib_per_gpu": chunk * G * 128 / 2 ** 20,
                          "workgroups_per_gpu": n_wg, "lines": T, "line_hops": line_hops, "status": sim.STATUS_NAMES[rc],
                          "setup_s": round(setup, 3), "run_s": run_s, "processed_cycles": int(cyc[0]),
                          "makespan_cycles": mk, "simulated_ns": sim_ns,
                          "simulated_ns_per_wall_s": sim_ns / run_s if run_s > 0 else None,
                          "line_hops_per_s": line_hops / run_s if run_s > 0 else None}), flush=True)
        s.close()
        del outs
        torch.cuda.empty_cache()
        if run_s > seconds_cap:
            stop.add(G)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="C5", choices=sorted(DESCR))
    ap.add_argument("--cpu-sample-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-verify", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--only-scenario", type=int, default=None,
                    help="run one scenario of a batched workload alone (per-cycle counters of a lone wave)")
    ap.add_argument("--sweep-allgather", default=None,
                    help="instead of the benchmark line: the Sec. 5.4 all-gather sweep, points 'G:MiB,G:MiB,...'")
    a = ap.parse_args()

    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(f"bench.py: simgpu runs on exactly one GPU (asked for {a.gpus}); "
              "batched scenarios would shard across GPUs with no exchange, but no "
              "multi-GPU path is built", file=sys.stderr)
        sys.exit(2)
    if a.calibrate_copy:
        copy_calibration()
        return
    if a.sweep_allgather:
        pts = [(int(g), float(mb)) for g, mb in (p.split(":") for p in a.sweep_allgather.split(","))]
        sweep_allgather(pts)
        return

    import torch
    import sim_inputs as si
    from paper_2606_10440_amd import sim

    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    w = si.config(a.workload)
    if a.only_scenario is not None:
        w = si.take_scenarios(w, [a.only_scenario])
    t0 = time.time()
    s = sim.Simulator.from_workload(w)
    T, m, S, line_hops = s.sizes()
    outs = s.alloc_outputs()
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    print(f"[bench] {a.workload}: T={T} S={S} m={m} line_hops/scenario={line_hops} setup {setup_s:.1f}s",
          file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    warm_s = 0.0
    for i in range(a.warmup):
        t1 = time.time()
        s.enqueue(outs, stream=stream)
        stream.synchronize()
        warm_s = time.time() - t1
        print(f"[bench] warmup {i} done ({warm_s:.1f} s)", file=sys.stderr, flush=True)
    # a workload whose launch runs for many seconds reports each timed step
    # as it ends (one host wait per step, inside the event-timed region)
    per_step = warm_s > 20.0
    if a.warmup > 0:
        rc, st, cyc = sim.sim_status_after_sync(s.ctx, S)
        if rc != 0:
            raise SystemExit(f"simulation failed: {sim.STATUS_NAMES[rc]} {sim.sim_last_error(s.ctx)}")

    # one event between launches on the launches' own stream: the K steps back
    # to back, and each launch's duration (median reported)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(a.steps):
        s.enqueue(outs, stream=stream)
        evs[i + 1].record(stream)
        if per_step:
            stream.synchronize()
            print(f"[bench] step {i} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    gpu_ms = evs[0].elapsed_time(evs[-1])
    launch_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(a.steps)]
    launch_med_ms = float(np.median(launch_ms))
    rc, st, cyc = sim.sim_status_after_sync(s.ctx, S)
    if rc != 0:
        raise SystemExit(f"simulation failed: {sim.STATUS_NAMES[rc]}")
    print(f"[bench] timed {a.steps} steps: {gpu_ms:.1f} ms (wall {wall * 1e3:.1f} ms)", file=sys.stderr, flush=True)

    verified = None
    if not a.no_verify and a.only_scenario is None:
        gpath = os.path.join(ROOT, "tests", "golden", f"{a.workload}.json")
        if os.path.exists(gpath):
            with open(gpath) as f:
                g = json.load(f)
            mk = outs[3].cpu().numpy()
            ok = np.array_equal(mk, np.array(g["makespan"]))
            for sc in sorted({0, S // 2, S - 1}):
                comp = outs[0][sc, :T].cpu().numpy().view(np.uint32).astype("<u4")
                ok = ok and hashlib.sha256(comp.tobytes()).hexdigest() == g["completion_sha256"][sc]
            verified = bool(ok)

    ms_per_step = gpu_ms / a.steps
    launch_s = launch_med_ms / 1e3
    total_hops = line_hops * S
    value = total_hops * a.steps / (gpu_ms / 1e3)
    alg_onchip = algorithmic_bytes(T, S, m)
    alg_hbm = algorithmic_bytes_hbm_state(T, S, m, line_hops)
    hbm_state = a.workload in HBM_STATE
    alg = alg_hbm if hbm_state else alg_onchip
    traffic, kernel = load_traffic(a.workload, launch_s)
    achieved = alg / launch_s / 1e9
    out = {
        "metric": "simulated line-hop events/sec on 1 MI355X (bit-exact vs CPU oracle)",
        "value": value,
        "unit": "line-hop events/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": f"{a.workload}: {DESCR[a.workload]}", "scenarios": S, "transactions": T * S,
                   "line_hops": total_hops, "links": m,
                   "processed_cycles_max": int(cyc.max()), "processed_cycles_sum": int(cyc.sum()),
                   "critical_scenario": int(np.argmax(cyc)),
                   "bit_exact_vs_golden": verified},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_frac": None if traffic is None else traffic / launch_s / 1e9 / HBM_PEAK_GBS,
                     "kernel": kernel, "launch_ms_median": launch_med_ms,
                     "launch_ms": [round(v, 3) for v in launch_ms],
                     "accounting": ("hbm-resident queue state: 20 B per line-hop + 12 B per line" if hbm_state
                                    else "on-chip scenario state: 4 B per line"),
                     "algorithmic_bytes_per_launch": alg,
                     "frac_onchip_accounting": alg_onchip / launch_s / 1e9 / HBM_PEAK_GBS,
                     "frac_hbm_state_accounting": alg_hbm / launch_s / 1e9 / HBM_PEAK_GBS},
        # a batch is bound by its critical scenario's chain of dependent cycles
        "latency": {"critical_processed_cycles": int(cyc.max()),
                    "ns_per_processed_cycle": launch_s * 1e9 / max(int(cyc.max()), 1),
                    "sq_per_simulated_cycle": load_latency_profile(a.workload)},
    }
    s.close()
    if not a.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_sample_seconds)
        if S > 1:
            out["cpu_baseline_all_cores"] = cpu_baseline_all_cores(a.workload, S, a.cpu_sample_seconds / 2)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
