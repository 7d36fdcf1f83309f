"""Driver for the sanitizer run of the library's host builder (test
infrastructure; run by tests/test_host_sanitize.py in a process with the
AddressSanitizer runtime preloaded and SIMGPU_LIB naming the host-only
build).  Every workload goes through sim_create, sim_set_credit, a load
(which expands the workload on the host and stops at its first device call:
there is no device in this build), sim_txn_info, sim_route and sim_sizes,
with the engine choice left to the library and forced to each engine in
turn."""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import sim_inputs as si  # noqa: E402
from paper_2606_10440_amd import sim  # noqa: E402
from tests.test_gpu_fuzz import draw  # noqa: E402

ENGINES = [None, "workgroup", "workgroup_scan", "lane", "lanehbm", "b1", "wave", "grid", "resident"]
HOST_DONE = (sim.SIM_ERR_DEVICE, sim.SIM_ERR_OOM)


def exercise(w, txns=None, engine=None, pairs=64):
    if engine:
        os.environ["SIMGPU_ENGINE"] = engine
    else:
        os.environ.pop("SIMGPU_ENGINE", None)
    ctx = sim.sim_create(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.n_scenarios, w.bw, w.lat, w.cap,
                         w.arb)
    try:
        if w.credit is not None:
            sim.sim_set_credit(ctx, w.credit)
        try:
            if txns is not None:
                sim.sim_load_transactions(ctx, *txns)
            elif w.meta.get("memcpy") is not None and w.meta["memcpy"].kind is not None:
                mc = w.meta["memcpy"]
                sim.sim_load_gpu_ops(ctx, mc.kind, mc.cu, mc.src_ptr, mc.src_space, mc.src_line, mc.dst_space,
                                     mc.dst_line, mc.n_lines, mc.space_channels, mc.n_ch, mc.unroll, mc.window)
            elif w.meta.get("memcpy") is not None:
                mc = w.meta["memcpy"]
                sim.sim_load_memcpy(ctx, mc.cu, mc.src_space, mc.dst_space, mc.src_line, mc.dst_line,
                                    mc.n_lines, mc.space_channels, mc.n_ch, mc.unroll, mc.window)
            else:
                sim.sim_load_collective(ctx, w.coll, w.bytes, w.group_size, w.order, w.dep)
        except sim.SimError as e:
            # the host expansion ran; a forced engine may decline the workload
            assert e.status in HOST_DONE or (engine and "SIMGPU_ENGINE" in str(e)), (e, engine)
            if e.status not in HOST_DONE:
                return
        T = None
        rng = np.random.default_rng(0)
        for x in range(0, 1 << 31, 1):
            try:
                sim.sim_txn_info(ctx, x)
            except sim.SimError:
                T = x
                break
            if x > 2000:
                break
        E = w.n_endpoints
        for s, d in rng.integers(0, E, size=(pairs, 2)):
            try:
                sim.sim_route(ctx, int(s), int(d))
            except sim.SimError as e:
                assert e.status == sim.SIM_ERR_UNREACHABLE
        try:
            sim.sim_sizes(ctx)
        except sim.SimError as e:
            assert e.status == sim.SIM_ERR_STATE
        return T
    finally:
        sim.sim_destroy(ctx)


def main():
    n = 0
    for seed in range(150):
        w, txns, engine = draw(seed)
        exercise(w, txns, engine)
        n += 1
    for name in ["C1", "C2", "C3", "C5", "C5_rhd", "C5_dbt", "C5_chunk", "C5_credit"]:
        w = si.config(name)
        for engine in ENGINES:
            exercise(w, None, engine)
            n += 1
    exercise(si.config("C4"), None, None, pairs=512)
    exercise(si.config("C4"), None, "grid", pairs=64)
    n += 2
    from sim_inputs import noc
    w, lay = noc.gpu_noc(4, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    for get in (True, False):
        mc = noc.reducescatter_ops(lay, 4 * 8 * 4, n_wg=8, unroll=3, window=7, get=get)
        for engine in ENGINES:
            exercise(noc.memcpy_workload(w, mc), None, engine)
            n += 1
    print(f"host builder under sanitizers: {n} workloads ok", flush=True)


if __name__ == "__main__":
    main()
