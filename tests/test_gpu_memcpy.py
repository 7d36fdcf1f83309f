"""GPU parity of memcpy programs on the generic GPU NoC (the injection side
of the GPU model) against the CPU oracle, line for line, through the C ABI.
"""
from __future__ import annotations

import numpy as np
import pytest

from sim_inputs import noc
from tests.test_gpu_parity import (ENGINES, check_engine, check_vs_oracle, simmod, torch_cuda,  # noqa: F401
                                   say)

pytestmark = pytest.mark.gpu


def tiny_noc(seed, n_ops=6, max_lines=9):
    w, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1,
                         noc=(4, 1, 8), cu_out=(2, 1, 4), mem=(1, 2, 3))
    rng = np.random.default_rng(seed)
    rows = [(int(rng.choice(lay.cus[0])), 0, 0, int(rng.integers(0, 20)), 40 + int(rng.integers(0, 20)),
             int(rng.integers(0, max_lines))) for _ in range(n_ops)]
    mc = noc._ops(rows, lay, int(rng.integers(1, 5)), int(rng.integers(1, 9)))
    wm = noc.memcpy_workload(w, mc, name=f"tiny_noc_{seed}")
    wm.arb = seed % 2
    return wm


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("seed", range(6))
def test_memcpy_tiny_noc(simmod, oracle_lib, engine, seed):
    w = tiny_noc(seed)
    if engine == "b1":
        w.bw[:] = 1
        w.cap[:] = np.maximum(w.cap, 2 * (w.lat + 1))
    check_engine(simmod, oracle_lib, w, engine)


@pytest.mark.parametrize("U,W", [(1, 1), (4, 16), (8, 64)])
def test_memcpy_generic_gpu_local_copy(simmod, oracle_lib, U, W):
    w, lay = noc.gpu_noc(1)
    wm = noc.memcpy_workload(w, noc.local_copy_ops(lay, 128 * 6, n_wg=128, unroll=U, window=W),
                             name=f"gpu_local_copy_U{U}_W{W}")
    say(f"{wm.name}")
    check_vs_oracle(simmod, oracle_lib, wm)


@pytest.mark.parametrize("engine", ["workgroup", "workgroup_scan", "lane", "lanehbm", "resident"])
def test_memcpy_generic_gpu_sweep(simmod, oracle_lib, engine):
    w, lay = noc.gpu_noc(1)
    wm = noc.memcpy_workload(w, noc.local_copy_ops(lay, 32 * 8, n_wg=32, unroll=4, window=8), name="gpu_sweep")
    wm = noc.with_scenarios(wm, 5, seed=7)
    check_engine(simmod, oracle_lib, wm, engine)


@pytest.mark.parametrize("kind", ["allgather", "alltoall"])
def test_memcpy_two_gpus(simmod, oracle_lib, kind):
    w, lay = noc.gpu_noc(2)
    mc = noc.allgather_ops(lay, 2 * 32 * 2, n_wg=32) if kind == "allgather" else noc.alltoall_ops(lay, 64, n_wg=32)
    wm = noc.memcpy_workload(w, mc, name=f"two_gpu_{kind}")
    say(wm.name)
    check_vs_oracle(simmod, oracle_lib, wm)


@pytest.mark.parametrize("S", [300, 700, 1100])
def test_memcpy_workgroup_batch_sizes(simmod, oracle_lib, S):
    """The workgroup engine's launch shape follows the batch size (threads per
    workgroup and register budget chosen so that every scenario's workgroup
    is resident at once); each shape against the oracle, scenario by
    scenario."""
    w = noc.with_scenarios(tiny_noc(3, n_ops=8, max_lines=24), S, seed=S)
    check_engine(simmod, oracle_lib, w, "workgroup")


@pytest.mark.parametrize("kind,size,U,W", [("alltoall", 4096, 1, 64), ("alltoall", 4096, 8, 64),
                                           ("alltoall", 64, 16, 64), ("allgather", 16384, 16, 8),
                                           ("allgather", 16384, 16, 256), ("allgather", 128, 16, 4)])
def test_memcpy_exploration_points(simmod, oracle_lib, kind, size, U, W):
    """Points of the unroll and outstanding-limit sweeps (Sec. 5.3) whose
    trends tests/test_oracle_exploration.py checks on the oracle: the GPU
    path gives the same completion cycle for every line."""
    w, lay = noc.gpu_noc(2)
    mc = (noc.alltoall_ops(lay, size, n_wg=32, unroll=U, window=W) if kind == "alltoall"
          else noc.allgather_ops(lay, size, n_wg=32, unroll=U, window=W))
    wm = noc.memcpy_workload(w, mc, name=f"two_gpu_{kind}_{size}_U{U}_W{W}")
    say(wm.name)
    check_vs_oracle(simmod, oracle_lib, wm)


# ------------------------------------------- reduces, releases and acquires

def tiny_ops(seed):
    from tests.test_oracle_gpu_ops import random_program
    w, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1,
                         noc=(4, 1, 8), cu_out=(2, 1, 4), mem=(1, 2, 3))
    rng = np.random.default_rng(500 + seed)
    rows = random_program(rng, lay.cus[0], 1, int(rng.integers(1, 4)))
    mc = noc._prog(rows, lay, int(rng.integers(1, 5)), int(rng.integers(1, 9)))
    wm = noc.memcpy_workload(w, mc, name=f"tiny_ops_{seed}")
    wm.arb = seed % 2
    return wm


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("seed", range(8))
def test_gpu_ops_tiny_noc(simmod, oracle_lib, engine, seed):
    """Random programs of copies, reduces, releases and acquires (some of
    them deadlock: both sides must say so at the same point)."""
    w = tiny_ops(seed)
    if engine == "b1":
        w.bw[:] = 1
        w.cap[:] = np.maximum(w.cap, 2 * (w.lat + 1))
    check_engine(simmod, oracle_lib, w, engine)


@pytest.mark.parametrize("get", [True, False])
@pytest.mark.parametrize("G", [2, 4])
def test_reducescatter_generic_gpu(simmod, oracle_lib, G, get):
    """Get- and put-based reduce-scatter (Sec. 5.2) on G generic GPUs, 32
    workgroups per GPU, two lines per workgroup slice."""
    w, lay = noc.gpu_noc(G)
    mc = noc.reducescatter_ops(lay, G * 32 * 2, n_wg=32, get=get)
    wm = noc.memcpy_workload(w, mc, name=f"rs_{'get' if get else 'put'}_G{G}")
    say(wm.name)
    check_vs_oracle(simmod, oracle_lib, wm)


@pytest.mark.parametrize("engine", ["workgroup", "workgroup_scan", "lane", "lanehbm", "resident"])
@pytest.mark.parametrize("get", [True, False])
def test_reducescatter_engines(simmod, oracle_lib, engine, get):
    w, lay = noc.gpu_noc(3, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    mc = noc.reducescatter_ops(lay, 3 * 8 * 3, n_wg=8, unroll=2, window=6, get=get)
    wm = noc.with_scenarios(noc.memcpy_workload(w, mc, name=f"rs_small_{int(get)}"), 4, seed=11)
    check_engine(simmod, oracle_lib, wm, engine)
