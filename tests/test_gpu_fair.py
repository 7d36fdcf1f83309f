"""GPU parity of class-fair arbitration (control and data messages take
turns) against the CPU oracle, through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from tests.test_gpu_parity import ENGINES, check_engine, check_vs_oracle, simmod, torch_cuda, say  # noqa: F401
from tests.test_gpu_memcpy import tiny_noc

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("seed", range(8))
def test_fair_tiny_noc(simmod, oracle_lib, engine, seed):
    w = tiny_noc(100 + seed)
    w.arb |= si.ARB_FAIR_CLASSES
    # both forms of the workgroup engine take class-fair arbitration
    check_engine(simmod, oracle_lib, w, engine, must_run=engine in ("workgroup", "resident"))


@pytest.mark.parametrize("get", [False, True])
@pytest.mark.parametrize("rr", [0, 1])
def test_fair_two_gpu_allgather(simmod, oracle_lib, get, rr):
    w, lay = noc.gpu_noc(2)
    wm = noc.memcpy_workload(w, noc.allgather_ops(lay, 2 * 32 * 2, n_wg=32, get=get), name=f"ag_get{int(get)}")
    wm.arb = rr | si.ARB_FAIR_CLASSES
    wm = noc.with_scenarios(wm, 3, seed=5)
    say(wm.name)
    check_vs_oracle(simmod, oracle_lib, wm)


def test_fair_collective_is_data_only(simmod, oracle_lib):
    w = si.torus2d(4, 4, n_scenarios=4, seed=31, bws=(1, 2, 4), lat_lo=1, lat_hi=20, depths=(2, 7, 32),
                   nbytes=128 * 16 * 3, arb=si.ARB_FAIR_CLASSES | 1)
    check_vs_oracle(simmod, oracle_lib, w)


@pytest.mark.parametrize("engine", ["resident", "workgroup"])
def test_fair_noc_allgather_512k(simmod, oracle_lib, engine):
    """Put-based all-gather of 512 KiB per GPU on two generic GPUs under
    round-robin with class turns (control and data), four scenarios of
    channel and cable latencies, on the LDS-resident and the generic
    workgroup engine."""
    w, lay = noc.gpu_noc(2)
    wm = noc.memcpy_workload(w, noc.allgather_ops(lay, 4096, n_wg=32, unroll=4, window=64), name="ag_fair_512k")
    wm.arb = 1 | si.ARB_FAIR_CLASSES
    wm = noc.with_scenarios(wm, 4, seed=9)
    check_engine(simmod, oracle_lib, wm, engine, must_run=True)
