"""GPU parity of the LDS-resident workgroup engine with its LDS capacities
cut down for the test (SIMGPU_RES_RCAP request records, SIMGPU_RES_TCAP
per-target words), so that most of a cycle's records and target words live
in the per-scenario HBM overflow areas: key, round-robin and class-fair
arbitration, GPU programs with reduces and releases, credit delays, against
the CPU oracle through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from tests.test_gpu_parity import check_engine, simmod, torch_cuda, say  # noqa: F401
from tests.test_gpu_memcpy import tiny_noc, tiny_ops

pytestmark = pytest.mark.gpu

# (request records, per-target words) kept in LDS; the rest in HBM
CAPS = [(1, 1), (16, 4), (64, 256)]


def _caps(monkeypatch, rcap, tcap):
    monkeypatch.setenv("SIMGPU_RES_RCAP", str(rcap))
    monkeypatch.setenv("SIMGPU_RES_TCAP", str(tcap))


@pytest.mark.parametrize("rcap,tcap", CAPS)
@pytest.mark.parametrize("fair", [False, True])
@pytest.mark.parametrize("seed", range(4))
def test_resident_overflow_tiny_noc(simmod, oracle_lib, monkeypatch, rcap, tcap, fair, seed):
    _caps(monkeypatch, rcap, tcap)
    w = tiny_noc(200 + seed)
    if fair:
        w.arb |= si.ARB_FAIR_CLASSES
    check_engine(simmod, oracle_lib, w, "resident", must_run=True)


@pytest.mark.parametrize("rcap,tcap", CAPS[:2])
@pytest.mark.parametrize("seed", range(4))
def test_resident_overflow_gpu_ops(simmod, oracle_lib, monkeypatch, rcap, tcap, seed):
    """Programs of copies, reduces, releases and acquires (some deadlock)."""
    _caps(monkeypatch, rcap, tcap)
    check_engine(simmod, oracle_lib, tiny_ops(seed), "resident", must_run=True)


@pytest.mark.parametrize("fair", [False, True])
def test_resident_overflow_two_gpu_allgather(simmod, oracle_lib, monkeypatch, fair):
    """Put-based all-gather of 64 KiB per GPU on two generic GPUs (a busy
    cycle has hundreds of requests), round-robin, three scenarios."""
    _caps(monkeypatch, 32, 8)
    w, lay = noc.gpu_noc(2)
    wm = noc.memcpy_workload(w, noc.allgather_ops(lay, 512, n_wg=32, unroll=4, window=64), name="ag_64k_spill")
    wm.arb = 1 | (si.ARB_FAIR_CLASSES if fair else 0)
    wm = noc.with_scenarios(wm, 3, seed=21)
    say(wm.name)
    check_engine(simmod, oracle_lib, wm, "resident", must_run=True)


def test_resident_overflow_credit(simmod, oracle_lib, monkeypatch):
    """Credit delays equal to the latency on sampled C5 scenarios."""
    _caps(monkeypatch, 8, 2)
    w = si.take_scenarios(si.config("C5"), [5, 1000, 3001])
    w.credit = w.lat.copy()
    check_engine(simmod, oracle_lib, w, "resident", must_run=True)


@pytest.mark.parametrize("engine", ["resident", "workgroup"])
@pytest.mark.parametrize("scap", [0, 3])
@pytest.mark.parametrize("fair", [False, True])
def test_short_spill_list(simmod, oracle_lib, monkeypatch, engine, scap, fair):
    """A FIFO offer longer than one chunk hands its later chunks to other
    threads through a spill list; with the list cut short (SIMGPU_SPILL_CAP)
    the chunks that do not fit are read inline by the link's own thread.
    Router links of b = 64 on two generic GPUs make such offers."""
    monkeypatch.setenv("SIMGPU_SPILL_CAP", str(scap))
    w, lay = noc.gpu_noc(2)
    wm = noc.memcpy_workload(w, noc.allgather_ops(lay, 512, n_wg=32, unroll=4, window=64), name="ag_64k_short_spill")
    wm.arb = (si.ARB_FAIR_CLASSES | 1) if fair else 0
    wm = noc.with_scenarios(wm, 3, seed=23)
    say(f"{wm.name} {engine} scap={scap}")
    check_engine(simmod, oracle_lib, wm, engine, must_run=True)
