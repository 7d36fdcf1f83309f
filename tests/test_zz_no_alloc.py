"""sim_run_noalloc (the allocation-free run) against sim_run, through the C
ABI, bit for bit: every engine's scratch placed in the library's fixed device
array.  Two calls in a row per engine, the second on a smaller workload, so
that the second run starts on the first one's leftovers."""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

import sim_inputs as si

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def simmod():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2606_10440_amd import sim
    sim.lib()
    return sim


def _outputs(s):
    return s.alloc_outputs()


def _run(simmod, s, noalloc):
    import torch
    outs = s.alloc_outputs()
    for t in outs:
        t.fill_(-1)
    st = torch.cuda.current_stream()
    comp, tx, busy, mk = outs
    fn = simmod.sim_run_noalloc if noalloc else simmod.sim_run
    fn(s.ctx, st.cuda_stream, comp.data_ptr(), tx.data_ptr(), busy.data_ptr(), mk.data_ptr(), 0)
    st.synchronize()
    rc, status, cycles = simmod.sim_status_after_sync(s.ctx, s.S)
    return rc, status, cycles, [t.cpu().numpy() for t in outs]


def _pair(simmod, w, engine):
    print(f"no-alloc vs sim_run: {w.name} S={w.n_scenarios} engine={engine}", file=sys.stderr, flush=True)
    old = os.environ.get("SIMGPU_ENGINE")
    os.environ["SIMGPU_ENGINE"] = engine
    try:
        s = simmod.Simulator.from_workload(w)
    finally:
        if old is None:
            os.environ.pop("SIMGPU_ENGINE", None)
        else:
            os.environ["SIMGPU_ENGINE"] = old
    try:
        want = _run(simmod, s, False)
        got = _run(simmod, s, True)
    finally:
        s.close()
    assert want[0] == got[0] == 0
    assert np.array_equal(want[1], got[1]) and np.array_equal(want[2], got[2])
    for a, b in zip(want[3], got[3]):
        assert np.array_equal(a, b)


def _torus(S, seed, nbytes):
    return si.torus2d(4, 4, n_scenarios=S, seed=seed, bws=(1, 2, 4), lat_lo=1, lat_hi=30, depths=(2, 5, 16, 32),
                      nbytes=nbytes)


@pytest.mark.parametrize("engine", ["wave", "lane", "lanehbm", "workgroup", "resident"])
def test_noalloc_matches_run_twice(simmod, engine):
    _pair(simmod, _torus(24, 300, 128 * 16 * 24), engine)
    _pair(simmod, _torus(5, 301, 128 * 16 * 6), engine)


def test_noalloc_compact_engine_twice(simmod):
    _pair(simmod, si.fat_tree(4, nbytes=128 * 40, cap=5, lat_lo=2, lat_hi=9, arb=1), "b1")
    _pair(simmod, si.fat_tree(4, nbytes=128 * 7, cap=3, lat_lo=1, lat_hi=4, arb=0), "b1")


def test_noalloc_grid_engine_twice(simmod):
    # one topology over several cooperating workgroups (one-line form), then
    # a smaller one
    _pair(simmod, si.scaled(si.config("C2"), bytes=128 * 8 * 40), "grid")
    _pair(simmod, si.scaled(si.config("C1"), bytes=128 * 4 * 6), "grid")


def test_noalloc_c5_then_smaller(simmod):
    w = si.take_scenarios(si.config("C5"), range(0, 4096, 16))
    _pair(simmod, si.scaled(w, bytes=128 * 16 * 64), "wave")
    _pair(simmod, si.scaled(si.take_scenarios(w, range(7)), bytes=128 * 16 * 8), "wave")


@pytest.mark.parametrize("engine", ["resident", "workgroup"])
def test_noalloc_noc_fair_then_credit(simmod, engine):
    """Class-fair arbitration on a small NoC running memcpy programs (four
    scenarios), then a torus with credit delays, on both workgroup engines."""
    from sim_inputs import noc
    from tests.test_gpu_memcpy import tiny_noc
    wm = tiny_noc(105, n_ops=8, max_lines=24)
    wm.arb = 1 | si.ARB_FAIR_CLASSES
    _pair(simmod, noc.with_scenarios(wm, 4, seed=3), engine)
    t = _torus(4, 303, 128 * 16 * 4)
    t.credit = t.lat.copy()
    _pair(simmod, t, engine)


def test_noalloc_rejects_oversized_scratch(simmod):
    w = _torus(4096, 302, 128 * 16)
    old = os.environ.get("SIMGPU_ENGINE")
    os.environ["SIMGPU_ENGINE"] = "workgroup"
    try:
        s = simmod.Simulator.from_workload(w)
    finally:
        if old is None:
            os.environ.pop("SIMGPU_ENGINE", None)
        else:
            os.environ["SIMGPU_ENGINE"] = old
    try:
        comp, tx, busy, mk = s.alloc_outputs()
        with pytest.raises(simmod.SimError) as e:
            simmod.sim_run_noalloc(s.ctx, 0, comp.data_ptr(), tx.data_ptr(), busy.data_ptr(), mk.data_ptr(), 0)
        assert e.value.status == simmod.SIM_ERR_SIZE
    finally:
        s.close()
