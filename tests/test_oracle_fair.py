"""Pins of class-fair arbitration (control and data messages take turns,
the remedy of Sec. 5.2 for control messages stuck behind data responses).

* with only data messages the flag changes nothing;
* two sources, one sending data and one control lines, share one link:
  lowest id passes all data first, fair arbitration alternates data and
  control cycle by cycle (closed forms);
* the literal stepper (its own interleaving) on random graphs, DAGs and
  classes, and on memcpy programs, whose load requests are control.
"""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from tests.ref_stepper import step_simulate
from tests.test_oracle_memcpy import model


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_data_only_unchanged(oracle_lib, name):
    w = si.config(name)
    a = oracle_lib.simulate_workload(w)
    w.arb |= si.ARB_FAIR_CLASSES
    b = oracle_lib.simulate_workload(w, check=True)
    assert np.array_equal(a.completion, b.completion)


def shared_link(N):
    """Endpoints 0 (data) and 1 (control) -> switch 3 -> endpoint 2."""
    edges = [(0, 3), (3, 0), (1, 3), (3, 1), (2, 3), (3, 2)]
    rp, ci, lid = si._csr(4, edges)
    m = len(lid)
    one = np.ones(m, np.int32)
    src = [0] * N + [1] * N
    dst = [2] * (2 * N)
    cls = [0] * N + [1] * N
    return rp, ci, one, np.full(m, 4 * N, np.int32), src, dst, cls


@pytest.mark.parametrize("N", [1, 3, 8])
def test_turns_on_a_shared_link(oracle_lib, N):
    rp, ci, one, cap, src, dst, cls = shared_link(N)
    txns = (src, dst, np.zeros(2 * N + 1, np.int64), np.zeros(0, np.int64))
    j = np.arange(N)
    # lowest id: the shared link admits data j at 1 + j, control j at 1 + N + j
    r = oracle_lib.simulate(4, 3, rp, ci, one, one, cap, 0, txns=txns, cls=cls, check=True)
    assert np.array_equal(r.completion, np.concatenate([1 + j + 2, 1 + N + j + 2]))
    # fair: data j at 1 + 2j, control j at 2 + 2j
    r = oracle_lib.simulate(4, 3, rp, ci, one, one, cap, 2, txns=txns, cls=cls, check=True)
    assert np.array_equal(r.completion, np.concatenate([1 + 2 * j + 2, 2 + 2 * j + 2]))


@pytest.mark.parametrize("seed", range(60))
def test_brute_force_vs_stepper(oracle_lib, seed):
    rng = np.random.default_rng(13000 + seed)
    n_end = int(rng.integers(2, 6))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 3)), int(rng.integers(0, 5)),
                                              bmax=3, Lmax=3, capmax=5)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 120)), max_preds=2)
    cls = rng.integers(0, 2, size=len(src)).astype(np.uint8)
    arb = 2 + seed % 2
    r = oracle_lib.simulate(n, n_end, rp, ci, bw, lat, cap, arb, txns=(src, dst, pptr, pidx), cls=cls, check=True)
    preds = [list(pidx[pptr[x]:pptr[x + 1]]) for x in range(len(src))]
    st = step_simulate(n, n_end, rp, ci, bw, lat, cap, arb, src, dst, preds, max_cycles=20000, cls=cls)
    assert r.status_name == st[0]
    if st[0] == "OK":
        assert list(r.completion) == st[1]


@pytest.mark.parametrize("seed", range(6))
def test_memcpy_requests_are_control(oracle_lib, seed):
    w, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1,
                         noc=(2, 1, 3), cu_out=(2, 1, 3), mem=(1, 2, 2))
    rng = np.random.default_rng(seed)
    rows = [(int(rng.choice(lay.cus[0])), 0, 0, int(rng.integers(0, 9)), 20 + int(rng.integers(0, 9)),
             int(rng.integers(1, 6))) for _ in range(5)]
    mc = noc._ops(rows, lay, int(rng.integers(1, 4)), int(rng.integers(1, 6)))
    wm = noc.memcpy_workload(w, mc)
    wm.arb = si.ARB_FAIR_CLASSES + seed % 2
    r = oracle_lib.simulate_workload(wm, check=True)
    src, dst, preds = model(mc)
    _, _, _, _, ocls = oracle_lib.memcpy_txns(mc, with_class=True)
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, wm.arb, src, dst, preds,
                       max_cycles=20000, cls=list(ocls))
    assert st[0] == r.status_name
    assert list(r.completion) == st[1]
    # the request lines are exactly the lines whose one dependant is their reply
    req = [i for i in range(len(src)) if ocls[i] == 1]
    assert all(preds[x + 1] == [x] and src[x + 1] == dst[x] and dst[x + 1] == src[x] for x in req)
    assert len(req) == int(mc.n_lines.sum())


@pytest.mark.parametrize("seed", [103, 105])
def test_fair_never_reorders_a_flow(oracle_lib, seed):
    """Regression: interleaving classes over all offered lines put a source's
    later control line ahead of its earlier data line within one cycle, so a
    flow delivered out of id order.  Picks are taken among heads only."""
    from tests.test_gpu_memcpy import tiny_noc
    w = tiny_noc(seed)
    w.arb |= si.ARB_FAIR_CLASSES
    r = oracle_lib.simulate_workload(w, check=True)   # check mode verifies per-flow order
    assert r.status_name in ("OK", "DEADLOCK")
    mc = w.meta["memcpy"]
    src, dst, _ = model(mc)
    last = {}
    for x, c in enumerate(r.completion):
        if c == 0xFFFFFFFF:
            continue
        assert c >= last.get((src[x], dst[x]), 0)
        last[(src[x], dst[x])] = int(c)
