"""Pins of the credit-delay flow-control variant: a slot freed by a line
leaving link l at cycle t is seen free by l's arbiter from t + D on (D = 1 is
the base model's start-of-cycle snapshot).

* D = 1 everywhere reproduces the base model exactly;
* one link, a stream of lines: the slot cycle becomes L + D, so admit(k) =
  floor(k/cap)(L + D) + floor((k mod cap)/b) while cap/b <= L + D;
* brute force against the literal stepper (which keeps owed credits as a
  plain list) on random tiny graphs, DAGs and delays, and on a small torus
  collective.
"""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from tests.ref_stepper import step_simulate


def one_link(b, L, cap, D):
    rp = np.array([0, 1, 2], np.int32)
    ci = np.array([1, 0], np.int32)
    return (2, 2, rp, ci, np.array([b, b], np.int32), np.array([L, L], np.int32), np.array([cap, cap], np.int32),
            np.array([D, D], np.int32))


@pytest.mark.parametrize("b,L,cap,D", [(1, 3, 2, 1), (1, 3, 2, 5), (2, 4, 4, 3), (3, 1, 6, 9), (4, 10, 8, 2),
                                       (1, 1, 1, 7)])
def test_single_link_slot_cycle(oracle_lib, b, L, cap, D):
    n, E, rp, ci, bw, lat, cp, cr = one_link(b, L, cap, D)
    N = 5 * cap + 3
    txns = ([0] * N, [1] * N, np.zeros(N + 1, np.int64), np.zeros(0, np.int64))
    r = oracle_lib.simulate(n, E, rp, ci, bw, lat, cp, 0, txns=txns, credit=cr, check=True)
    assert r.status_name == "OK"
    k = np.arange(N)
    admit = (k // cap) * (L + D) + (k % cap) // b
    assert np.array_equal(r.completion, admit + L + 1)


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_unit_delay_is_the_base_model(oracle_lib, name):
    w = si.config(name)
    a = oracle_lib.simulate_workload(w)
    w.credit = np.ones_like(w.cap)
    b = oracle_lib.simulate_workload(w, check=True)
    assert np.array_equal(a.completion, b.completion) and a.makespan == b.makespan
    assert a.processed_cycles == b.processed_cycles


@pytest.mark.parametrize("seed", range(80))
def test_brute_force_vs_stepper(oracle_lib, seed):
    rng = np.random.default_rng(9000 + seed)
    n_end = int(rng.integers(2, 6))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 3)), int(rng.integers(0, 5)),
                                              bmax=3, Lmax=4, capmax=5)
    m = len(ci)
    credit = rng.integers(1, 6, size=m).astype(np.int32)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 120)), max_preds=2)
    arb = seed % 2
    r = oracle_lib.simulate(n, n_end, rp, ci, bw, lat, cap, arb, txns=(src, dst, pptr, pidx), credit=credit,
                            check=True)
    preds = [list(pidx[pptr[x]:pptr[x + 1]]) for x in range(len(src))]
    st = step_simulate(n, n_end, rp, ci, bw, lat, cap, arb, src, dst, preds, max_cycles=20000, credit=credit)
    assert r.status_name == st[0]
    if st[0] == "OK":
        assert list(r.completion) == st[1]
        assert list(r.tx_lines) == st[2] and list(r.busy_cycles) == st[3]
    else:
        done = [c for c in st[1] if c is not None]
        assert sorted(done) == sorted(int(c) for c in r.completion if c != 0xFFFFFFFF)


@pytest.mark.parametrize("seed", range(4))
def test_torus_collective_vs_stepper(oracle_lib, seed):
    w = si.torus2d(3, 2, n_scenarios=1, seed=700 + seed, bws=(1, 2), lat_lo=1, lat_hi=4, depths=(2, 3, 5),
                   nbytes=128 * 6 * 3, coll=[si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE][seed % 2],
                   arb=seed // 2)
    w.credit = np.random.default_rng(seed).integers(1, 5, size=w.n_links).astype(np.int32)
    r = oracle_lib.simulate_workload(w, check=True)
    T = len(r.completion)
    dec = [oracle_lib.txn(w.coll, w.bytes, 0, w.n_endpoints, x)[1:4] for x in range(T)]
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb,
                       [d[0] for d in dec], [d[1] for d in dec], [d[2] for d in dec], max_cycles=50000,
                       credit=w.credit)
    assert st[0] == r.status_name == "OK"
    assert list(r.completion) == st[1]


def test_bad_delay_rejected(oracle_lib):
    n, E, rp, ci, bw, lat, cp, cr = one_link(1, 1, 1, 0)
    r = oracle_lib.simulate(n, E, rp, ci, bw, lat, cp, 0, txns=([0], [1], np.zeros(2, np.int64),
                                                              np.zeros(0, np.int64)), credit=cr)
    assert r.status_name == "TOPOLOGY"
