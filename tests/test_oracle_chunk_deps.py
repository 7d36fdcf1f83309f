"""Pins of the oracle's chunk-dependency mode (put + signal: a collective step
waits for the whole chunk of the step before it), against closed forms and
against the plain definition written out as an explicit DAG.

Dependency granularity follows Sec. 4.2 and 5.2 (get-style line-level
overlap versus put + signal per chunk).  The closed forms hold on dedicated
one-hop links (full mesh) with buffers of at least b(L+1) lines, where no
line ever waits for a slot: a chunk of C lines leaves at b lines per cycle,
its last line is delivered D = floor((C-1)/b) + L + 1 cycles after the step
starts, and the next step starts then.
"""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from tests.ref_stepper import step_simulate

DEP_CHUNK = si.DEP_CHUNK


@pytest.mark.parametrize("p,C,b,L", [(2, 5, 1, 3), (3, 8, 1, 2), (4, 6, 2, 9), (5, 4, 1, 10), (8, 16, 1, 50),
                                     (6, 12, 3, 2), (4, 7, 2, 5)])
def test_ring_chunk_closed_form(oracle_lib, p, C, b, L):
    # comp(s, i, j) = s*D + floor(j/b) + L + 1, makespan 2(p-1) D.
    w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=si.COLL_RING_ALLREDUCE, nbytes=128 * C * p)
    w.dep = DEP_CHUNK
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.status_name == "OK"
    D = (C - 1) // b + L + 1
    ids = np.arange(len(r.completion))
    j = ids % C
    s = ids // (C * p)
    assert np.array_equal(r.completion, s * D + j // b + L + 1)
    assert r.makespan == 2 * (p - 1) * D


@pytest.mark.parametrize("p,C,b,L", [(2, 4, 1, 3), (3, 6, 1, 4), (4, 128, 1, 10), (4, 8, 2, 20), (5, 10, 1, 2)])
def test_direct_chunk_closed_form(oracle_lib, p, C, b, L):
    # Reduce-scatter: comp = floor(j/b) + L + 1; all-gather starts when every
    # reduce-scatter chunk into its source is delivered, at D; makespan 2D.
    w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=si.COLL_DIRECT_ALLREDUCE, nbytes=128 * C * p)
    w.dep = DEP_CHUNK
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.status_name == "OK"
    D = (C - 1) // b + L + 1
    ids = np.arange(len(r.completion))
    j = ids % C
    ph = ids // (C * p * (p - 1))
    assert np.array_equal(r.completion, ph * D + j // b + L + 1)
    assert r.makespan == 2 * D


def test_c1_chunk_makespan(oracle_lib):
    # C1 with chunk dependencies: 2 * (128 + 10) = 276, against 266 per line.
    w = si.config("C1")
    w.dep = DEP_CHUNK
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.makespan == 276


def explicit_dag(oracle_lib, w):
    """The workload with every chunk predecessor written out as all its lines."""
    rc, _, _, _, T = oracle_lib.txn(w.coll, w.bytes, 0, w.n_endpoints, 0, w.order, w.dep)
    assert rc == 0
    C = w.bytes // 128 // w.n_endpoints
    src, dst, preds = [], [], []
    for x in range(T):
        rc, s, d, pr, _ = oracle_lib.txn(w.coll, w.bytes, 0, w.n_endpoints, x, w.order, w.dep)
        src.append(s)
        dst.append(d)
        full = []
        for q in pr:
            if q >= 0:
                full.append(q)
            else:
                c = -1 - q
                full.extend(range(c * C, (c + 1) * C))
        preds.append(full)
    return src, dst, preds


def to_csr(preds):
    ptr = np.zeros(len(preds) + 1, np.int64)
    ptr[1:] = np.cumsum([len(p) for p in preds])
    idx = np.array([q for p in preds for q in p], np.int64)
    return ptr, idx


@pytest.mark.parametrize("seed", range(10))
def test_chunk_mode_equals_explicit_dag(oracle_lib, seed):
    """The join counters reproduce the definition: every line waits for all
    lines of its predecessor chunks."""
    coll = [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE][seed % 2]
    X, Y = [(2, 2), (3, 2), (2, 3)][seed % 3]
    w = si.torus2d(X, Y, n_scenarios=1, seed=300 + seed, bws=(1, 2, 3), lat_lo=1, lat_hi=6, depths=(1, 2, 4, 7),
                   nbytes=128 * X * Y * [3, 5][seed % 2], coll=coll, arb=seed // 2 % 2)
    w.dep = DEP_CHUNK
    got = oracle_lib.simulate_workload(w, check=True)
    src, dst, preds = explicit_dag(oracle_lib, w)
    ptr, idx = to_csr(preds)
    want = oracle_lib.simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb,
                               txns=(src, dst, ptr, idx), check=True)
    assert got.status_name == want.status_name == "OK"
    assert np.array_equal(got.completion, want.completion)
    assert np.array_equal(got.tx_lines, want.tx_lines) and np.array_equal(got.busy_cycles, want.busy_cycles)
    assert got.makespan == want.makespan
    # and the literal per-cycle stepper agrees with both
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb, src, dst, preds,
                       max_cycles=50000)
    assert st[0] == "OK" and list(got.completion) == st[1]


def test_chunk_mode_not_defined_for_hierarchical(oracle_lib):
    rc, *_ = oracle_lib.txn(si.COLL_HIER_ALLREDUCE, 128 * 8 * 4, 2, 4, 0, None, DEP_CHUNK)
    assert rc == 1  # invalid argument


def test_c2_chunk_closed_form(oracle_lib):
    # 8-endpoint mesh ring, C = 16384 lines, b = 1, L = 50, cap 64 >= b(L+1):
    # D = 16383 + 51 and the makespan is 14 D.
    w = si.config("C2_chunk")
    assert w.dep == si.DEP_CHUNK
    r = oracle_lib.simulate_workload(w, check=True)
    D = 16383 + 51
    assert r.makespan == 14 * D
    ids = np.arange(len(r.completion))
    assert np.array_equal(r.completion, (ids // (16384 * 8)) * D + ids % 16384 + 51)
