"""Pins of the oracle's memcpy programs: the injection side of the GPU model
(Sec. 4.4.3 wavefront requests, 4.4.4 loop unrolling, the outstanding
request limit of Sec. 5.3) compiled into line transfers.

* an independent model of the CU programs (written here from the rules:
  per CU, U loads, wait, U stores; a load = request + data; at most W
  outstanding, retired in order; ids step-major over CUs) must give the
  oracle's senders, receivers and dependency sets line for line;
* hand-derived timelines on the smallest topology (one CU, one router, a
  source and a destination channel): W = 1 serialises every wavefront
  request, W and U unbounded overlap all loads;
* a max-plus recursion (per-stream rate, release = latest dependency,
  contention-free paths) on that topology for every U and W;
* the literal stepper on a tiny NoC;
* the generic GPU: 448 nodes per GPU as the paper counts them.
"""
from __future__ import annotations

from collections import defaultdict

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from tests.ref_stepper import step_simulate


def model(mc):
    """(src, dst, preds) of every line, from the program rules."""
    chan = lambda s, a: int(mc.space_channels[s * mc.n_ch + a % mc.n_ch])
    progs = defaultdict(list)   # cu -> [(kind, channel, group of load indices)]
    for o in range(len(mc.cu)):
        c, n = int(mc.cu[o]), int(mc.n_lines[o])
        for j0 in range(0, n, mc.unroll):
            grp = list(range(j0, min(n, j0 + mc.unroll)))
            first = len(progs[c])
            for j in grp:
                progs[c].append(("load", chan(int(mc.src_space[o]), int(mc.src_line[o]) + j), None))
            loads = list(range(first, first + len(grp)))
            for j in grp:
                progs[c].append(("store", chan(int(mc.dst_space[o]), int(mc.dst_line[o]) + j), loads))
    ids = {}
    order = []
    for k in range(max((len(p) for p in progs.values()), default=0)):
        for c in sorted(progs):
            if k < len(progs[c]):
                ids[(c, k)] = len(order)
                kind = progs[c][k][0]
                order.append((c, k, "issue"))
                if kind == "load":
                    order.append((c, k, "data"))
    done = lambda c, k: ids[(c, k)] + (1 if progs[c][k][0] == "load" else 0)
    src, dst, preds = [], [], []
    for c, k, part in order:
        kind, ch, grp = progs[c][k]
        if part == "data":
            src.append(ch), dst.append(c), preds.append([ids[(c, k)]])
            continue
        p = [done(c, k - mc.window)] if k >= mc.window else []
        if kind == "store":
            p += [ids[(c, g)] + 1 for g in grp]
        src.append(c), dst.append(ch), preds.append(p)
    return src, dst, preds


def tiny(Lc=1, Lm=1, bc=1, bm=8):
    """Nodes: CU 0, channels 1 (source) and 2 (destination), router 3."""
    edges = [(0, 3), (3, 0), (1, 3), (3, 1), (2, 3), (3, 2)]
    rp, ci, lid = si._csr(4, edges)
    m = len(lid)
    bw = np.full(m, 64, np.int32)
    lat = np.full(m, 1, np.int32)
    cap = np.full(m, 4096, np.int32)
    for (u, v), i in lid.items():
        if u == 0:
            bw[i], lat[i] = bc, Lc
        if 3 in (u, v) and 0 not in (u, v):
            bw[i], lat[i] = bm, Lm
        if v == 0:
            lat[i] = Lc
    return si.Workload("tiny", 4, 3, rp, ci, 1, bw, lat, cap, 0, -1, 0)


def copy(n, U, W, n_ops=1):
    return noc.Memcpy(np.zeros(n_ops, np.int32), np.zeros(n_ops, np.int32), np.ones(n_ops, np.int32),
                      np.arange(n_ops, dtype=np.int64) * n, np.arange(n_ops, dtype=np.int64) * n,
                      np.full(n_ops, n, np.int64), np.array([1, 2], np.int32), 1, U, W)


def run(oracle_lib, w, mc, check=True):
    return oracle_lib.simulate_workload(noc.memcpy_workload(w, mc), check=check)


@pytest.mark.parametrize("U,W", [(1, 1), (1, 3), (4, 64), (3, 5), (8, 2), (2, 1000)])
def test_expansion_matches_model(oracle_lib, U, W):
    w, lay = noc.gpu_noc(2, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    rng = np.random.default_rng(U * 100 + W)
    rows = []
    for _ in range(9):
        cu = int(rng.choice(lay.cus.reshape(-1)))
        rows.append((cu, int(rng.integers(0, 2)), int(rng.integers(0, 2)), int(rng.integers(0, 50)),
                     int(rng.integers(0, 50)), int(rng.integers(0, 7))))
    mc = noc._ops(rows, lay, U, W)
    src, dst, pptr, pidx = oracle_lib.memcpy_txns(mc)
    ms, md, mp = model(mc)
    assert list(src) == ms and list(dst) == md
    assert [sorted(pidx[pptr[x]:pptr[x + 1]].tolist()) for x in range(len(src))] == [sorted(p) for p in mp]


@pytest.mark.parametrize("n,Lc,Lm", [(1, 1, 1), (5, 1, 1), (7, 3, 2), (4, 2, 9)])
def test_window_one_serialises(oracle_lib, n, Lc, Lm):
    # W = 1: request, data, store, next request ... each one after the other;
    # every leg crosses two links: a request Lc + Lm + 1, data Lm + Lc + 1, a
    # store Lc + Lm + 1; a line takes 3 (Lc + Lm + 1) cycles.
    r = run(oracle_lib, tiny(Lc, Lm), copy(n, U=1, W=1))
    leg = Lc + Lm + 1
    want = []
    for j in range(n):
        t0 = 3 * leg * j
        want += [t0 + leg, t0 + 2 * leg, t0 + 3 * leg]
    assert list(r.completion) == want
    assert r.makespan == 3 * leg * n


@pytest.mark.parametrize("n", [1, 2, 6, 13])
def test_unbounded_overlap(oracle_lib, n):
    # U = n, W large, one request per cycle: load j leaves at cycle j (data
    # back at j + 6); the stores wait for all data (n + 5) and then leave one
    # per cycle: store j completes at n + 5 + j + 3; makespan 2n + 7.
    r = run(oracle_lib, tiny(), copy(n, U=n, W=10 ** 6))
    comp = list(r.completion)
    loads = [comp[2 * j] for j in range(n)], [comp[2 * j + 1] for j in range(n)]
    assert loads[0] == [j + 3 for j in range(n)] and loads[1] == [j + 6 for j in range(n)]
    assert comp[2 * n:] == [n + 5 + j + 3 for j in range(n)]
    assert r.makespan == 2 * n + 7


def max_plus(w, src, dst, preds):
    """Completion times when only the injection streams can hold a line back
    (every later link has spare bandwidth and buffer): stream (src, first
    link) admits in id order, at most b per cycle, once released; a line then
    needs the latencies of its path plus one."""
    rp, ci = w.row_ptr, w.col_idx
    link = {(u, int(ci[l])): l for u in range(w.n_nodes) for l in range(rp[u], rp[u + 1])}
    hub = 3
    T = len(src)
    comp = [0] * T
    while True:
        new = [0] * T
        streams = defaultdict(list)
        for x in range(T):
            l1, l2 = link[(src[x], hub)], link[(hub, dst[x])]
            a = streams[l1]
            v = max((comp[q] for q in preds[x]), default=0)
            if a:
                v = max(v, a[-1])
            b = int(w.bw[l1])
            if len(a) >= b:
                v = max(v, a[-b] + 1)
            a.append(v)
            new[x] = v + int(w.lat[l1]) + int(w.lat[l2]) + 1
        if new == comp:
            return comp
        comp = new


@pytest.mark.parametrize("U,W,n,ops", [(1, 2, 9, 1), (2, 3, 8, 2), (4, 4, 9, 1), (4, 8, 16, 3), (3, 100, 10, 2),
                                       (5, 7, 12, 1), (1, 64, 20, 1)])
@pytest.mark.parametrize("bc", [1, 2, 5])
def test_max_plus_on_tiny(oracle_lib, U, W, n, ops, bc):
    w = tiny(Lc=2, Lm=3, bc=bc)
    mc = copy(n, U, W, ops)
    r = run(oracle_lib, w, mc)
    src, dst, preds = model(mc)
    assert list(r.completion) == max_plus(w, src, dst, preds)


@pytest.mark.parametrize("seed", range(6))
def test_stepper_on_tiny_noc(oracle_lib, seed):
    w, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=1, ch_per_router=2, ports_per_router=1,
                         noc=(2, 1, 3), cu_out=(1, 1, 2), mem=(1, 2, 2))
    rng = np.random.default_rng(seed)
    rows = [(int(rng.choice(lay.cus[0])), 0, 0, int(rng.integers(0, 9)), 20 + int(rng.integers(0, 9)),
             int(rng.integers(1, 6))) for _ in range(4)]
    mc = noc._ops(rows, lay, int(rng.integers(1, 4)), int(rng.integers(1, 6)))
    wm = noc.memcpy_workload(w, mc)
    wm.arb = seed % 2
    r = oracle_lib.simulate_workload(wm, check=True)
    src, dst, preds = model(mc)
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, wm.arb, src, dst,
                       preds, max_cycles=20000)
    assert st[0] == r.status_name
    assert list(r.completion) == st[1]


def test_generic_gpu_counts():
    # 32 routers + 128 CUs + 256 channels + 32 ports = 448 nodes per GPU.
    for G in (1, 2, 4):
        w, lay = noc.gpu_noc(G)
        switches = 32 if G > 1 else 0
        assert w.n_nodes == 448 * G + switches and w.n_endpoints == 384 * G
        assert lay.cus.size == 128 * G and lay.channels.size == 256 * G and lay.ports.size == 32 * G


def test_bad_programs_rejected(oracle_lib):
    mc = copy(4, 2, 2)
    mc.unroll = 0
    with pytest.raises(ValueError):
        oracle_lib.memcpy_txns(mc)
    mc = copy(4, 2, 2)
    mc.src_space = np.array([5], np.int32)
    with pytest.raises(ValueError):
        oracle_lib.memcpy_txns(mc)
