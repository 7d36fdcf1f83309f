"""Pins of the oracle's GPU programs beyond memcpy: reduces (a copy from
several sources), releases and acquires (Sec. 4.1.1-4.1.2 GPU instructions
and operations, 4.4.2-4.4.3 compute unit and wavefront requests), and the
get- and put-based reduce-scatter built from them (Sec. 5.2).

* an independent model of the CU programs, written here from the rules:
  per group of U lines the loads of every source, then the stores, which
  wait for all of them; a release waits for every earlier store of its CU
  (literally all of them here; the oracle lists a shorter set that gives
  the same times); an acquire's request waits for the release of its
  semaphore, and the request after it for its reply;
* hand-derived timelines: with W = 1 every request of a CU waits for the
  one before, so each leg of a reduce, and a release -> acquire hand-off
  between two CUs, follow one another;
* a max-plus recursion (contention-free star) and the literal stepper on a
  tiny NoC, both fed the model's dependencies;
* a program whose acquire comes before its own release deadlocks.
"""
from __future__ import annotations

from collections import defaultdict

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from sim_inputs.noc import OP_ACQUIRE, OP_COPY, OP_RELEASE
from tests.ref_stepper import step_simulate


def model(mc):
    """(src, dst, class, preds, what) of every line, from the program rules."""
    chan = lambda s, a: int(mc.space_channels[s * mc.n_ch + a % mc.n_ch])
    progs = defaultdict(list)   # cu -> [(kind, channel, loads of the group, semaphore)]
    for o in range(len(mc.cu)):
        c, n, kind = int(mc.cu[o]), int(mc.n_lines[o]), int(mc.kind[o])
        sem = (int(mc.dst_space[o]), int(mc.dst_line[o]))
        if kind == OP_RELEASE:
            progs[c].append(("release", chan(*sem), None, sem))
            continue
        if kind == OP_ACQUIRE:
            progs[c].append(("acquire", chan(*sem), None, sem))
            continue
        srcs = [(int(mc.src_space[i]), int(mc.src_line[i])) for i in range(mc.src_ptr[o], mc.src_ptr[o + 1])]
        for j0 in range(0, n, mc.unroll):
            grp = range(j0, min(n, j0 + mc.unroll))
            first = len(progs[c])
            for s, a in srcs:
                for j in grp:
                    progs[c].append(("load", chan(s, a + j), None, None))
            loads = list(range(first, len(progs[c])))
            for j in grp:
                progs[c].append(("store", chan(sem[0], sem[1] + j), loads, None))
    two = ("load", "acquire")
    ids, order = {}, []
    for k in range(max((len(p) for p in progs.values()), default=0)):
        for c in sorted(progs):
            if k < len(progs[c]):
                ids[(c, k)] = len(order)
                order.append((c, k, "issue"))
                if progs[c][k][0] in two:
                    order.append((c, k, "back"))
    released = {progs[c][k][3]: ids[(c, k)] for c in progs for k in range(len(progs[c]))
                if progs[c][k][0] == "release"}
    done = lambda c, k: ids[(c, k)] + (1 if progs[c][k][0] in two else 0)
    src, dst, cls, preds, what = [], [], [], [], []
    for c, k, part in order:
        kind, ch, grp, sem = progs[c][k]
        what.append(kind if part == "issue" else kind + " reply")
        if part == "back":
            src.append(ch), dst.append(c), cls.append(0 if kind == "load" else 1), preds.append({ids[(c, k)]})
            continue
        p = set()
        if k >= mc.window:
            p.add(done(c, k - mc.window))
        if k > 0 and progs[c][k - 1][0] == "acquire":
            p.add(done(c, k - 1))
        if kind == "store":
            p |= {ids[(c, g)] + 1 for g in grp}
        if kind == "release":
            p |= {ids[(c, j)] for j in range(k) if progs[c][j][0] in ("store", "release")}
        if kind == "acquire":
            p.add(released[sem])
        src.append(c), dst.append(ch), cls.append(0 if kind == "store" else 1), preds.append(p)
    return src, dst, cls, preds, what


def star(n_cu=1, bc=1, bm=8, Lc=1, Lm=1):
    """Nodes: CUs 0 .. n_cu - 1, channels n_cu (space 0) and n_cu + 1
    (space 1), the router n_cu + 2; every path is leaf -> router -> leaf."""
    hub = n_cu + 2
    edges = [e for v in range(hub) for e in ((v, hub), (hub, v))]
    rp, ci, lid = si._csr(hub + 1, edges)
    m = len(lid)
    bw = np.full(m, 64, np.int32)
    lat = np.full(m, 1, np.int32)
    cap = np.full(m, 4096, np.int32)
    for (u, v), i in lid.items():
        leaf = u if v == hub else v
        lat[i] = Lc if leaf < n_cu else Lm
        if u == leaf:
            bw[i] = bc if leaf < n_cu else bm
    return si.Workload("star", hub + 1, hub, rp, ci, 1, bw, lat, cap, 0, -1, 0)


def prog(rows, n_cu, U, W):
    """rows: (kind, cu, sources, dst_space, dst_line, n_lines) on the star."""
    kind = np.array([r[0] for r in rows], np.int32)
    sptr = np.concatenate([[0], np.cumsum([len(r[2]) for r in rows])]).astype(np.int64)
    srcs = [s for r in rows for s in r[2]]
    return noc.Memcpy(np.array([r[1] for r in rows], np.int32), np.array([s for s, _ in srcs], np.int32),
                      np.array([r[3] for r in rows], np.int32), np.array([a for _, a in srcs], np.int64),
                      np.array([r[4] for r in rows], np.int64), np.array([r[5] for r in rows], np.int64),
                      np.array([n_cu, n_cu + 1], np.int32), 1, U, W, kind, sptr)


def run(oracle_lib, w, mc, check=True):
    return oracle_lib.simulate_workload(noc.memcpy_workload(w, mc), check=check)


def random_program(rng, cus, n_spaces, n_sem_pairs):
    """Copies and reduces on random CUs, plus release/acquire pairs between
    distinct CUs (each semaphore released once, acquired once or twice);
    acquires follow every release of their CU, so no program waits on
    itself."""
    rows = []
    cus = list(cus)
    for _ in range(int(rng.integers(2, 6))):
        k = int(rng.integers(1, 4))
        rows.append((OP_COPY, int(rng.choice(cus)),
                     [(int(rng.integers(0, n_spaces)), int(rng.integers(0, 40))) for _ in range(k)],
                     int(rng.integers(0, n_spaces)), 50 + int(rng.integers(0, 40)), int(rng.integers(0, 6))))
    acq = []
    for q in range(n_sem_pairs):
        a, b = (int(v) for v in rng.choice(cus, 2, replace=False))
        sem = (int(rng.integers(0, n_spaces)), 200 + q)
        rows.append((OP_RELEASE, a, [], sem[0], sem[1], 1))
        acq.append((OP_ACQUIRE, b, [], sem[0], sem[1], 1))
        if rng.integers(0, 2):
            acq.append((OP_ACQUIRE, a if rng.integers(0, 2) else b, [], sem[0], sem[1], 1))
    rows += acq
    # a copy after the acquires on some CUs
    for c in cus:
        if rng.integers(0, 2):
            rows.append((OP_COPY, int(c), [(int(rng.integers(0, n_spaces)), 0)], int(rng.integers(0, n_spaces)),
                         100, int(rng.integers(1, 4))))
    return rows


@pytest.mark.parametrize("seed", range(12))
def test_expansion_matches_model(oracle_lib, seed):
    rng = np.random.default_rng(seed)
    w, lay = noc.gpu_noc(2, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    rows = random_program(rng, lay.cus.reshape(-1)[:5], 2, int(rng.integers(0, 4)))
    mc = noc._prog(rows, lay, int(rng.integers(1, 5)), int(rng.integers(1, 9)))
    src, dst, pptr, pidx, cls = oracle_lib.memcpy_txns(mc, with_class=True)
    ms, md, mcls, mp, what = model(mc)
    assert list(src) == ms and list(dst) == md and list(cls) == mcls
    for x in range(len(src)):
        got = set(pidx[pptr[x]:pptr[x + 1]].tolist())
        if what[x] == "release":
            # the oracle's set is part of the model's; the rest are earlier
            # stores that its members already wait for
            assert got <= mp[x], x
        else:
            assert got == mp[x], x


def test_plain_memcpy_is_a_one_source_copy(oracle_lib):
    w, lay = noc.gpu_noc(2, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    mc = noc.allgather_ops(lay, 2 * 4 * 3, n_wg=4, unroll=2, window=5)
    rows = [(OP_COPY, int(mc.cu[o]), [(int(mc.src_space[o]), int(mc.src_line[o]))], int(mc.dst_space[o]),
             int(mc.dst_line[o]), int(mc.n_lines[o])) for o in range(len(mc.cu))]
    a = oracle_lib.memcpy_txns(mc, with_class=True)
    b = oracle_lib.memcpy_txns(noc._prog(rows, lay, 2, 5), with_class=True)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("n,K,Lc,Lm", [(1, 2, 1, 1), (4, 2, 1, 1), (3, 3, 2, 5), (5, 4, 3, 1)])
def test_reduce_window_one_serialises(oracle_lib, n, K, Lc, Lm):
    # W = 1, U = 1: for each line the K loads (request leg, data leg) and the
    # store follow one another; every leg crosses two links: Lc + Lm + 1.
    w = star(1, Lc=Lc, Lm=Lm)
    mc = prog([(OP_COPY, 0, [(s % 2, 10 * s) for s in range(K)], 1, 100, n)], 1, U=1, W=1)
    r = run(oracle_lib, w, mc)
    leg = Lc + Lm + 1
    per = 2 * K + 1
    want = [leg * (per * j + i + 1) for j in range(n) for i in range(per)]
    # line ids follow program order here (one CU)
    assert list(r.completion) == want
    assert r.makespan == per * leg * n


@pytest.mark.parametrize("Lc,Lm", [(1, 1), (2, 3), (4, 1)])
def test_release_acquire_handoff(oracle_lib, Lc, Lm):
    # CU 0 copies one line and releases; CU 1 acquires, then copies the line
    # on.  W = 1 on both, so every request waits for the one before; the
    # acquire's request waits for the release.  Ids (step-major): k = 0: CU 0
    # load 0/1, CU 1 acquire 2/3; k = 1: CU 0 store 4, CU 1 load 5/6; k = 2:
    # CU 0 release 7, CU 1 store 8.
    w = star(2, Lc=Lc, Lm=Lm)
    rows = [(OP_COPY, 0, [(0, 0)], 1, 0, 1), (OP_RELEASE, 0, [], 1, 9, 1),
            (OP_ACQUIRE, 1, [], 1, 9, 1), (OP_COPY, 1, [(1, 0)], 0, 5, 1)]
    mc = prog(rows, 2, U=1, W=1)
    r = run(oracle_lib, w, mc)
    leg = Lc + Lm + 1
    want = {0: 1, 1: 2, 4: 3, 7: 4, 2: 5, 3: 6, 5: 7, 6: 8, 8: 9}
    assert list(r.completion) == [leg * want[x] for x in range(9)]
    assert r.makespan == 9 * leg


def test_acquire_before_own_release_deadlocks(oracle_lib):
    w = star(1)
    rows = [(OP_ACQUIRE, 0, [], 0, 3, 1), (OP_RELEASE, 0, [], 0, 3, 1)]
    r = run(oracle_lib, w, prog(rows, 1, U=1, W=4), check=False)
    assert r.status_name == "DEADLOCK"


def test_bad_semaphores_rejected(oracle_lib):
    bad = [
        [(OP_RELEASE, 0, [], 0, 3, 1), (OP_RELEASE, 1, [], 0, 3, 1)],      # released twice
        [(OP_ACQUIRE, 0, [], 0, 3, 1)],                                    # never released
        [(OP_RELEASE, 0, [(0, 1)], 0, 3, 1)],                              # a release with a source
        [(OP_RELEASE, 0, [], 0, 3, 2)],                                    # more than one line
        [(OP_COPY, 0, [], 0, 3, 2)],                                       # a copy without a source
        [(7, 0, [], 0, 3, 1)],                                             # unknown kind
    ]
    for rows in bad:
        with pytest.raises(ValueError):
            from oracle import memcpy_txns
            memcpy_txns(prog(rows, 2, U=1, W=1))


def max_plus(w, src, dst, preds, hub):
    """Completion times when only the injection streams can hold a line back
    (every later link has spare bandwidth and buffer): stream (src, first
    link) admits in id order, at most b per cycle, once released; a line then
    needs the latencies of its path plus one."""
    rp, ci = w.row_ptr, w.col_idx
    link = {(u, int(ci[l])): l for u in range(w.n_nodes) for l in range(rp[u], rp[u + 1])}
    T = len(src)
    comp = [0] * T
    for _ in range(T + 2):   # an acyclic system settles within T rounds
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
    return None   # a cycle of waits: the lines on it never complete


@pytest.mark.parametrize("seed", range(16))
def test_max_plus_on_star(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    n_cu = int(rng.integers(2, 4))
    w = star(n_cu, bc=int(rng.integers(1, 3)), bm=int(rng.integers(1, 3)), Lc=int(rng.integers(1, 4)),
             Lm=int(rng.integers(1, 5)))
    rows = random_program(rng, range(n_cu), 2, int(rng.integers(1, 4)))
    mc = prog(rows, n_cu, int(rng.integers(1, 5)), int(rng.integers(1, 7)))
    r = run(oracle_lib, w, mc, check=False)
    src, dst, _, preds, _ = model(mc)
    want = max_plus(w, src, dst, preds, n_cu + 2)
    # a channel returns its lines in id order, so an acquire's reply that
    # waits for a late release holds back the channel's later replies; in an
    # unbalanced program that can close a cycle (a deadlock)
    if want is None:
        assert r.status_name == "DEADLOCK"
    else:
        assert r.status_name == "OK" and list(r.completion) == want


@pytest.mark.parametrize("seed", range(8))
def test_stepper_on_tiny_noc(oracle_lib, seed):
    w, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=1, ch_per_router=2, ports_per_router=1,
                         noc=(2, 1, 3), cu_out=(1, 1, 2), mem=(1, 2, 2))
    rng = np.random.default_rng(200 + seed)
    rows = random_program(rng, lay.cus[0], 1, int(rng.integers(1, 3)))
    mc = noc._prog(rows, lay, int(rng.integers(1, 4)), int(rng.integers(1, 6)))
    wm = noc.memcpy_workload(w, mc)
    wm.arb = seed % 2
    r = oracle_lib.simulate_workload(wm, check=False)
    src, dst, _, preds, _ = model(mc)
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, wm.arb, src, dst,
                       [sorted(p) for p in preds], max_cycles=20000)
    assert st[0] == r.status_name
    assert list(r.completion) == [0xFFFFFFFF if v is None else v for v in st[1]]


@pytest.mark.parametrize("get", [True, False])
def test_reducescatter_programs(oracle_lib, get):
    # G = 3 GPUs, 4 workgroups, 2 lines per slice: the expansion follows the
    # model, every line completes, and the counts are those of the program:
    # get: per workgroup 2 lines x (3 loads + 1 store); put: per workgroup
    # and peer 2 x (load + store) + a release, 2 acquires, then 2 x (3 local
    # loads + store).
    w, lay = noc.gpu_noc(3, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1)
    G, n_wg, c = 3, 4, 2
    mc = noc.reducescatter_ops(lay, G * n_wg * c, n_wg=n_wg, unroll=2, window=6, get=get)
    src, dst, pptr, pidx, cls = oracle_lib.memcpy_txns(mc, with_class=True)
    ms, md, mcls, _, _ = model(mc)
    assert list(src) == ms and list(dst) == md and list(cls) == mcls
    per_wg = c * (3 * 2 + 1) if get else (G - 1) * (c * 3 + 1) + (G - 1) * 2 + c * (3 * 2 + 1)
    assert len(src) == G * n_wg * per_wg
    r = run(oracle_lib, w, mc)
    assert r.status_name == "OK" and min(r.completion) > 0
    # every workgroup's last store lands in its own GPU's memory
    chans = {g: set(lay.channels[g].tolist()) for g in range(G)}
    for g in range(G):
        for wg in range(n_wg):
            cu = noc.wg_cu(lay, g, wg, n_wg)
            last = max(x for x in range(len(src)) if src[x] == cu)
            assert dst[last] in chans[g] and cls[last] == 0
