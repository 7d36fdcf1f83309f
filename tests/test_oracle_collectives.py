"""Pins of the oracle's further collectives: ring and direct all-gather and
reduce-scatter, recursive halving-doubling (RHD) all-reduce and double
binary tree (DBT) all-reduce -- the textbook algorithms listed in Sec. 1 and
2.2 -- in both dependency modes.

The oracle decodes every transaction id arithmetically.  Here each algorithm
is written once more, differently: as a sequential program over participants
and buffer positions that records every message (sender, receiver, the
positions it carries) and, per position, which earlier arrivals at the
sender it builds on.  Against that model:

* every oracle transaction has the model's sender, receiver and id, and each
  of its predecessors is an earlier arrival of the same position at the
  sender (so no dependency is invented);
* the oracle's dependencies are sufficient: propagating contribution sets
  through them leaves every participant with everything the collective
  promises (all-reduce: every contribution everywhere; reduce-scatter: every
  contribution at the owner; all-gather: every owner's data everywhere);
* on a full mesh with buffers of at least b(L+1) lines (dedicated one-hop
  links, never full) every injection stream follows the max-plus recursion
  admit(k) = max(rel(k), admit(k-1), admit(k-b) + 1), completion = admit +
  L + 1, with rel taken over the model's own dependencies; the oracle's
  simulation must match it line for line;
* special cases: RHD on two participants is the direct all-reduce, a
  hand-derived DBT makespan, ring all-gather's closed form;
* brute force against the literal stepper on small tori.
"""
from __future__ import annotations

from collections import defaultdict

import numpy as np
import pytest

import sim_inputs as si
from tests.ref_stepper import step_simulate


# ------------------------------------------------------------- the model

class Program:
    """Messages of a collective in program order.  send() builds on the
    arrivals recorded so far; a step's arrivals become visible at commit()."""

    def __init__(self):
        self.msgs = []          # [key, src, dst, positions, preds per line]
        self.arrived = defaultdict(list)
        self.pending = []

    def send(self, key, src, dst, positions, build_on=True):
        preds = [list(self.arrived[(src, q)]) if build_on else [] for q in positions]
        self.msgs.append([key, src, dst, list(positions), preds])
        self.pending.append(len(self.msgs) - 1)

    def commit(self):
        for mi in self.pending:
            _, _, dst, pos, _ = self.msgs[mi]
            for li, q in enumerate(pos):
                self.arrived[(dst, q)].append((mi, li))
        self.pending = []

    def finish(self):
        """Order by key (the id layout), number the lines, resolve preds."""
        self.commit()
        order = sorted(range(len(self.msgs)), key=lambda mi: self.msgs[mi][0])
        first = {}
        x = 0
        for mi in order:
            first[mi] = x
            x += len(self.msgs[mi][3])
        T = x
        src, dst, pos, preds, msg = [0] * T, [0] * T, [0] * T, [None] * T, [0] * T
        for rank, mi in enumerate(order):
            _, s, d, ps, pr = self.msgs[mi]
            for li, q in enumerate(ps):
                y = first[mi] + li
                src[y], dst[y], pos[y], msg[y] = s, d, q, rank
                preds[y] = sorted(first[m2] + l2 for m2, l2 in pr[li])
        return src, dst, pos, preds, msg


def ring(p, N, steps):
    C = N // p
    P = Program()
    for s in range(steps):
        for i in range(p):
            c = (i - s) % p if s < p - 1 else (i + 1 - (s - p + 1)) % p
            P.send((s, i), i, (i + 1) % p, range(c * C, (c + 1) * C))
        P.commit()
    return P.finish()


def direct(p, N, phases):
    """phases: 'rs' (i sends chunk i+k to its owner), 'ag' (i sends chunk i)."""
    C = N // p
    P = Program()
    for ph, kind in enumerate(phases):
        for k in range(1, p):
            for i in range(p):
                c = (i + k) % p if kind == "rs" else i
                P.send((ph, k, i), i, (i + k) % p, range(c * C, (c + 1) * C))
        P.commit()
    return P.finish()


def rhd(p, N):
    K = p.bit_length() - 1
    C = N // p
    P = Program()
    blocks = {i: (0, N) for i in range(p)}            # the range each participant reduces
    for j in range(K):
        d = p >> (j + 1)
        new = {}
        for i in range(p):
            lo, hi = blocks[i]
            mid = (lo + hi) // 2
            keep_upper = bool(i & d)
            new[i] = (mid, hi) if keep_upper else (lo, mid)
            send = (lo, mid) if keep_upper else (mid, hi)
            P.send((0, j, i), i, i ^ d, range(*send))
        P.commit()
        blocks = new
    assert all(blocks[i] == (i * C, (i + 1) * C) for i in range(p))
    for j in range(K):
        d = 1 << j
        for i in range(p):
            lo, hi = blocks[i]
            P.send((1, j, i), i, i ^ d, range(lo, hi))
        P.commit()
        blocks = {i: (min(blocks[i][0], blocks[i ^ d][0]), max(blocks[i][1], blocks[i ^ d][1])) for i in range(p)}
    return P.finish()


def tree_parent(u, p):
    """Parent position in the in-order binary tree over positions 0..p-1."""
    if u == 0:
        return None
    low = u & -u
    up = (u - low) | (2 * low)
    return up if up < p else u - low


def dbt(p, N):
    H = N // 2
    P = Program()
    for t in range(2):
        part = (lambda u: u) if t == 0 else (lambda u: p - 1 - u)   # position -> participant
        par = {u: tree_parent(u, p) for u in range(p)}
        kids = defaultdict(list)
        for u in range(1, p):
            kids[par[u]].append(u)
        edge = (lambda c: c - 1) if t == 0 else (lambda c: c)
        half = range(t * H, (t + 1) * H)

        def post(u):
            for v in kids[u]:
                post(v)
            if u != 0:
                P.send((0, t, edge(part(u))), part(u), part(par[u]), half)
                P.commit()

        def pre(u):
            for v in kids[u]:
                P.send((1, t, edge(part(v))), part(u), part(v), half)
            P.commit()
            for v in kids[u]:
                pre(v)

        post(0)
        pre(0)
    return P.finish()


COLLS = {
    si.COLL_RING_ALLREDUCE: lambda p, N: ring(p, N, 2 * p - 2),
    si.COLL_RING_ALLGATHER: lambda p, N: ring(p, N, p - 1),
    si.COLL_RING_REDUCESCATTER: lambda p, N: ring(p, N, p - 1),
    si.COLL_DIRECT_ALLREDUCE: lambda p, N: direct(p, N, ["rs", "ag"]),
    si.COLL_DIRECT_ALLGATHER: lambda p, N: direct(p, N, ["ag"]),
    si.COLL_DIRECT_REDUCESCATTER: lambda p, N: direct(p, N, ["rs"]),
    si.COLL_RHD_ALLREDUCE: rhd,
    si.COLL_DBT_ALLREDUCE: dbt,
}
KIND = {si.COLL_RING_ALLREDUCE: "ar", si.COLL_DIRECT_ALLREDUCE: "ar", si.COLL_RHD_ALLREDUCE: "ar",
        si.COLL_DBT_ALLREDUCE: "ar", si.COLL_RING_ALLGATHER: "ag", si.COLL_DIRECT_ALLGATHER: "ag",
        si.COLL_RING_REDUCESCATTER: "rs", si.COLL_DIRECT_REDUCESCATTER: "rs"}
NEW = [si.COLL_RING_ALLGATHER, si.COLL_RING_REDUCESCATTER, si.COLL_DIRECT_ALLGATHER,
       si.COLL_DIRECT_REDUCESCATTER, si.COLL_RHD_ALLREDUCE, si.COLL_DBT_ALLREDUCE]
CASES = [(c, p, N) for c in NEW for p, N in [(2, 8), (4, 8), (4, 16), (8, 16), (3, 6), (5, 10), (6, 12)]
         if not (c == si.COLL_RHD_ALLREDUCE and p & (p - 1))]


def decode_all(oracle_lib, coll, p, N, order=None, dep=0):
    rc, _, _, _, T = oracle_lib.txn(coll, 128 * N, 0, p, 0, order, dep)
    assert rc == 0
    return T, [oracle_lib.txn(coll, 128 * N, 0, p, x, order, dep)[1:4] for x in range(T)]


# ------------------------------------------------------------- decoder

def topo_order(preds):
    """Ids in an order where predecessors come first (DBT's edge-major ids
    are not)."""
    T = len(preds)
    indeg = [len(p) for p in preds]
    succ = defaultdict(list)
    for x, pr in enumerate(preds):
        for q in pr:
            succ[q].append(x)
    ready = [x for x in range(T) if indeg[x] == 0]
    out = []
    while ready:
        x = ready.pop()
        out.append(x)
        for y in succ[x]:
            indeg[y] -= 1
            if indeg[y] == 0:
                ready.append(y)
    assert len(out) == T, "predecessor cycle"
    return out


@pytest.mark.parametrize("coll,p,N", CASES)
def test_decoder_matches_model(oracle_lib, coll, p, N):
    src, dst, pos, preds, _ = COLLS[coll](p, N)
    T, dec = decode_all(oracle_lib, coll, p, N)
    assert T == len(src)
    for x in range(T):
        s, d, pr = dec[x]
        assert (s, d) == (src[x], dst[x]), x
        assert set(pr) <= set(preds[x]), (x, pr, preds[x])
        for q in pr:
            assert dst[q] == s and pos[q] == pos[x]


@pytest.mark.parametrize("coll,p,N", CASES + [(si.COLL_RING_ALLREDUCE, 5, 10), (si.COLL_DIRECT_ALLREDUCE, 4, 8)])
def test_dependencies_deliver_everything(oracle_lib, coll, p, N):
    src, dst, pos, _, _ = COLLS[coll](p, N)
    T, dec = decode_all(oracle_lib, coll, p, N)
    kind = KIND[coll]
    C = N // p
    own = (lambda i, q: q // C == i) if kind == "ag" else (lambda i, q: True)
    carried = [None] * T
    have = [[({i} if own(i, q) else set()) for q in range(N)] for i in range(p)]
    for x in topo_order([d[2] for d in dec]):
        s, d, pr = dec[x]
        c = {s} if own(s, pos[x]) else set()
        for q in pr:
            c |= carried[q]
        if kind == "ag":
            assert c, f"line {x} sent before its sender holds it"
        carried[x] = c
        have[d][pos[x]] |= c
    everyone = set(range(p))
    for q in range(N):
        if kind == "ar":
            assert all(have[i][q] == everyone for i in range(p)), q
        elif kind == "ag":
            assert all(q // C in have[i][q] for i in range(p)), q
        else:
            assert any(have[i][q] == everyone for i in range(p)), q


def test_rhd_rejects_non_power_of_two(oracle_lib):
    assert oracle_lib.txn(si.COLL_RHD_ALLREDUCE, 128 * 12, 0, 6, 0)[0] == 1
    assert oracle_lib.txn(si.COLL_RHD_ALLREDUCE, 128 * 12, 0, 8, 0)[0] == 4   # 12 lines over 8
    assert oracle_lib.txn(si.COLL_DBT_ALLREDUCE, 128 * 7, 0, 4, 0)[0] == 4    # odd buffer


def test_dbt_trees_are_complementary():
    # The tree over positions is a spanning tree rooted at 0 with at most two
    # children per node; its leaves are the odd positions, so for even p the
    # mirrored tree's leaves are the even participants and no participant is
    # a leaf in both trees.
    for p in range(2, 70):
        kids = defaultdict(int)
        for u in range(1, p):
            seen, v = set(), u
            while v != 0:
                assert v not in seen
                seen.add(v)
                v = tree_parent(v, p)
            kids[tree_parent(u, p)] += 1
        assert max(kids.values()) <= 2
        leaves = set(range(p)) - set(kids)
        assert leaves == set(range(1, p, 2)), p
        if p % 2 == 0:
            assert leaves.isdisjoint({p - 1 - u for u in leaves})


# ------------------------------------------------------------- timing

def max_plus(src, dst, preds, b, L, msg=None):
    """Completion times on dedicated one-hop links that never fill.  Each
    (sender, receiver) stream injects in id order; the recursion is iterated
    to its least fixed point (ids need not be in dependency order)."""
    T = len(src)
    msg_lines = defaultdict(list)
    if msg is not None:
        for x in range(T):
            msg_lines[msg[x]].append(x)
    stream_of = defaultdict(list)
    for x in range(T):
        stream_of[(src[x], dst[x])].append(x)
    comp = [0] * T
    while True:
        new = [0] * T
        for ids in stream_of.values():
            a = []
            for x in ids:
                if msg is None:
                    rel = max((comp[q] for q in preds[x]), default=0)
                else:
                    # per message: wait for every line of each message feeding it
                    feeders = {msg[q] for y in msg_lines[msg[x]] for q in preds[y]}
                    rel = max((comp[y] for m in feeders for y in msg_lines[m]), default=0)
                v = rel
                if a:
                    v = max(v, a[-1])
                if len(a) >= b:
                    v = max(v, a[-b] + 1)
                a.append(v)
                new[x] = v + L + 1
        if new == comp:
            return comp
        comp = new


@pytest.mark.parametrize("coll", NEW + [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE])
@pytest.mark.parametrize("p,C,b,L", [(2, 5, 1, 3), (4, 4, 1, 6), (4, 6, 2, 2), (8, 3, 1, 9), (6, 4, 3, 5), (5, 7, 2, 1)])
@pytest.mark.parametrize("dep", [0, 1])
def test_full_mesh_max_plus(oracle_lib, coll, p, C, b, L, dep):
    if coll == si.COLL_RHD_ALLREDUCE and p & (p - 1):
        pytest.skip("RHD needs a power of two")
    N = C * p * (2 if coll == si.COLL_DBT_ALLREDUCE and C * p % 2 else 1)
    src, dst, _, preds, msg = COLLS[coll](p, N)
    w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=coll, nbytes=128 * N)
    w.dep = dep
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.status_name == "OK"
    want = max_plus(src, dst, preds, b, L, msg if dep else None)
    assert list(r.completion) == want
    assert r.makespan == max(want)


@pytest.mark.parametrize("p,C,b,L", [(2, 5, 1, 3), (4, 6, 2, 9), (8, 16, 1, 50), (6, 12, 3, 2)])
def test_ring_allgather_closed_form(oracle_lib, p, C, b, L):
    # The first p-1 steps of the ring all-reduce: comp(s, i, j) = sM +
    # floor(j/b) + L + 1, M = max(C/b, L+1); makespan (p-2) M + C/b + L.
    for coll in (si.COLL_RING_ALLGATHER, si.COLL_RING_REDUCESCATTER):
        w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=coll, nbytes=128 * C * p)
        r = oracle_lib.simulate_workload(w, check=True)
        Cp, M = C // b, max(C // b, L + 1)
        ids = np.arange(len(r.completion))
        assert np.array_equal(r.completion, (ids // (C * p)) * M + (ids % C) // b + L + 1)
        assert r.makespan == (p - 2) * M + Cp + L


def test_rhd_on_two_is_direct(oracle_lib):
    # With two participants recursive halving-doubling is one exchange of
    # halves and one exchange of the reduced halves: the direct all-reduce,
    # id for id, on any topology.
    for seed in range(4):
        w = si.torus2d(2, 1, n_scenarios=1, seed=60 + seed, bws=(1, 2), lat_lo=1, lat_hi=9, depths=(1, 3, 8),
                       nbytes=128 * 2 * 9, coll=si.COLL_DIRECT_ALLREDUCE, arb=seed % 2)
        a = oracle_lib.simulate_workload(w, check=True)
        w.coll = si.COLL_RHD_ALLREDUCE
        b = oracle_lib.simulate_workload(w, check=True)
        assert a.status_name == b.status_name == "OK"
        assert np.array_equal(a.completion, b.completion) and a.makespan == b.makespan


@pytest.mark.parametrize("H,L", [(4, 10), (20, 3), (1, 1), (7, 7)])
def test_dbt_two_participants_by_hand(oracle_lib, H, L):
    # Tree 0: 0 is the root, 1 below it; tree 1 the mirror.  Link 1->0 carries
    # tree 0's reduce (j + L + 1) then tree 1's broadcast; link 0->1 tree 1's
    # reduce then tree 0's broadcast, which waits for the reduce line j:
    # admit = max(j + L + 1, H + j), completion admit + L + 1 (b = 1).
    w = si.full_mesh(2, b=1, L=L, cap=L + 1, coll=si.COLL_DBT_ALLREDUCE, nbytes=128 * 2 * H)
    r = oracle_lib.simulate_workload(w, check=True)
    j = np.arange(H)
    red = j + L + 1
    bc = np.maximum(j + L + 1, H + j) + L + 1
    assert np.array_equal(r.completion, np.concatenate([red, red, bc, bc]))
    assert r.makespan == max(H - 1 + L + 1, 2 * H - 1) + L + 1


# ------------------------------------------------------------- brute force

def explicit(oracle_lib, w):
    T, dec = decode_all(oracle_lib, w.coll, w.n_endpoints, w.bytes // 128, w.order, w.dep)
    if w.dep == 0:
        return [d[0] for d in dec], [d[1] for d in dec], [d[2] for d in dec]
    # chunk mode: a predecessor -1-m is every line of message m; messages are
    # the id ranges over which the (sender, receiver, predecessor set) is fixed
    # -- recovered here from the model of the same collective
    _, _, _, _, msg = COLLS[w.coll](w.n_endpoints, w.bytes // 128)
    lines = defaultdict(list)
    for x, m in enumerate(msg):
        lines[m].append(x)
    preds = [[y for q in d[2] for y in lines[-1 - q]] for d in dec]
    return [d[0] for d in dec], [d[1] for d in dec], preds


@pytest.mark.parametrize("coll", NEW)
@pytest.mark.parametrize("dep", [0, 1])
@pytest.mark.parametrize("seed", range(2))
def test_brute_force_on_small_torus(oracle_lib, coll, dep, seed):
    X, Y = (2, 2) if coll == si.COLL_RHD_ALLREDUCE else [(3, 2), (2, 2)][seed]
    p = X * Y
    w = si.torus2d(X, Y, n_scenarios=1, seed=500 + seed + 7 * coll, bws=(1, 2, 3), lat_lo=1, lat_hi=5,
                   depths=(1, 2, 4, 7), nbytes=128 * p * 2, coll=coll, arb=seed % 2)
    w.dep = dep
    got = oracle_lib.simulate_workload(w, check=True)
    src, dst, preds = explicit(oracle_lib, w)
    st = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb, src, dst, preds,
                       max_cycles=50000)
    assert st[0] == got.status_name == "OK"
    assert list(got.completion) == st[1]


def test_order_permutes_participants(oracle_lib):
    # With a participant order every participant index i is endpoint order[i].
    p, N = 4, 8
    order = [2, 0, 3, 1]
    for coll in NEW:
        src, dst, _, _, _ = COLLS[coll](p, N)
        T, dec = decode_all(oracle_lib, coll, p, N, order)
        assert [d[0] for d in dec] == [order[s] for s in src]
        assert [d[1] for d in dec] == [order[d] for d in dst]


def test_gray_order_makes_rhd_partners_neighbours(oracle_lib):
    # The 4x4 torus is the 4-cube: in Gray-code participant order every
    # halving-doubling partner (one bit apart) is one hop away, so no route
    # has a second hop and no cyclic buffer dependency can form.
    w = si.config("C5_rhd")
    rc, pp, _ = oracle_lib.paths(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx)
    assert rc == 0
    E = w.n_endpoints
    for i in range(E):
        for b in range(4):
            s, d = int(w.order[i]), int(w.order[i ^ (1 << b)])
            assert pp[s * E + d + 1] - pp[s * E + d] == 1
    # in rank order some partners are two hops apart, and the same sweep
    # deadlocks (cyclic buffer dependencies around the torus rings)
    w2 = si.take_scenarios(si.config("C5"), [0])
    w2.coll = si.COLL_RHD_ALLREDUCE
    assert oracle_lib.simulate_workload(w2).status_name == "DEADLOCK"
