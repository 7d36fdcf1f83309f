"""Pins of the CPU oracle against facts it does not define itself.

* published hash / PRNG test vectors (MurmurHash3, SplitMix64);
* closed forms of the alpha-beta regime (contention-free pipelining,
  first-hop bottleneck, bandwidth-delay throttling, ring and direct
  all-reduce), exact per line;
* a max-plus (Lindley-type) recursion for an in-order stream with release
  times, computed independently in the test;
* the collective expansions checked semantically: every endpoint ends with
  every contribution of every buffer line (all-reduce) / every pair gets its
  lines (all-to-all), counts per flow;
* routing: minimality against an independent BFS, fat-tree path lengths,
  per-link line counts at full C4 size;
* invariants on scaled workloads (oracle check mode);
* brute force: the literal Python stepper on random tiny graphs and DAGs;
* error paths: deadlock, guard overrun, unreachable pair, bad sizes.
"""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from tests.ref_stepper import hop_distances, step_simulate


# ------------------------------------------------------------------ vectors

def test_fmix32_published_vectors(oracle_lib):
    # MurmurHash3_x86_32 of the empty input is fmix32(seed): published
    # verification values for seeds 1 and 0xffffffff.
    assert oracle_lib.fmix32(1) == 0x514E28B7
    assert oracle_lib.fmix32(0xFFFFFFFF) == 0x81F16F39
    assert oracle_lib.fmix32(0) == 0


def test_splitmix64_published_vectors():
    g = si.splitmix64(0)
    assert [next(g) for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


# ------------------------------------------------------------------ helpers

def chain(h, b, L, cap):
    """Endpoint 0 -> h-1 switches -> endpoint 1, with return links."""
    n = h + 1
    # node ids: 0 (src endpoint), 1 (dst endpoint), 2.. switches
    seq = [0] + list(range(2, 2 + h - 1)) + [1]
    edges = set()
    for a, c in zip(seq, seq[1:]):
        edges.add((a, c))
        edges.add((c, a))
    edges = sorted(edges)
    row_ptr = np.zeros(n + 1, np.int32)
    for u, _ in edges:
        row_ptr[u + 1] += 1
    row_ptr = np.cumsum(row_ptr).astype(np.int32)
    col_idx = np.array([v for _, v in edges], np.int32)
    m = len(edges)
    bws = np.full(m, b, np.int32) if np.isscalar(b) else None
    return n, row_ptr, col_idx, edges, seq, bws, np.full(m, L, np.int32), np.full(m, cap, np.int32)


def sim_custom(oracle_lib, n, E, row_ptr, col_idx, bw, lat, cap, arb, src, dst, preds, **kw):
    pptr = np.zeros(len(src) + 1, np.int64)
    for i, p in enumerate(preds):
        pptr[i + 1] = pptr[i] + len(p)
    pidx = np.array([q for p in preds for q in p], np.int64)
    return oracle_lib.simulate(n, E, row_ptr, col_idx, bw, lat, cap, arb,
                               txns=(np.array(src), np.array(dst), pptr, pidx), **kw)


# ------------------------------------------------------------------ closed forms

@pytest.mark.parametrize("h,b,L,nlines", [(1, 1, 1, 5), (1, 1, 7, 40), (3, 1, 4, 33), (2, 2, 5, 41),
                                           (4, 3, 2, 50), (5, 4, 9, 97)])
def test_contention_free_pipeline(oracle_lib, h, b, L, nlines):
    # n lines over h hops with uniform b, L and cap >= b(L+1):
    # comp(k) = floor(k/b) + h*L + 1, so the last is h*L + ceil(n/b).
    n, rp, ci, edges, seq, bws, lat, cap = chain(h, b, L, b * (L + 1))
    r = sim_custom(oracle_lib, n, 2, rp, ci, bws, lat, cap, 0, [0] * nlines, [1] * nlines,
                   [[] for _ in range(nlines)], check=True)
    assert r.status_name == "OK"
    k = np.arange(nlines)
    assert np.array_equal(r.completion, k // b + h * L + 1)
    assert r.makespan == h * L + -(-nlines // b)


def test_first_hop_bottleneck(oracle_lib):
    # b_1 <= b_i and cap_i >= b_i(L_i+1): comp(k) = floor(k/b_1) + sum L + 1.
    h = 4
    n, rp, ci, edges, seq, _, _, _ = chain(h, 1, 1, 1)
    m = len(edges)
    bw = np.zeros(m, np.int32)
    lat = np.zeros(m, np.int32)
    fwd = list(zip(seq, seq[1:]))
    Ls = [3, 7, 2, 5]
    bs = [2, 3, 5, 2]
    for i, e in enumerate(edges):
        if e in fwd:
            j = fwd.index(e)
            bw[i], lat[i] = bs[j], Ls[j]
        else:
            bw[i], lat[i] = 1, 1
    cap = (bw * (lat + 1)).astype(np.int32)
    N = 77
    r = sim_custom(oracle_lib, n, 2, rp, ci, bw, lat, cap, 0, [0] * N, [1] * N, [[] for _ in range(N)],
                   check=True)
    k = np.arange(N)
    assert np.array_equal(r.completion, k // 2 + sum(Ls) + 1)


@pytest.mark.parametrize("b,L,cap", [(1, 9, 4), (2, 6, 8), (3, 10, 12), (2, 3, 8), (1, 1, 2)])
def test_bandwidth_delay_throttle(oracle_lib, b, L, cap):
    # One hop, b | cap, cap <= b(L+1): lines enter in bursts of cap, then wait
    # for the burst to drain: admit(k) = floor(k/cap)(L+1) + floor((k mod cap)/b).
    n, rp, ci, edges, seq, bws, lat, capa = chain(1, b, L, cap)
    N = 53
    r = sim_custom(oracle_lib, n, 2, rp, ci, bws, lat, capa, 0, [0] * N, [1] * N, [[] for _ in range(N)],
                   check=True)
    k = np.arange(N)
    admit = (k // cap) * (L + 1) + (k % cap) // b
    assert np.array_equal(r.completion, admit + L + 1)


@pytest.mark.parametrize("p,C,b,L", [(2, 5, 1, 3), (3, 8, 1, 2), (4, 6, 2, 9), (5, 4, 1, 10), (8, 16, 1, 50),
                                     (6, 12, 3, 2)])
def test_ring_allreduce_closed_form(oracle_lib, p, C, b, L):
    # Dedicated one-hop ring links (full mesh), uniform b and L, cap >= b(L+1):
    # comp(s, i, j) = s*M + floor(j/b) + L + 1 with C' = C/b, M = max(C', L+1);
    # makespan (2p-3) M + C' + L; every ring link carries 2(p-1) C lines.
    w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=si.COLL_RING_ALLREDUCE, nbytes=128 * C * p)
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.status_name == "OK"
    Cp = C // b
    M = max(Cp, L + 1)
    ids = np.arange(len(r.completion))
    j = ids % C
    s = ids // (C * p)
    assert np.array_equal(r.completion, s * M + j // b + L + 1)
    assert r.makespan == (2 * p - 3) * M + Cp + L
    ring = sorted(r.tx_lines)[-p:]
    assert all(v == 2 * (p - 1) * C for v in ring) and sum(r.tx_lines) == 2 * (p - 1) * C * p


@pytest.mark.parametrize("p,C,b,L", [(2, 4, 1, 3), (3, 6, 1, 4), (4, 128, 1, 10), (4, 8, 2, 20), (5, 10, 1, 2)])
def test_direct_allreduce_closed_form(oracle_lib, p, C, b, L):
    # Reduce-scatter lines: comp = floor(j/b) + L + 1; all-gather lines:
    # comp = M + floor(j/b) + L + 1, M = max(C/b, L+1); makespan M + C/b + L.
    w = si.full_mesh(p, b=b, L=L, cap=b * (L + 1), coll=si.COLL_DIRECT_ALLREDUCE, nbytes=128 * C * p)
    r = oracle_lib.simulate_workload(w, check=True)
    Cp = C // b
    M = max(Cp, L + 1)
    ids = np.arange(len(r.completion))
    j = ids % C
    ph = ids // (C * p * (p - 1))
    assert np.array_equal(r.completion, ph * M + j // b + L + 1)
    assert r.makespan == M + Cp + L
    assert set(r.tx_lines.tolist()) == {2 * C}


def test_c1_c2_full_size(oracle_lib):
    r1 = oracle_lib.simulate_workload(si.config("C1"), check=True)
    assert r1.makespan == 266 and set(r1.tx_lines.tolist()) == {256} and set(r1.busy_cycles.tolist()) == {256}
    r2 = oracle_lib.simulate_workload(si.config("C2"))
    assert r2.makespan == 229426
    assert sorted(set(r2.tx_lines.tolist())) == [0, 229376]
    assert int((r2.tx_lines == 229376).sum()) == 8
    assert np.array_equal(r2.tx_lines, r2.busy_cycles)
    ids = np.arange(len(r2.completion), dtype=np.int64)
    assert np.array_equal(r2.completion, 16384 * (ids // (16384 * 8)) + ids % 16384 + 51)


def test_release_max_plus_recursion(oracle_lib):
    # Endpoint 0 feeds endpoint 1 over link g (b=3, L=Lg); line x_k from 1 to 2
    # over link f (b=2, L=Lf, cap large) waits for feeder line y_k.  Feeder
    # completions follow the pipeline form a_k = floor(k/3) + Lg + 1 and the
    # injected stream obeys admit(k) = max(a_k, admit(k-1), admit(k-2) + 1).
    n, E = 3, 3
    edges = sorted({(0, 1), (1, 0), (1, 2), (2, 1)})
    rp = np.array([0, 1, 3, 4], np.int32)
    ci = np.array([v for _, v in edges], np.int32)
    Lg, Lf = 4, 6
    bw = np.array([3, 1, 2, 1], np.int32)
    lat = np.array([Lg, 1, Lf, 1], np.int32)
    cap = np.array([64, 8, 64, 8], np.int32)
    K = 40
    src = [0] * K + [1] * K
    dst = [1] * K + [2] * K
    preds = [[] for _ in range(K)] + [[k] for k in range(K)]
    r = sim_custom(oracle_lib, n, E, rp, ci, bw, lat, cap, 0, src, dst, preds, check=True)
    a = [k // 3 + Lg + 1 for k in range(K)]
    assert list(r.completion[:K]) == a
    admit = []
    for k in range(K):
        v = a[k]
        if k >= 1:
            v = max(v, admit[k - 1])
        if k >= 2:
            v = max(v, admit[k - 2] + 1)
        admit.append(v)
    assert list(r.completion[K:]) == [v + Lf + 1 for v in admit]


# ------------------------------------------------------------------ expansion

def _buffer_line(coll, x, E, N, M=0):
    """Which buffer line of the all-reduce vector a transaction carries,
    from the textbook algorithms (independent of the oracle)."""
    if coll == si.COLL_RING_ALLREDUCE:
        p, C = E, N // E
        j, q = x % C, x // C
        i, s = q % p, q // p
        chunk = (i - s) % p if s < p - 1 else (i + 1 - (s - p + 1)) % p
        return chunk * C + j
    if coll == si.COLL_DIRECT_ALLREDUCE:
        p, C = E, N // E
        j, q = x % C, x // C
        i = q % p
        q //= p
        k, ph = q % (p - 1) + 1, q // (p - 1)
        return ((i + k) % p if ph == 0 else i) * C + j
    G = E // M
    C1 = N // M
    C2 = C1 // G
    B2 = (M - 1) * G * M * C1
    B3 = B2 + (2 * G - 2) * M * G * C2
    if x < B2:
        j, q = x % C1, x // C1
        r = q % M
        q //= M
        k = q // G + 1
        return ((r + k) % M) * C1 + j
    if x < B3:
        y = x - B2
        j, q = y % C2, y // C2
        d = q % G
        q //= G
        r, s = q % M, q // M
        sub = (d - s) % G if s < G - 1 else (d + 1 - (s - G + 1)) % G
        return r * C1 + sub * C2 + j
    y = x - B3
    j, q = y % C1, y // C1
    r = q % M
    return r * C1 + j


@pytest.mark.parametrize("coll,E,N,M", [(si.COLL_RING_ALLREDUCE, 4, 8, 0), (si.COLL_RING_ALLREDUCE, 5, 10, 0),
                                        (si.COLL_DIRECT_ALLREDUCE, 4, 8, 0), (si.COLL_DIRECT_ALLREDUCE, 3, 6, 0),
                                        (si.COLL_HIER_ALLREDUCE, 6, 12, 3), (si.COLL_HIER_ALLREDUCE, 8, 16, 4),
                                        (si.COLL_HIER_ALLREDUCE, 6, 12, 2)])
def test_allreduce_expansion_reduces_everything(oracle_lib, coll, E, N, M):
    # Each transfer carries its source's contribution plus everything its
    # predecessors carried.  At the end every endpoint must hold, for every
    # buffer line, the contributions of all endpoints, and no transfer may
    # carry a line its sender does not yet hold in reduced-so-far form.
    rc, _, _, _, T = oracle_lib.txn(coll, 128 * N, M, E, 0)
    assert rc == 0
    info = [oracle_lib.txn(coll, 128 * N, M, E, x) for x in range(T)]
    carried = [None] * T
    have = [[{e} for _ in range(N)] for e in range(E)]
    done = set()
    order = []
    pending = set(range(T))
    while pending:  # topological order by predecessors
        ready = sorted(x for x in pending if all(p in done for p in info[x][3]))
        assert ready, "predecessor cycle"
        for x in ready:
            order.append(x)
            done.add(x)
            pending.discard(x)
    for x in order:
        _, s, d, preds, _ = info[x]
        assert s != d
        line = _buffer_line(coll, x, E, N, M)
        c = {s}
        for p in preds:
            assert _buffer_line(coll, p, E, N, M) == line and info[p][2] == s
            c |= carried[p]
        carried[x] = c
        have[d][line] |= c
    for e in range(E):
        for line in range(N):
            assert have[e][line] == set(range(E)), (e, line)


def test_alltoall_expansion_counts(oracle_lib):
    E, C = 5, 3
    rc, _, _, _, T = oracle_lib.txn(si.COLL_ALLTOALL, 128 * C, 0, E, 0)
    assert T == E * (E - 1) * C
    cnt = {}
    for x in range(T):
        _, s, d, preds, _ = oracle_lib.txn(si.COLL_ALLTOALL, 128 * C, 0, E, x)
        assert s != d and preds == []
        cnt[(s, d)] = cnt.get((s, d), 0) + 1
    assert len(cnt) == E * (E - 1) and set(cnt.values()) == {C}


# ------------------------------------------------------------------ routing

def test_routes_minimal_and_valid(oracle_lib):
    rng = np.random.default_rng(7)
    for trial in range(6):
        n, rp, ci, *_ = si.random_graph(rng, 4 + trial, 3, 4)
        E = 4 + trial
        rc, pp, pl = oracle_lib.paths(n, E, rp, ci)
        assert rc == 0
        tail = np.repeat(np.arange(n), np.diff(rp))
        for s in range(E):
            for d in range(E):
                path = pl[pp[s * E + d]:pp[s * E + d + 1]]
                if s == d:
                    assert len(path) == 0
                    continue
                dist = hop_distances(n, list(rp), list(ci), d)
                assert len(path) == dist[s]
                v = s
                for l in path:
                    assert tail[l] == v
                    v = ci[l]
                assert v == d


def test_leaf_spine_ecmp_is_hash_mod_spines(oracle_lib):
    # At a leaf with 4 equal uplinks the spine is byte 0 of fmix32(src<<16|dst) mod 4.
    w = si.config("C3")
    rc, pp, pl = oracle_lib.paths(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx)
    E = w.n_endpoints
    spine0 = E + 8
    for s, d in [(0, 8), (9, 17), (63, 7), (12, 44), (5, 21)]:
        path = pl[pp[s * E + d]:pp[s * E + d + 1]]
        assert len(path) == 4
        spine = w.col_idx[path[1]] - spine0
        assert spine == (oracle_lib.fmix32((s << 16) | d) & 255) % 4


def test_fat_tree_paths_and_line_counts(oracle_lib):
    # k=16: same edge 2 hops, same pod 4, else 6; every host uplink carries
    # 1023*512 lines; total line-hops 3,144,679,424.
    w = si.config("C4")
    E = w.n_endpoints
    rc, pp, pl = oracle_lib.paths(w.n_nodes, E, w.row_ptr, w.col_idx)
    assert rc == 0
    lens = np.diff(pp).reshape(E, E)
    s = np.arange(E)[:, None]
    d = np.arange(E)[None, :]
    want = np.where(s == d, 0, np.where(s // 8 == d // 8, 2, np.where(s // 64 == d // 64, 4, 6)))
    assert np.array_equal(lens, want)
    C = w.bytes // 128
    assert int(lens.sum()) * C == 3_144_679_424
    per_link = np.bincount(pl, minlength=w.n_links) * C
    host_up = [w.row_ptr[h] for h in range(E)]
    assert set(per_link[host_up].tolist()) == {1023 * 512}
    assert int(per_link.sum()) == 3_144_679_424


def test_fat_tree_latency_draws():
    w = si.config("C4")
    lat = w.meta["cable_lat"]
    assert len(lat) == 3072 and lat.min() >= 100 and lat.max() <= 300
    g = si.splitmix64(4)
    assert lat[0] == 100 + next(g) % 201


# ------------------------------------------------------------------ invariants

@pytest.mark.parametrize("name,changes", [
    ("C3", dict(bytes=64 * 128 * 8 * 2)),
    ("C5", dict(bytes=16 * 128 * 6)),
])
def test_invariants_scaled(oracle_lib, name, changes):
    w = si.scaled(si.config(name), **changes)
    for s in range(min(w.n_scenarios, 6)):
        r = oracle_lib.simulate_workload(w, s, check=True)
        assert r.status_name == "OK"


def test_invariants_small_fat_tree(oracle_lib):
    w = si.fat_tree(4, nbytes=128 * 6, lat_lo=2, lat_hi=9, cap=5)
    r = oracle_lib.simulate_workload(w, check=True)
    assert r.status_name == "OK"
    assert int(r.tx_lines.sum()) == r.line_hops


# ------------------------------------------------------------------ brute force

def _random_case(seed, arb):
    rng = np.random.default_rng(seed)
    n_end = int(rng.integers(2, 5))
    n_sw = int(rng.integers(0, 3))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, n_sw, int(rng.integers(0, 4)))
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 13)), max_preds=2)
    preds = [list(pidx[pptr[i]:pptr[i + 1]]) for i in range(len(src))]
    return n, n_end, rp, ci, bw, lat, cap, arb, src, dst, preds, (pptr, pidx)


@pytest.mark.parametrize("seed", range(120))
def test_brute_force_vs_literal_stepper(oracle_lib, seed):
    n, E, rp, ci, bw, lat, cap, arb, src, dst, preds, (pptr, pidx) = _random_case(seed, seed % 2)
    want = step_simulate(n, E, rp, ci, bw, lat, cap, arb, src, dst, preds, max_cycles=5000)
    got = oracle_lib.simulate(n, E, rp, ci, bw, lat, cap, arb, txns=(src, dst, pptr, pidx), check=True)
    assert got.status_name == want[0]
    if want[0] == "OK":
        assert list(got.completion) == want[1]
        assert list(got.tx_lines) == want[2]
        assert list(got.busy_cycles) == want[3]
        assert got.makespan == want[4]


@pytest.mark.parametrize("seed", range(8))
def test_brute_force_collectives_on_small_torus(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    w = si.torus2d(3, 2, n_scenarios=1, seed=seed, bws=(1, 2, 3), lat_lo=1, lat_hi=4, depths=(1, 2, 3, 5),
                   nbytes=128 * 6 * 2, coll=[si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE][seed % 2],
                   arb=seed // 2 % 2)
    rc, _, _, _, T = oracle_lib.txn(w.coll, w.bytes, 0, w.n_endpoints, 0)
    info = [oracle_lib.txn(w.coll, w.bytes, 0, w.n_endpoints, x) for x in range(T)]
    src = [i[1] for i in info]
    dst = [i[2] for i in info]
    preds = [i[3] for i in info]
    want = step_simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb, src, dst,
                         preds, max_cycles=20000)
    got = oracle_lib.simulate_workload(w, check=True)
    assert got.status_name == want[0] == "OK"
    assert list(got.completion) == want[1]
    assert list(got.tx_lines) == want[2] and list(got.busy_cycles) == want[3]
    del rng


# ------------------------------------------------------------------ error paths

def directed_ring3():
    rp = np.array([0, 1, 2, 3], np.int32)
    ci = np.array([1, 2, 0], np.int32)
    one = np.ones(3, np.int32)
    return rp, ci, one


def test_deadlock_on_cyclic_buffers(oracle_lib):
    # Directed 3-ring, cap 1: lines two hops long fill every buffer and wait
    # on each other forever.
    rp, ci, one = directed_ring3()
    src = [0, 1, 2] * 4
    dst = [2, 0, 1] * 4
    preds = [[] for _ in src]
    r = sim_custom(oracle_lib, 3, 3, rp, ci, one, one, one, 0, src, dst, preds)
    want = step_simulate(3, 3, rp, ci, one, one, one, 0, src, dst, preds)
    assert r.status_name == want[0] == "DEADLOCK"


def test_deadlock_on_cyclic_predecessors(oracle_lib):
    rp, ci, one = directed_ring3()
    r = sim_custom(oracle_lib, 3, 3, rp, ci, one, one * 4, one * 4, 0, [0, 1], [1, 2], [[1], [0]])
    assert r.status_name == "DEADLOCK"


def test_max_cycles_guard(oracle_lib):
    w = si.config("C1")
    r = oracle_lib.simulate_workload(w, max_cycles=100)
    assert r.status_name == "MAX_CYCLES"
    r = oracle_lib.simulate_workload(w, max_cycles=265)
    assert r.status_name == "OK"


def test_unreachable_and_size_errors(oracle_lib):
    rp = np.array([0, 1, 1], np.int32)   # 0 -> 1 only
    ci = np.array([1], np.int32)
    one = np.ones(1, np.int32)
    r = sim_custom(oracle_lib, 2, 2, rp, ci, one, one, one, 0, [1], [0], [[]])
    assert r.status_name == "UNREACHABLE"
    w = si.config("C2")
    assert oracle_lib.simulate_workload(si.scaled(w, bytes=128 * 7)).status_name == "SIZE"
    assert oracle_lib.simulate_workload(si.scaled(w, bytes=100)).status_name == "SIZE"
