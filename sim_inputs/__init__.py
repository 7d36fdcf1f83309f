"""Seeded synthetic inputs: topologies, per-link parameters and collective specs.

This module is shared by the GPU path's tests/bench and by the CPU oracle's
tests.  It holds only input generation (graph wiring, seeded parameter draws,
collective descriptors); it performs none of the simulated method's
arithmetic (no routing, no transaction expansion, no timing).

Graphs are directed and stored in CSR form: the out-links of node ``u`` are
``col_idx[row_ptr[u]:row_ptr[u+1]]`` (their head nodes), sorted by head node,
and a link's id is its CSR index.  Endpoints are nodes ``0..E-1``; switches
follow.  Every physical cable is two directed links with equal parameters.

The wiring follows the paper's infrastructure descriptions: full-mesh
scale-up domains, a leaf/spine (two-tier Clos) scale-out fabric and a k-ary
three-tier fat-tree (the ``SingleTierFabric``/``ClosFatTreeFabric`` blueprints
of the InfraGraph section), plus a 2D torus for the batched design sweep.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

LINE_BYTES = 128  # one cache line = one transaction (the paper's wavefront request)

ARB_LOWEST_ID = 0
ARB_ROUND_ROBIN = 1
ARB_FAIR_CLASSES = 2   # flag: control and data messages take turns at every link

COLL_RING_ALLREDUCE = 0
COLL_DIRECT_ALLREDUCE = 1
COLL_HIER_ALLREDUCE = 2
COLL_ALLTOALL = 3
COLL_RING_ALLGATHER = 4
COLL_RING_REDUCESCATTER = 5
COLL_DIRECT_ALLGATHER = 6
COLL_DIRECT_REDUCESCATTER = 7
COLL_RHD_ALLREDUCE = 8      # recursive halving-doubling, power-of-two participants
COLL_DBT_ALLREDUCE = 9      # double binary tree

DEP_LINE = 0   # a step's line waits for the matching line of the step before
DEP_CHUNK = 1  # a step's line waits for the whole chunk of the step before

MASK64 = (1 << 64) - 1


def splitmix64(seed: int):
    """SplitMix64 (Steele, Lea & Flood 2014; Vigna's reference C code).

    Yields an endless stream of 64-bit outputs from a 64-bit state."""
    state = seed & MASK64
    while True:
        state = (state + 0x9E3779B97F4A7C15) & MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        yield z ^ (z >> 31)


@dataclass
class Workload:
    """One simulation input: topology, per-scenario link parameters, collective."""
    name: str
    n_nodes: int
    n_endpoints: int
    row_ptr: np.ndarray          # int32 [n_nodes+1]
    col_idx: np.ndarray          # int32 [m]
    n_scenarios: int
    bw: np.ndarray               # int32 [S*m] lines/cycle
    lat: np.ndarray              # int32 [S*m] cycles
    cap: np.ndarray              # int32 [S*m] lines (in flight + waiting)
    arb: int
    coll: int
    bytes: int                   # per endpoint (all-reduce) or per ordered pair (all-to-all)
    group_size: int = 0          # hierarchical: endpoints per domain
    order: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)
    dep: int = 0                 # 0: per-line step dependencies, 1: per-chunk
    credit: Optional[np.ndarray] = None  # int32 [S*m] credit return delay (None: 1)

    @property
    def n_links(self) -> int:
        return int(self.row_ptr[-1])


def _csr(n: int, edges) -> tuple[np.ndarray, np.ndarray, dict]:
    """Directed edge list -> CSR sorted by (tail, head); returns link-id map."""
    edges = sorted(set(edges))
    row_ptr = np.zeros(n + 1, dtype=np.int32)
    for u, _ in edges:
        row_ptr[u + 1] += 1
    row_ptr = np.cumsum(row_ptr).astype(np.int32)
    col_idx = np.array([v for _, v in edges], dtype=np.int32)
    lid = {e: i for i, e in enumerate(edges)}
    return row_ptr, col_idx, lid


def _both(u, v):
    return [(u, v), (v, u)]


def _uniform(m: int, S: int, b: int, L: int, c: int):
    return (np.full(S * m, b, np.int32), np.full(S * m, L, np.int32),
            np.full(S * m, c, np.int32))


def full_mesh(p: int, *, b=1, L=10, cap=16, coll=COLL_DIRECT_ALLREDUCE,
              nbytes=64 * 1024, arb=ARB_LOWEST_ID, name="full_mesh") -> Workload:
    """p endpoints, every ordered pair joined by a direct link (no switches)."""
    edges = [(u, v) for u in range(p) for v in range(p) if u != v]
    row_ptr, col_idx, _ = _csr(p, edges)
    bw, lat, cp = _uniform(len(edges), 1, b, L, cap)
    return Workload(name, p, p, row_ptr, col_idx, 1, bw, lat, cp, arb, coll, nbytes)


def domains_leaf_spine(G=8, M=8, n_leaf=8, n_spine=4, *, intra=(2, 40, 64),
                       fabric=(1, 200, 64), nbytes=64 << 20,
                       arb=ARB_ROUND_ROBIN, name="domains_leaf_spine") -> Workload:
    """G full-mesh domains of M endpoints; endpoint (d, r) = d*M + r.

    Each endpoint also has a NIC cable to leaf switch ``d mod n_leaf`` (one leaf
    per domain), and every leaf is cabled to every spine.  Node ids: endpoints
    0..G*M-1, leaves next, spines last."""
    E = G * M
    leaf0, spine0 = E, E + n_leaf
    n = E + n_leaf + n_spine
    kinds = {}
    edges = []
    for d in range(G):
        for r in range(M):
            for r2 in range(M):
                if r2 != r:
                    e = (d * M + r, d * M + r2)
                    edges.append(e)
                    kinds[e] = intra
    for d in range(G):
        for r in range(M):
            for e in _both(d * M + r, leaf0 + d % n_leaf):
                edges.append(e)
                kinds[e] = fabric
    for lf in range(n_leaf):
        for s in range(n_spine):
            for e in _both(leaf0 + lf, spine0 + s):
                edges.append(e)
                kinds[e] = fabric
    row_ptr, col_idx, lid = _csr(n, edges)
    m = len(lid)
    bw = np.zeros(m, np.int32)
    lat = np.zeros(m, np.int32)
    cp = np.zeros(m, np.int32)
    for e, i in lid.items():
        bw[i], lat[i], cp[i] = kinds[e]
    return Workload(name, n, E, row_ptr, col_idx, 1, bw, lat, cp, arb,
                    COLL_HIER_ALLREDUCE, nbytes, group_size=M)


def fat_tree(k=16, *, lat_seed=4, lat_lo=100, lat_hi=300, b=1, cap=32,
             nbytes=64 * 1024, arb=ARB_ROUND_ROBIN, coll=COLL_ALLTOALL,
             name="fat_tree") -> Workload:
    """Standard k-ary three-tier fat-tree.

    k pods; each pod has k/2 edge and k/2 aggregation switches; each edge
    switch serves k/2 hosts; (k/2)^2 core switches.  Host (p, e, i) has id
    p*(k/2)^2 + e*(k/2) + i; edge (p, e) = H + p*(k/2) + e; aggregation
    (p, a) = H + k*(k/2) + p*(k/2) + a; core c = H + 2*k*(k/2) + c.
    Aggregation switch a of every pod is cabled to cores a*(k/2) .. a*(k/2)+k/2-1.

    Latencies: one SplitMix64 draw per cable, in order host-edge (ascending
    host), edge-agg (ascending (edge, agg)), agg-core (ascending (agg, core));
    latency = lat_lo + u mod (lat_hi - lat_lo + 1); both directions equal."""
    h = k // 2
    H = k * h * h
    edge0 = H
    agg0 = H + k * h
    core0 = H + 2 * k * h
    n = core0 + h * h
    cables = []
    for p in range(k):
        for e in range(h):
            for i in range(h):
                cables.append((p * h * h + e * h + i, edge0 + p * h + e))
    ea = []
    for p in range(k):
        for e in range(h):
            for a in range(h):
                ea.append((edge0 + p * h + e, agg0 + p * h + a))
    cables += sorted(ea)
    ac = []
    for p in range(k):
        for a in range(h):
            for c in range(a * h, a * h + h):
                ac.append((agg0 + p * h + a, core0 + c))
    cables += sorted(ac)
    rng = splitmix64(lat_seed)
    span = lat_hi - lat_lo + 1
    cable_lat = [lat_lo + next(rng) % span for _ in cables]
    edges = []
    for u, v in cables:
        edges += _both(u, v)
    row_ptr, col_idx, lid = _csr(n, edges)
    m = len(lid)
    lat = np.zeros(m, np.int32)
    for (u, v), L in zip(cables, cable_lat):
        lat[lid[(u, v)]] = L
        lat[lid[(v, u)]] = L
    bw = np.full(m, b, np.int32)
    cp = np.full(m, cap, np.int32)
    return Workload(name, n, H, row_ptr, col_idx, 1, bw, lat, cp, arb, coll,
                    nbytes, meta={"k": k, "cable_lat": np.array(cable_lat)})


def torus2d(X=4, Y=4, *, n_scenarios=4096, seed=5, bws=(1, 2, 4), lat_lo=20,
            lat_hi=200, depths=(16, 32, 64), nbytes=4 << 20,
            arb=ARB_LOWEST_ID, coll=COLL_RING_ALLREDUCE,
            name="torus2d_batched") -> Workload:
    """X*Y 2D torus of endpoints (rank r = X*y + x), every node cabled to its
    four neighbours (+-x, +-y, with wrap-around), repeated over S scenarios.

    Per scenario, three SplitMix64 draws in order give the bandwidth
    ``bws[u mod len]``, the latency ``lat_lo + u mod (lat_hi-lat_lo+1)`` and
    the buffer depth ``depths[u mod len]``, applied to every link of that
    scenario (one design point per scenario)."""
    n = X * Y
    edges = set()
    for y in range(Y):
        for x in range(X):
            u = y * X + x
            for dx, dy in ((1, 0), (-1, 0), (0, 1), (0, -1)):
                v = ((y + dy) % Y) * X + (x + dx) % X
                if v != u:
                    edges.add((u, v))
    row_ptr, col_idx, lid = _csr(n, edges)
    m = len(lid)
    rng = splitmix64(seed)
    span = lat_hi - lat_lo + 1
    bw = np.empty(n_scenarios * m, np.int32)
    lat = np.empty(n_scenarios * m, np.int32)
    cp = np.empty(n_scenarios * m, np.int32)
    for s in range(n_scenarios):
        bw[s * m:(s + 1) * m] = bws[next(rng) % len(bws)]
        lat[s * m:(s + 1) * m] = lat_lo + next(rng) % span
        cp[s * m:(s + 1) * m] = depths[next(rng) % len(depths)]
    return Workload(name, n, n, row_ptr, col_idx, n_scenarios, bw, lat, cp, arb,
                    coll, nbytes, meta={"torus": (X, Y)})


def config(name: str) -> Workload:
    """The five benchmark workloads at full size.

    C1  4-endpoint full mesh, direct all-reduce of 64 KiB, b=1 L=10 cap=16.
    C2  8-endpoint full mesh, ring all-reduce of 16 MiB, b=1 L=50 cap=64.
    C3  8 full-mesh domains of 8 + leaf/spine fabric, hierarchical all-reduce
        of 64 MiB, round-robin arbitration.
    C4  k=16 fat-tree (1024 hosts, 320 switches), all-to-all 64 KiB per pair.
    C5  4096 scenarios of a 4x4 torus, ring all-reduce of 4 MiB, seeded params.
    NOC2_ag is the GPU-as-NoC sweep (see sim_inputs.noc).
    Suffixes change one thing of the workload: "_rhd", "_dbt" and "_ag" the
    collective (recursive halving-doubling or double binary tree all-reduce,
    ring all-gather; same buffer), "_chunk" the dependencies (per chunk, put
    + signal), "_credit" the flow control (credit delay = link latency);
    e.g. "C5_dbt_chunk".
    """
    if name == "NOC2_ag":
        # two generic GPUs (448 nodes each) joined by 32 scale-up switches;
        # put-based all-gather of 2 MiB of output per GPU by 32 workgroups
        # per GPU (unroll 4, 64 outstanding); 1024 scenarios sweep the
        # channel and scale-up cable latencies
        from . import noc
        w, lay = noc.gpu_noc(2)
        w = noc.memcpy_workload(w, noc.allgather_ops(lay, 16384, n_wg=32, unroll=4, window=64),
                                name="NOC2_2gpu_noc_allgather_2MiB_x1024")
        return noc.with_scenarios(w, 1024, seed=2)
    if "_" in name:
        base, mod = name.rsplit("_", 1)
        w = config(base)
        if mod == "chunk":
            return replace(w, dep=DEP_CHUNK, name=w.name + "_chunkdep")
        if mod == "credit":
            # credits travel back over the link: credit delay = link latency
            return replace(w, credit=w.lat.copy(), name=w.name + "_creditlat")
        colls = {"rhd": (COLL_RHD_ALLREDUCE, "rhd_ar"), "dbt": (COLL_DBT_ALLREDUCE, "dbt_ar"),
                 "ag": (COLL_RING_ALLGATHER, "ring_ag")}
        if mod in colls and w.coll in (COLL_RING_ALLREDUCE, COLL_DIRECT_ALLREDUCE):
            coll, tag = colls[mod]
            w = replace(w, coll=coll, name=w.name.replace("ring_ar", tag).replace("direct_ar", tag))
            if mod == "rhd" and w.meta.get("torus"):
                # halving-doubling partners differ in one bit: in Gray-code
                # order each of them is a torus neighbour
                w = replace(w, order=gray_torus_order(*w.meta["torus"]), name=w.name + "_gray")
            return w
        raise KeyError(name)
    if name == "C1":
        return full_mesh(4, b=1, L=10, cap=16, coll=COLL_DIRECT_ALLREDUCE,
                         nbytes=64 * 1024, name="C1_mesh4_direct_ar_64KiB")
    if name == "C2":
        return full_mesh(8, b=1, L=50, cap=64, coll=COLL_RING_ALLREDUCE,
                         nbytes=16 << 20, name="C2_mesh8_ring_ar_16MiB")
    if name == "C3":
        return domains_leaf_spine(name="C3_8x8mesh_leafspine_hier_ar_64MiB")
    if name == "C4":
        return fat_tree(16, name="C4_fattree16_alltoall_64KiB")
    if name == "C5":
        return torus2d(name="C5_4096x_torus4x4_ring_ar_4MiB")
    raise KeyError(name)


def gray_torus_order(X: int, Y: int) -> np.ndarray:
    """Participant order for an X x Y torus (X, Y powers of two): participant
    i = (high bits hy, low bits hx) sits at ring positions (gray(hx),
    gray(hy)), gray(v) = v ^ (v >> 1), i.e. at rank X * y + x with x, y the
    positions whose Gray codes are hx, hy.  Participants that differ in one
    bit are then torus neighbours when X, Y <= 4."""
    bx = X.bit_length() - 1
    inv = lambda n: {v ^ (v >> 1): v for v in range(n)}  # Gray code -> position
    ix, iy = inv(X), inv(Y)
    order = np.zeros(X * Y, np.int32)
    for i in range(X * Y):
        hx, hy = i & (X - 1), i >> bx
        order[i] = X * iy[hy] + ix[hx]
    return order


def scaled(w: Workload, **changes) -> Workload:
    """Copy of a workload with fields replaced (e.g. a smaller message)."""
    return replace(w, **changes)


def take_scenarios(w: Workload, idx) -> Workload:
    """Sub-batch of a batched workload (scenario parameters kept verbatim)."""
    idx = np.asarray(idx, dtype=np.int64)
    m = w.n_links
    sel = (idx[:, None] * m + np.arange(m)[None, :]).reshape(-1)
    return replace(w, n_scenarios=len(idx), bw=w.bw[sel].copy(),
                   lat=w.lat[sel].copy(), cap=w.cap[sel].copy(),
                   credit=None if w.credit is None else w.credit[sel].copy())


def random_graph(rng: np.random.Generator, n_end: int, n_sw: int, extra: int,
                 bmax=3, Lmax=3, capmax=4, S=1):
    """Small random strongly connected digraph for brute-force tests.

    A bidirectional spanning tree over all nodes plus ``extra`` random
    directed links; parameters drawn per link and scenario."""
    n = n_end + n_sw
    order = rng.permutation(n)
    edges = set()
    for i in range(1, n):
        u, v = int(order[i]), int(order[rng.integers(0, i)])
        edges.add((u, v))
        edges.add((v, u))
    for _ in range(extra):
        u, v = (int(t) for t in rng.integers(0, n, size=2))
        if u != v:
            edges.add((u, v))
    row_ptr, col_idx, lid = _csr(n, edges)
    m = len(lid)
    bw = rng.integers(1, bmax + 1, size=S * m).astype(np.int32)
    lat = rng.integers(1, Lmax + 1, size=S * m).astype(np.int32)
    cp = rng.integers(1, capmax + 1, size=S * m).astype(np.int32)
    return n, row_ptr, col_idx, bw, lat, cp


def random_dag(rng: np.random.Generator, n_end: int, n_txn: int, max_preds=2):
    """Random transaction list over endpoints ``0..n_end-1`` for custom-DAG
    tests: each transaction gets a random (src != dst) pair and up to
    ``max_preds`` distinct predecessors among lower ids (so the graph is a DAG)."""
    src = rng.integers(0, n_end, size=n_txn).astype(np.int32)
    off = rng.integers(1, n_end, size=n_txn).astype(np.int32)
    dst = ((src + off) % n_end).astype(np.int32)
    pred_ptr = [0]
    pred_idx = []
    for x in range(n_txn):
        k = int(rng.integers(0, max_preds + 1)) if x else 0
        k = min(k, x)
        if k:
            pred_idx += sorted(int(v) for v in rng.choice(x, size=k, replace=False))
        pred_ptr.append(len(pred_idx))
    return (src, dst, np.array(pred_ptr, np.int64), np.array(pred_idx, np.int64))
