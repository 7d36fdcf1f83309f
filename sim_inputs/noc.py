"""Seeded inputs for the GPU-as-NoC case: the generic GPU of the paper's
case studies (Sec. 5.1) and memcpy programs run by its compute units.

Per GPU: a 2D mesh of 8 x 4 routers; four compute units (CUs) on every
router; 16 memory channels on every router of the top and bottom rows (256
channels); four I/O ports on every router of the left and right columns (32
ports).  GPUs are joined through scale-up switches, one per I/O port index
(port k of every GPU is cabled to switch k).

Node ids: endpoints first -- per GPU its 128 CUs, then its 256 memory
channels -- then per GPU its 32 routers and 32 I/O ports, then the scale-up
switches.  CUs and channels inject and eject lines; routers, I/O ports and
switches only forward them.

Link parameters (b lines/cycle, L cycles, cap lines).  The paper gives
bandwidths only: 1 TiB/s on-chip links, 4 TiB/s over the 256 channels
(16 GiB/s each), 1 TiB/s of scale-up bandwidth over the 32 ports (32 GiB/s
each) with 1 us of latency.  Links carry whole lines per cycle, so the cycle
is taken as the time one channel needs for a line: 128 B / 16 GiB/s = 7.45
ns.  Then an on-chip link moves 64 lines per cycle, a channel 1, a port 2,
and 1 us is 134 cycles (67 on each of the two cables between GPUs).  A CU
dispatches up to 8 requests per cycle (one per GPU clock of about 1 ns).
Hop latencies on chip, buffer depths and the CU dispatch rate are this
module's choices (the paper states none of them); every buffer holds at
least b(L+1) lines except the channels', which hold 4.

This module only wires graphs and writes operation lists; it performs none
of the simulated method's arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np

from . import Workload, _csr, ARB_ROUND_ROBIN

CYCLE_NS = 128 / (16 * 2 ** 30) * 1e9   # one line on one memory channel

NOC = (64, 1, 128)        # router <-> router, router -> CU, router <-> port
CU_OUT = (8, 1, 16)       # CU -> router: the CU's request dispatch rate
MEM = (1, 1, 4)           # channel <-> router
IO = (2, 67, 270)         # port <-> scale-up switch, each way


@dataclass
class NocLayout:
    n_gpus: int
    mesh: tuple
    cus: np.ndarray        # [G, 128] endpoint ids
    channels: np.ndarray   # [G, 256] endpoint ids
    routers: np.ndarray    # [G, 32] node ids
    ports: np.ndarray      # [G, 32] node ids


OP_COPY, OP_RELEASE, OP_ACQUIRE = 0, 1, 2


@dataclass
class Memcpy:
    """GPU operations, each run by one CU in list order per CU.

    Without ``kind`` every operation is a memcpy from (src_space[o],
    src_line[o]).  With ``kind`` (OP_COPY, OP_RELEASE, OP_ACQUIRE) and
    ``src_ptr`` the sources of operation o are entries src_ptr[o] ..
    src_ptr[o+1] - 1 of src_space / src_line: a copy has one or more (more
    than one: a reduce into the destination), a release or acquire none and
    names its semaphore line as the destination, with n_lines 1.

    Line a of address space s (a GPU's memory) lives on memory channel
    ``space_channels[s * n_ch + a % n_ch]``."""
    cu: np.ndarray          # int32 [n_ops] endpoint executing the operation
    src_space: np.ndarray   # int32 [n_ops] (or [src_ptr[-1]])
    dst_space: np.ndarray   # int32 [n_ops]
    src_line: np.ndarray    # int64 [n_ops] (or [src_ptr[-1]]) first source line address
    dst_line: np.ndarray    # int64 [n_ops]
    n_lines: np.ndarray     # int64 [n_ops]
    space_channels: np.ndarray  # int32 [n_spaces * n_ch]
    n_ch: int
    unroll: int = 4
    window: int = 64
    kind: np.ndarray | None = None     # int32 [n_ops]
    src_ptr: np.ndarray | None = None  # int64 [n_ops + 1]


def gpu_noc(n_gpus: int = 1, *, mesh=(8, 4), cus_per_router=4, ch_per_router=16, ports_per_router=4,
            noc=NOC, cu_out=CU_OUT, mem=MEM, io=IO, arb=ARB_ROUND_ROBIN,
            name="gpu_noc") -> tuple[Workload, NocLayout]:
    X, Y = mesh
    R = X * Y
    n_cu = R * cus_per_router
    edge_routers = [(x, y) for y in range(Y) for x in range(X) if y in (0, Y - 1)]
    side_routers = [(x, y) for y in range(Y) for x in range(X) if x in (0, X - 1)]
    n_ch = len(edge_routers) * ch_per_router
    n_port = len(side_routers) * ports_per_router
    E_per = n_cu + n_ch
    E = n_gpus * E_per
    cus = np.zeros((n_gpus, n_cu), np.int32)
    chans = np.zeros((n_gpus, n_ch), np.int32)
    routers = np.zeros((n_gpus, R), np.int32)
    ports = np.zeros((n_gpus, n_port), np.int32)
    for g in range(n_gpus):
        cus[g] = g * E_per + np.arange(n_cu)
        chans[g] = g * E_per + n_cu + np.arange(n_ch)
        routers[g] = E + g * (R + n_port) + np.arange(R)
        ports[g] = E + g * (R + n_port) + R + np.arange(n_port)
    sw0 = E + n_gpus * (R + n_port)
    n = sw0 + (n_port if n_gpus > 1 else 0)
    params = {}

    def cable(u, v, fwd, back):
        params[(u, v)] = fwd
        params[(v, u)] = back

    rid = lambda g, x, y: int(routers[g][y * X + x])
    for g in range(n_gpus):
        for y in range(Y):
            for x in range(X):
                if x + 1 < X:
                    cable(rid(g, x, y), rid(g, x + 1, y), noc, noc)
                if y + 1 < Y:
                    cable(rid(g, x, y), rid(g, x, y + 1), noc, noc)
        for r in range(R):
            for k in range(cus_per_router):
                cable(int(cus[g][r * cus_per_router + k]), int(routers[g][r]), cu_out, noc)
        for e, (x, y) in enumerate(edge_routers):
            for k in range(ch_per_router):
                cable(int(chans[g][e * ch_per_router + k]), rid(g, x, y), mem, mem)
        for e, (x, y) in enumerate(side_routers):
            for k in range(ports_per_router):
                p = int(ports[g][e * ports_per_router + k])
                cable(rid(g, x, y), p, noc, noc)
                if n_gpus > 1:
                    cable(p, sw0 + e * ports_per_router + k, io, io)
    row_ptr, col_idx, lid = _csr(n, list(params))
    m = len(lid)
    bw = np.zeros(m, np.int32)
    lat = np.zeros(m, np.int32)
    cap = np.zeros(m, np.int32)
    for e, i in lid.items():
        bw[i], lat[i], cap[i] = params[e]
    w = Workload(name, n, E, row_ptr, col_idx, 1, bw, lat, cap, arb, -1, 0)
    lay = NocLayout(n_gpus, mesh, cus, chans, routers, ports)
    w.meta["noc"] = lay
    return w, lay


def _space_channels(lay: NocLayout) -> np.ndarray:
    return lay.channels.reshape(-1).astype(np.int32)


def _ops(rows, lay, unroll, window) -> Memcpy:
    a = np.array(rows, dtype=np.int64).reshape(-1, 6)
    return Memcpy(a[:, 0].astype(np.int32), a[:, 1].astype(np.int32), a[:, 2].astype(np.int32),
                  a[:, 3].copy(), a[:, 4].copy(), a[:, 5].copy(), _space_channels(lay),
                  lay.channels.shape[1], unroll, window)


def _prog(rows, lay, unroll, window) -> Memcpy:
    """rows: (kind, cu, [(src_space, src_line), ...], dst_space, dst_line, n_lines)."""
    kind = np.array([r[0] for r in rows], np.int32)
    cu = np.array([r[1] for r in rows], np.int32)
    sptr = np.zeros(len(rows) + 1, np.int64)
    sptr[1:] = np.cumsum([len(r[2]) for r in rows])
    srcs = [sl for r in rows for sl in r[2]]
    ssp = np.array([a for a, _ in srcs], np.int32)
    sln = np.array([b for _, b in srcs], np.int64)
    return Memcpy(cu, ssp, np.array([r[3] for r in rows], np.int32), sln, np.array([r[4] for r in rows], np.int64),
                  np.array([r[5] for r in rows], np.int64), _space_channels(lay), lay.channels.shape[1], unroll,
                  window, kind, sptr)


def wg_cu(lay: NocLayout, g: int, wg: int, n_wg: int) -> int:
    """CU of workgroup wg (of n_wg) on GPU g: spread over the routers first."""
    n_cu = lay.cus.shape[1]
    R = lay.routers.shape[1]
    per = n_cu // R
    return int(lay.cus[g][(wg % R) * per + (wg // R) % per])


def allgather_ops(lay: NocLayout, out_lines: int, n_wg: int = 32, unroll=4, window=64, get=False) -> Memcpy:
    """All-gather (the scalability workload of Sec. 5.4): GPU g's input of
    out_lines / G lines (at address 0) is copied into every GPU's output
    buffer (at address out_lines / G, slot g).  Put-based: the n_wg
    workgroups of GPU g split g's input and write it to the peers g, g+1,
    ... (remote stores).  Get-based (Sec. 5.2): the workgroups of GPU h split
    each peer's input and read it into h's output, peers h, h+1, ... (remote
    loads: their requests are control messages)."""
    G = lay.n_gpus
    chunk = out_lines // G
    assert chunk * G == out_lines and chunk % n_wg == 0
    c = chunk // n_wg
    rows = []
    for g in range(G):
        for wg in range(n_wg):
            cu = wg_cu(lay, g, wg, n_wg)
            for d in range(G):
                h = (g + d) % G
                if get:   # GPU g reads h's input into its own output slot h
                    rows.append((cu, h, g, wg * c, chunk + h * chunk + wg * c, c))
                else:
                    rows.append((cu, g, h, wg * c, chunk + g * chunk + wg * c, c))
    return _ops(rows, lay, unroll, window)


def reducescatter_ops(lay: NocLayout, in_lines: int, n_wg: int = 32, unroll=4, window=64, get=True) -> Memcpy:
    """Reduce-scatter (Sec. 5.2): every GPU holds in_lines input lines at
    address 0, in G chunks; GPU g ends with the sum of every GPU's chunk g in
    its output (address in_lines).  The n_wg workgroups of a GPU split each
    chunk into slices.

    Get-based: workgroup w of GPU g reads its slice of chunk g from every GPU
    (g first, then g+1, ...: local and remote loads) and stores the reduced
    slice; no synchronisation.
    Put-based: workgroup w of GPU g first copies its slice of chunk h to
    GPU h's scratch slot g (address in_lines + chunk + g chunk; remote
    stores) and releases the semaphore (h, w, from g) on GPU h, for the peers
    h = g+1, g+2, ...; then it acquires its own semaphores from every peer
    and reduces its input slice with the G - 1 received slices (local loads)
    into its output.  Semaphore (h, w, from g) is line
    2 in_lines + chunk + g n_wg + w of GPU h."""
    G = lay.n_gpus
    chunk = in_lines // G
    assert chunk * G == in_lines and chunk % n_wg == 0
    c = chunk // n_wg
    out, scratch, sem = in_lines, in_lines + chunk, 2 * in_lines + chunk
    rows = []
    for g in range(G):
        for w in range(n_wg):
            cu = wg_cu(lay, g, w, n_wg)
            peers = [(g + d) % G for d in range(1, G)]
            if get:
                rows.append((OP_COPY, cu, [((g + d) % G, g * chunk + w * c) for d in range(G)], g, out + w * c, c))
                continue
            for h in peers:
                rows.append((OP_COPY, cu, [(g, h * chunk + w * c)], h, scratch + g * chunk + w * c, c))
                rows.append((OP_RELEASE, cu, [], h, sem + g * n_wg + w, 1))
            for h in peers:
                rows.append((OP_ACQUIRE, cu, [], g, sem + h * n_wg + w, 1))
            rows.append((OP_COPY, cu, [(g, g * chunk + w * c)] + [(g, scratch + h * chunk + w * c) for h in peers],
                         g, out + w * c, c))
    return _prog(rows, lay, unroll, window)


def alltoall_ops(lay: NocLayout, pair_lines: int, n_wg: int = 32, unroll=4, window=64) -> Memcpy:
    """All-to-all: GPU g sends pair_lines lines to every other GPU h (from
    input slot h to output slot g), split over its workgroups."""
    G = lay.n_gpus
    assert pair_lines % n_wg == 0
    c = pair_lines // n_wg
    rows = []
    for g in range(G):
        for wg in range(n_wg):
            cu = wg_cu(lay, g, wg, n_wg)
            for d in range(1, G):
                h = (g + d) % G
                rows.append((cu, g, h, h * pair_lines + wg * c, G * pair_lines + g * pair_lines + wg * c, c))
    return _ops(rows, lay, unroll, window)


def local_copy_ops(lay: NocLayout, lines: int, n_wg: int = 128, unroll=4, window=64, gpu=0) -> Memcpy:
    """One GPU copies lines lines inside its own memory (address 0 to address
    lines), split over n_wg workgroups."""
    assert lines % n_wg == 0
    c = lines // n_wg
    rows = [(wg_cu(lay, gpu, wg, n_wg), gpu, gpu, wg * c, lines + wg * c, c) for wg in range(n_wg)]
    return _ops(rows, lay, unroll, window)


def memcpy_workload(w: Workload, mc: Memcpy, name=None) -> Workload:
    w = replace(w, name=name or w.name, meta=dict(w.meta))
    w.meta["memcpy"] = mc
    return w


def with_scenarios(w: Workload, S: int, seed: int, *, mem_lat=(1, 2, 4, 8), io_lat=(40, 67, 134)) -> Workload:
    """S scenarios of the same NoC: per scenario one SplitMix64 draw picks
    the channel-link latency, a second one the scale-up cable latency."""
    from . import splitmix64
    m = w.n_links
    bw = np.tile(w.bw[:m], S)
    lat = np.tile(w.lat[:m], S)
    cap = np.tile(w.cap[:m], S)
    lay = w.meta["noc"]
    chans = set(lay.channels.reshape(-1).tolist())
    io_cable = lat[:m] == IO[1]
    tails = np.repeat(np.arange(w.n_nodes), np.diff(w.row_ptr))
    mem_link = np.array([int(t) in chans or int(h) in chans for t, h in zip(tails, w.col_idx)])
    rng = splitmix64(seed)
    for s in range(S):
        lm = mem_lat[next(rng) % len(mem_lat)]
        li = io_lat[next(rng) % len(io_lat)]
        sl = slice(s * m, (s + 1) * m)
        lat[sl][mem_link] = lm
        lat[sl][io_cable] = li
        cap[sl][mem_link] = np.maximum(cap[sl][mem_link], bw[sl][mem_link] * (lm + 1))
        cap[sl][io_cable] = bw[sl][io_cable] * (li + 1)
    return replace(w, n_scenarios=S, bw=bw, lat=lat, cap=cap)
