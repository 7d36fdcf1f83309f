"""Literal per-cycle stepper of the network model, in pure Python.

An independent second implementation used only as a brute-force pin of the
CPU oracle on tiny inputs: it does its own routing, walks every cycle
t = 0, 1, 2, ... (no event skipping) and keeps state in plain lists.  It
shares nothing with ``oracle/oracle.c`` or with the GPU library.

Model (the reading documented with the design notes): every link is a FIFO
with bandwidth b, latency L and capacity cap (lines in flight plus waiting);
per cycle, from the state at the start of the cycle, sources offer up to b
lines, each link grants min(b, cap - occupancy, #requests) in key order, the
longest granted prefix of each source departs, departing lines enter their
target in grant order with ready = t + L, and a line leaving its last hop
completes at t + 1.
"""
from __future__ import annotations

from collections import deque

SINK = None


def murmur_fmix32(h: int) -> int:
    h &= 0xFFFFFFFF
    h ^= h >> 16
    h = (h * 0x85EBCA6B) & 0xFFFFFFFF
    h ^= h >> 13
    h = (h * 0xC2B2AE35) & 0xFFFFFFFF
    h ^= h >> 16
    return h


def hop_distances(n, row_ptr, col_idx, d):
    """Hops from every node to d, by repeated relaxation (no queue)."""
    INF = 10 ** 9
    dist = [INF] * n
    dist[d] = 0
    changed = True
    while changed:
        changed = False
        for u in range(n):
            for l in range(row_ptr[u], row_ptr[u + 1]):
                v = col_idx[l]
                if dist[v] + 1 < dist[u]:
                    dist[u] = dist[v] + 1
                    changed = True
    return dist


def route(n, row_ptr, col_idx, s, d, dist):
    if dist[s] >= 10 ** 9:
        return None
    h = murmur_fmix32((s << 16) | d)
    path, v, choice = [], s, 0
    while v != d:
        cands = [l for l in range(row_ptr[v], row_ptr[v + 1]) if dist[col_idx[l]] == dist[v] - 1]
        if len(cands) == 1:
            l = cands[0]
        else:
            if choice and choice % 4 == 0:
                h = murmur_fmix32(h)
            l = cands[((h >> (8 * (choice % 4))) & 255) % len(cands)]
            choice += 1
        path.append(l)
        v = col_idx[l]
    return path


def step_simulate(n, E, row_ptr, col_idx, bw, lat, cap, arb, src, dst, preds, max_cycles=10 ** 6, credit=None,
                  cls=None):
    """Returns (status, completion list, tx_lines, busy, makespan).  credit:
    per-link credit delay D (default 1): the slot a line frees by leaving
    link l at cycle t can be granted again from cycle t + D on.  arb: 0
    lowest id, 1 round-robin, +2 class-fair: picks alternate between the
    classes (cls[x], 0 data, 1 control) starting from the class the link's
    pointer names, each the lowest key of that class among the sources' next
    requests (or of any class); after appending, the pointer names the class
    other than the last appended line's."""
    row_ptr = [int(v) for v in row_ptr]
    col_idx = [int(v) for v in col_idx]
    m = row_ptr[-1]
    bw = [int(v) for v in bw[:m]]
    lat = [int(v) for v in lat[:m]]
    cap = [int(v) for v in cap[:m]]
    credit = [1] * m if credit is None else [int(v) for v in credit[:m]]
    owed = [[] for _ in range(m)]   # [cycle the credits come back, how many]
    tail = [u for u in range(n) for _ in range(row_ptr[u], row_ptr[u + 1])]
    ports = {v: sorted(l for l in range(m) if col_idx[l] == v) for v in range(n)}
    port_of = {l: ports[col_idx[l]].index(l) for l in range(m)}
    nports = [len(ports[v]) + (1 if v < E else 0) for v in range(n)]
    T = len(src)
    dist_to = {}
    paths = []
    for x in range(T):
        s, d = int(src[x]), int(dst[x])
        if d not in dist_to:
            dist_to[d] = hop_distances(n, row_ptr, col_idx, d)
        p = route(n, row_ptr, col_idx, s, d, dist_to[d])
        if p is None:
            return "UNREACHABLE", None, None, None, None
        paths.append(p)
    streams = {}
    for x in range(T):
        streams.setdefault(paths[x][0], []).append(x)
    cursor = {f: 0 for f in streams}
    fifo = [deque() for _ in range(m)]   # [line, ready, hop]
    rr = [0] * m
    cptr = [0] * m
    cls = [0] * len(src) if cls is None else [int(v) for v in cls]
    comp = [None] * T
    tx = [0] * m
    busy = [0] * m
    t = 0
    while any(c is None for c in comp):
        if t > max_cycles:
            return "MAX_CYCLES", comp, tx, busy, None
        for l in range(m):
            owed[l] = [c for c in owed[l] if c[0] > t]
        reqs = []   # dict(source, k, x, target, port, hop)
        for l in range(m):
            for k, (x, ready, hop) in enumerate(list(fifo[l])[:bw[l]]):
                if ready > t:
                    break
                p = paths[x]
                tgt = p[hop + 1] if hop + 1 < len(p) else SINK
                reqs.append(dict(source=("fifo", l), k=k, x=x, target=tgt, port=port_of[l], hop=hop + 1))
        for f, lst in streams.items():
            for k in range(bw[f]):
                i = cursor[f] + k
                if i >= len(lst):
                    break
                x = lst[i]
                if not all(comp[q] is not None and comp[q] <= t for q in preds[x]):
                    break
                reqs.append(dict(source=("stream", f), k=k, x=x, target=f, port=nports[tail[f]] - 1, hop=0))
        for r in reqs:
            r["granted"] = r["target"] is SINK
        order_of = {}
        for f in set(r["target"] for r in reqs if r["target"] is not SINK):
            rs = [r for r in reqs if r["target"] == f]
            P = nports[tail[f]]
            if arb & 1 == 0:
                rs.sort(key=lambda r: r["x"])
            else:
                rs.sort(key=lambda r: (r["k"], (r["port"] - rr[f]) % P))
            if arb & 2:
                # class turns, picking only among each source's next request
                left, rs, turn = list(rs), [], cptr[f]
                while left:
                    heads = [r for r in left
                             if not any(o["source"] == r["source"] and o["k"] < r["k"] for o in left)]
                    mine = [r for r in heads if cls[r["x"]] == turn]
                    r = (mine or heads)[0]
                    rs.append(r)
                    left.remove(r)
                    turn = 1 - cls[r["x"]]
            g = min(bw[f], cap[f] - len(fifo[f]) - sum(c[1] for c in owed[f]), len(rs))
            for r in rs[:g]:
                r["granted"] = True
            order_of[f] = rs
        by_source = {}
        for r in reqs:
            by_source.setdefault(r["source"], []).append(r)
        for rs in by_source.values():
            rs.sort(key=lambda r: r["k"])
            ok = True
            for r in rs:
                ok = ok and r["granted"]
                r["departs"] = ok
        departed = sum(1 for r in reqs if r["departs"])
        for f, rs in order_of.items():
            moved = [r for r in rs if r["departs"]]
            for r in moved:
                fifo[f].append([r["x"], t + lat[f], r["hop"]])
            if moved:
                tx[f] += len(moved)
                busy[f] += 1
                if arb & 1:
                    rr[f] = (moved[-1]["port"] + 1) % nports[tail[f]]
                if arb & 2:
                    cptr[f] = 1 - cls[moved[-1]["x"]]
        for (kind, idx), rs in by_source.items():
            ndep = sum(1 for r in rs if r["departs"])
            for r in rs:
                if r["departs"] and r["target"] is SINK:
                    comp[r["x"]] = t + 1
            if kind == "fifo":
                for _ in range(ndep):
                    fifo[idx].popleft()
                if ndep and credit[idx] > 1:
                    owed[idx].append([t + credit[idx], ndep])
            else:
                cursor[idx] += ndep
        if departed == 0 and not any(e[1] > t for q in fifo for e in q) and not any(owed) and \
                any(c is None for c in comp):
            return "DEADLOCK", comp, tx, busy, None
        t += 1
    return "OK", comp, tx, busy, max(comp) if comp else 0
