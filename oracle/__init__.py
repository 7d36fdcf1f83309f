"""CPU oracle of the line-granularity network model -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does, and the
two share no code: this package loads ``liboracle.so`` built from
``oracle.c`` with gcc, and ``stepper.py`` holds an independent per-cycle
Python stepper used as the brute-force pin for tiny inputs.

Functions mirror the model rules documented at the top of ``oracle.c``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

STATUS = {0: "OK", 1: "INVALID_ARG", 2: "TOPOLOGY", 3: "UNREACHABLE", 4: "SIZE",
          5: "OOM", 7: "DEADLOCK", 8: "MAX_CYCLES", 100: "INVARIANT"}


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (plain -O2, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-D_POSIX_C_SOURCE=199309L",
                               "-Wall", "-shared", "-fPIC", "-o", tmp,
                               os.path.join(_HERE, "oracle.c")])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Stats(C.Structure):
    _fields_ = [("processed_cycles", C.c_uint64), ("line_hops", C.c_uint64),
                ("seconds", C.c_double)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = C.CDLL(_LIB_PATH)
        P = C.c_void_p
        L.oracle_fmix32.argtypes = [C.c_uint32]
        L.oracle_fmix32.restype = C.c_uint32
        L.oracle_paths.argtypes = [C.c_int32, C.c_int32, P, P, P, P, C.c_int64]
        L.oracle_paths.restype = C.c_int
        L.oracle_txn.argtypes = [C.c_int, C.c_uint64, C.c_int32, C.c_int32, P, C.c_int32, C.c_int64,
                                 P, P, P, P, C.c_int32, P]
        L.oracle_txn.restype = C.c_int
        L.oracle_simulate.argtypes = [C.c_int32, C.c_int32, P, P, P, P, P, P, C.c_int32,
                                      C.c_int32, C.c_uint64, C.c_int32, P, C.c_int32,
                                      C.c_int64, P, P, P, P, P,
                                      C.c_uint64, C.c_int32, P, P, P, P, P]
        L.oracle_simulate.restype = C.c_int
        i32, i64 = C.c_int32, C.c_int64
        L.oracle_memcpy.argtypes = [i64, P, P, P, P, P, P, i32, i32, P, i32, i32, i64, i64,
                                    P, P, P, P, P, P, P]
        L.oracle_memcpy.restype = C.c_int
        L.oracle_gpu_ops.argtypes = [i64, P, P, P, P, P, P, P, P, i32, i32, P, i32, i32, i64, i64,
                                     P, P, P, P, P, P, P]
        L.oracle_gpu_ops.restype = C.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def fmix32(h: int) -> int:
    return int(lib().oracle_fmix32(h & 0xFFFFFFFF))


def paths(n, E, row_ptr, col_idx):
    """Return (status, path_ptr[E*E+1] int64, path_link int32)."""
    row_ptr = np.ascontiguousarray(row_ptr, np.int32)
    col_idx = np.ascontiguousarray(col_idx, np.int32)
    pp = np.zeros(E * E + 1, np.int64)
    cap = max(16, E * E * 8)
    pl = np.zeros(cap, np.int32)
    rc = lib().oracle_paths(n, E, _p(row_ptr), _p(col_idx), _p(pp), _p(pl), cap)
    if rc == 4:
        cap = int(pp[-1])
        pl = np.zeros(cap, np.int32)
        rc = lib().oracle_paths(n, E, _p(row_ptr), _p(col_idx), _p(pp), _p(pl), cap)
    return rc, pp, pl[:int(pp[-1])] if rc == 0 else pl


def txn(coll, nbytes, group, E, x, order=None, dep=0):
    """Decode one transaction: (status, src, dst, preds list, T).  With
    dep=1 (chunk dependencies) a predecessor -1-m stands for whole message m
    (one step's transfer between two participants)."""
    src = np.zeros(1, np.int32)
    dst = np.zeros(1, np.int32)
    npred = np.zeros(1, np.int32)
    preds = np.zeros(64, np.int64)
    T = np.zeros(1, np.int64)
    o = None if order is None else np.ascontiguousarray(order, np.int32)
    rc = lib().oracle_txn(coll, nbytes, group, E, _p(o), dep, x, _p(src), _p(dst), _p(npred),
                          _p(preds), len(preds), _p(T))
    if rc == 4 and npred[0] > len(preds):  # more predecessors than the first buffer holds
        preds = np.zeros(int(npred[0]), np.int64)
        rc = lib().oracle_txn(coll, nbytes, group, E, _p(o), dep, x, _p(src), _p(dst), _p(npred),
                              _p(preds), len(preds), _p(T))
    return rc, int(src[0]), int(dst[0]), [int(v) for v in preds[:npred[0]]], int(T[0])


def memcpy_txns(mc, with_class=False):
    """Expand GPU programs (``sim_inputs.noc.Memcpy``: copies, reduces,
    releases and acquires) into the line list (src, dst, pred_ptr, pred_idx)
    [+ per-line class: 1 = control message]."""
    n_ops = len(mc.cu)
    if mc.kind is None:   # plain memcpy: one source per operation
        kind = np.zeros(n_ops, np.int32)
        sptr = np.arange(n_ops + 1, dtype=np.int64)
    else:
        kind = np.ascontiguousarray(mc.kind, np.int32)
        sptr = np.ascontiguousarray(mc.src_ptr, np.int64)
    cu = np.ascontiguousarray(mc.cu, np.int32)
    ssp = np.ascontiguousarray(mc.src_space, np.int32)
    dsp = np.ascontiguousarray(mc.dst_space, np.int32)
    sl = np.ascontiguousarray(mc.src_line, np.int64)
    dl = np.ascontiguousarray(mc.dst_line, np.int64)
    nl = np.ascontiguousarray(mc.n_lines, np.int64)
    ch = np.ascontiguousarray(mc.space_channels, np.int32)
    if len(sptr) != n_ops + 1 or len(ssp) < sptr[-1] or len(sl) < sptr[-1] or len(dsp) < n_ops:
        raise ValueError("gpu programs: inconsistent array lengths")
    n_spaces = len(ch) // mc.n_ch
    T = np.zeros(1, np.int64)
    P = np.zeros(1, np.int64)
    args = (n_ops, _p(kind), _p(cu), _p(sptr), _p(ssp), _p(sl), _p(dsp), _p(dl), _p(nl), n_spaces, mc.n_ch,
            _p(ch), mc.unroll, mc.window)
    rc = lib().oracle_gpu_ops(*args, 0, 0, None, None, None, None, None, _p(T), _p(P))
    if rc:
        raise ValueError(f"oracle_gpu_ops: status {rc}")
    src = np.zeros(max(int(T[0]), 1), np.int32)
    dst = np.zeros(max(int(T[0]), 1), np.int32)
    pptr = np.zeros(int(T[0]) + 1, np.int64)
    pidx = np.zeros(max(int(P[0]), 1), np.int64)
    cls = np.zeros(max(int(T[0]), 1), np.uint8)
    rc = lib().oracle_gpu_ops(*args, int(T[0]), int(P[0]), _p(src), _p(dst), _p(pptr), _p(pidx), _p(cls),
                              _p(T), _p(P))
    assert rc == 0
    t = int(T[0])
    if with_class:
        return src[:t], dst[:t], pptr, pidx[:int(P[0])], cls[:t]
    return src[:t], dst[:t], pptr, pidx[:int(P[0])]


@dataclass
class Result:
    status: int
    completion: np.ndarray
    tx_lines: np.ndarray
    busy_cycles: np.ndarray
    makespan: int
    processed_cycles: int
    line_hops: int
    seconds: float

    @property
    def status_name(self):
        return STATUS.get(self.status, str(self.status))


def simulate(n, E, row_ptr, col_idx, bw, lat, cap, arb, *, coll=-1, nbytes=0, group=0,
             order=None, dep=0, txns=None, max_cycles=0, check=False, credit=None, cls=None) -> Result:
    """Run one scenario.  ``txns`` = (src, dst, pred_ptr, pred_idx) for a custom
    transaction list (coll = -1); otherwise ``coll``/``nbytes``/``group``."""
    row_ptr = np.ascontiguousarray(row_ptr, np.int32)
    col_idx = np.ascontiguousarray(col_idx, np.int32)
    m = int(row_ptr[-1])
    bw = np.ascontiguousarray(bw, np.int32)[:m]
    lat = np.ascontiguousarray(lat, np.int32)[:m]
    cap = np.ascontiguousarray(cap, np.int32)[:m]
    cr = None if credit is None else np.ascontiguousarray(credit, np.int32)[:m]
    o = None if order is None else np.ascontiguousarray(order, np.int32)
    if txns is not None:
        coll = -1
        src, dst, pptr, pidx = (np.ascontiguousarray(txns[0], np.int32),
                                np.ascontiguousarray(txns[1], np.int32),
                                np.ascontiguousarray(txns[2], np.int64),
                                np.ascontiguousarray(txns[3], np.int64))
        if len(pidx) == 0:
            pidx = np.zeros(1, np.int64)
        T = len(src)
        cls = None if cls is None else np.ascontiguousarray(cls, np.uint8)
    else:
        cls = None
        src = dst = pptr = pidx = None
        rc, _, _, _, T = txn(coll, nbytes, group, E, 0, order, dep)
        if rc:
            return Result(rc, np.zeros(0, np.uint32), np.zeros(m, np.uint64),
                          np.zeros(m, np.uint64), 0, 0, 0, 0.0)
    comp = np.empty(max(T, 1), np.uint32)
    tx = np.zeros(m, np.uint64)
    busy = np.zeros(m, np.uint64)
    mk = np.zeros(1, np.uint32)
    st = _Stats()
    rc = lib().oracle_simulate(n, E, _p(row_ptr), _p(col_idx), _p(bw), _p(lat), _p(cap), _p(cr), arb,
                               coll, nbytes, group, _p(o), dep, T, _p(src), _p(dst), _p(cls), _p(pptr),
                               _p(pidx), max_cycles, 1 if check else 0, _p(comp), _p(tx),
                               _p(busy), _p(mk), C.byref(st))
    return Result(rc, comp[:T], tx, busy, int(mk[0]), int(st.processed_cycles),
                  int(st.line_hops), float(st.seconds))


def simulate_workload(w, scenario: int = 0, *, max_cycles=0, check=False) -> Result:
    """Run scenario ``scenario`` of a ``sim_inputs.Workload``."""
    m = w.n_links
    sl = slice(scenario * m, (scenario + 1) * m)
    txns = cls = None
    if w.meta.get("memcpy") is not None:
        *txns, cls = memcpy_txns(w.meta["memcpy"], with_class=True)
    credit = None if getattr(w, "credit", None) is None else w.credit[sl]
    return simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw[sl], w.lat[sl],
                    w.cap[sl], w.arb, coll=w.coll, nbytes=w.bytes, group=w.group_size,
                    order=w.order, dep=w.dep, txns=txns, max_cycles=max_cycles, check=check,
                    credit=credit, cls=cls)
