"""Thin ctypes binding of libsimgpu (argument marshalling only).

Functions keep the C ABI's names (``sim_create``, ``sim_set_credit``, ``sim_load_collective``,
``sim_load_transactions``, ``sim_load_memcpy``, ``sim_load_gpu_ops``, ``sim_sizes``, ``sim_run``,
``sim_status_after_sync``, ``sim_route``, ``sim_txn_info``, ``sim_last_error``,
``sim_destroy``); ``Simulator`` bundles them with torch device buffers and
the current HIP stream.  Every step of the simulation runs in the library's
HIP kernels; there is no host fallback: if the library is missing, loading
fails with an error.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SIMGPU_LIB", os.path.join(_HERE, "libsimgpu.so"))

SIM_OK, SIM_ERR_INVALID_ARG, SIM_ERR_TOPOLOGY, SIM_ERR_UNREACHABLE, SIM_ERR_SIZE = 0, 1, 2, 3, 4
SIM_ERR_OOM, SIM_ERR_DEVICE, SIM_ERR_DEADLOCK, SIM_ERR_MAX_CYCLES, SIM_ERR_STATE = 5, 6, 7, 8, 9
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "TOPOLOGY", 3: "UNREACHABLE", 4: "SIZE", 5: "OOM",
                6: "DEVICE", 7: "DEADLOCK", 8: "MAX_CYCLES", 9: "STATE"}
EXPORTS = ("sim_create", "sim_set_credit", "sim_load_collective", "sim_load_transactions", "sim_load_memcpy",
           "sim_load_gpu_ops", "sim_sizes", "sim_run", "sim_run_noalloc",
           "sim_status_after_sync", "sim_route", "sim_txn_info", "sim_last_error", "sim_destroy")

_lib = None


class SimError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib():
    """Load libsimgpu.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2606_10440_amd/build.py")
        L = C.CDLL(LIB_PATH)
        P, i32, i64, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64
        L.sim_create.argtypes = [i32, i32, P, P, i32, P, P, P, i32, C.POINTER(P)]
        L.sim_set_credit.argtypes = [P, P]
        L.sim_load_collective.argtypes = [P, i32, u64, i32, P, i32]
        L.sim_load_transactions.argtypes = [P, i64, P, P, P, P]
        L.sim_load_memcpy.argtypes = [P, i64, P, P, P, P, P, P, C.c_int32, C.c_int32, P, C.c_int32, C.c_int32]
        L.sim_load_gpu_ops.argtypes = [P, i64, P, P, P, P, P, P, P, P, i32, i32, P, i32, i32]
        L.sim_sizes.argtypes = [P, P, P, P, P]
        L.sim_run.argtypes = [P, P, P, P, P, P, u64]
        L.sim_run_noalloc.argtypes = [P, P, P, P, P, P, u64]
        L.sim_status_after_sync.argtypes = [P, P, P]
        L.sim_route.argtypes = [P, i32, i32, P, i32, P]
        L.sim_txn_info.argtypes = [P, i64, P, P, P, P]
        L.sim_last_error.argtypes = [P]
        L.sim_last_error.restype = C.c_char_p
        L.sim_destroy.argtypes = [P]
        L.sim_destroy.restype = None
        for name in EXPORTS[:-2]:
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(ctx, st: int):
    if st != SIM_OK:
        msg = lib().sim_last_error(ctx).decode() if ctx else ""
        raise SimError(st, msg)


# ------------------------------------------------------------------ reporting

_BUS_FACTOR = {0: "ar", 1: "ar", 2: "ar", 8: "ar", 9: "ar", 4: "one", 5: "one", 6: "one", 7: "one", 3: "a2a"}


def bus_bandwidth(coll, nbytes, p, seconds):
    """Bus bandwidth in bits/s of a collective that took ``seconds`` (the
    measure the paper reports next to the completion time): algorithm
    bandwidth nbytes / seconds times 2(p-1)/p for all-reduce, (p-1)/p for
    reduce-scatter and all-gather (nbytes = the full buffer per endpoint),
    and (p-1)/p for all-to-all with nbytes per ordered pair (p * nbytes per
    endpoint).  With seconds in cycles the result is in bits per cycle."""
    kind = _BUS_FACTOR[int(coll)]
    per_ep = nbytes * p if kind == "a2a" else nbytes
    factor = 2.0 * (p - 1) / p if kind == "ar" else (p - 1) / p
    return 8.0 * per_ep / seconds * factor


# ---------------------------------------------------------------- C-ABI names

def sim_create(n_nodes, n_endpoints, row_ptr, col_idx, n_scenarios, bw, lat, cap, arb):
    arrs = [np.ascontiguousarray(a, np.int32) for a in (row_ptr, col_idx, bw, lat, cap)]
    ctx = C.c_void_p()
    st = lib().sim_create(n_nodes, n_endpoints, _ptr(arrs[0]), _ptr(arrs[1]), n_scenarios,
                          _ptr(arrs[2]), _ptr(arrs[3]), _ptr(arrs[4]), arb, C.byref(ctx))
    _check(None, st)
    return ctx


def sim_set_credit(ctx, credit=None):
    c = None if credit is None else np.ascontiguousarray(credit, np.int32)
    _check(ctx, lib().sim_set_credit(ctx, _ptr(c)))


def sim_load_collective(ctx, coll, nbytes, group_size=0, order=None, dep=0):
    o = None if order is None else np.ascontiguousarray(order, np.int32)
    _check(ctx, lib().sim_load_collective(ctx, coll, nbytes, group_size, _ptr(o), dep))


def sim_load_transactions(ctx, src, dst, pred_ptr, pred_idx):
    src = np.ascontiguousarray(src, np.int32)
    dst = np.ascontiguousarray(dst, np.int32)
    pptr = np.ascontiguousarray(pred_ptr, np.int64)
    pidx = np.ascontiguousarray(pred_idx, np.int64)
    if pidx.size == 0:
        pidx = np.zeros(1, np.int64)
    _check(ctx, lib().sim_load_transactions(ctx, len(src), _ptr(src), _ptr(dst), _ptr(pptr), _ptr(pidx)))


def sim_load_memcpy(ctx, cu, src_space, dst_space, src_line, dst_line, n_lines, space_channels, n_ch,
                    unroll, window):
    a32 = [np.ascontiguousarray(v, np.int32) for v in (cu, src_space, dst_space)]
    a64 = [np.ascontiguousarray(v, np.int64) for v in (src_line, dst_line, n_lines)]
    ch = np.ascontiguousarray(space_channels, np.int32)
    n_spaces = len(ch) // n_ch if n_ch > 0 else 0
    _check(ctx, lib().sim_load_memcpy(ctx, len(a32[0]), *(_ptr(v) for v in a32), *(_ptr(v) for v in a64),
                                      n_spaces, n_ch, _ptr(ch), unroll, window))


SIM_OP_COPY, SIM_OP_RELEASE, SIM_OP_ACQUIRE = 0, 1, 2


def sim_load_gpu_ops(ctx, kind, cu, src_ptr, src_space, src_line, dst_space, dst_line, n_lines, space_channels,
                     n_ch, unroll, window):
    k32 = [np.ascontiguousarray(v, np.int32) for v in (kind, cu)]
    sp = np.ascontiguousarray(src_ptr, np.int64)
    ssp = np.ascontiguousarray(src_space, np.int32)
    sln = np.ascontiguousarray(src_line, np.int64)
    if ssp.size == 0:
        ssp, sln = np.zeros(1, np.int32), np.zeros(1, np.int64)
    dsp = np.ascontiguousarray(dst_space, np.int32)
    a64 = [np.ascontiguousarray(v, np.int64) for v in (dst_line, n_lines)]
    ch = np.ascontiguousarray(space_channels, np.int32)
    n_spaces = len(ch) // n_ch if n_ch > 0 else 0
    if len(sp) != len(k32[0]) + 1:
        raise ValueError("src_ptr needs n_ops + 1 entries")
    _check(ctx, lib().sim_load_gpu_ops(ctx, len(k32[0]), *(_ptr(v) for v in k32), _ptr(sp), _ptr(ssp), _ptr(sln),
                                       _ptr(dsp), *(_ptr(v) for v in a64), n_spaces, n_ch, _ptr(ch), unroll,
                                       window))


def sim_sizes(ctx):
    T, m, S, lh = C.c_int64(), C.c_int32(), C.c_int32(), C.c_uint64()
    _check(ctx, lib().sim_sizes(ctx, C.byref(T), C.byref(m), C.byref(S), C.byref(lh)))
    return T.value, m.value, S.value, lh.value


def sim_run(ctx, stream_ptr, d_completion, d_tx_lines, d_busy_cycles, d_makespan, max_cycles=0):
    """Enqueue a run; the buffers are raw device addresses (ints)."""
    _check(ctx, lib().sim_run(ctx, C.c_void_p(stream_ptr), C.c_void_p(d_completion),
                              C.c_void_p(d_tx_lines), C.c_void_p(d_busy_cycles),
                              C.c_void_p(d_makespan), max_cycles))


def sim_run_noalloc(ctx, stream_ptr, d_completion, d_tx_lines, d_busy_cycles, d_makespan, max_cycles=0):
    """sim_run with the engines' scratch in the library's fixed device array
    (no device allocation)."""
    _check(ctx, lib().sim_run_noalloc(ctx, C.c_void_p(stream_ptr), C.c_void_p(d_completion),
                                      C.c_void_p(d_tx_lines), C.c_void_p(d_busy_cycles),
                                      C.c_void_p(d_makespan), max_cycles))


def sim_status_after_sync(ctx, n_scenarios):
    st = np.zeros(n_scenarios, np.int32)
    cyc = np.zeros(n_scenarios, np.uint64)
    rc = lib().sim_status_after_sync(ctx, _ptr(st), _ptr(cyc))
    return rc, st, cyc


def sim_route(ctx, src, dst, cap=256):
    out = np.zeros(cap, np.int32)
    n = C.c_int32()
    _check(ctx, lib().sim_route(ctx, src, dst, _ptr(out), cap, C.byref(n)))
    return out[:n.value].copy()


def sim_txn_info(ctx, x):
    """(src, dst, phase_step, line) of line id x of the loaded workload."""
    v = [C.c_int32() for _ in range(4)]
    _check(ctx, lib().sim_txn_info(ctx, x, *(C.byref(a) for a in v)))
    return tuple(a.value for a in v)


def sim_last_error(ctx) -> str:
    return lib().sim_last_error(ctx).decode()


def sim_destroy(ctx):
    lib().sim_destroy(ctx)


# ---------------------------------------------------------------- convenience

@dataclass
class RunResult:
    completion: "object"   # torch.uint32-compatible int32 tensor [S, T] on the device
    tx_lines: "object"     # int64 tensor [S, m]
    busy_cycles: "object"  # int64 tensor [S, m]
    makespan: "object"     # int32 tensor [S]
    status: int
    scenario_status: np.ndarray
    cycles: np.ndarray


class Simulator:
    """One context: a topology with S scenarios plus a loaded workload."""

    def __init__(self, n_nodes, n_endpoints, row_ptr, col_idx, bw, lat, cap, arb, n_scenarios=1):
        self.ctx = sim_create(n_nodes, n_endpoints, row_ptr, col_idx, n_scenarios, bw, lat, cap, arb)
        self.S = n_scenarios

    @classmethod
    def from_workload(cls, w):
        sim = cls(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb,
                  w.n_scenarios)
        if w.credit is not None:
            sim.set_credit(w.credit)
        if w.meta.get("memcpy") is not None:
            sim.load_memcpy(w.meta["memcpy"])
        elif w.coll >= 0:
            sim.load_collective(w.coll, w.bytes, w.group_size, w.order, w.dep)
        return sim

    def load_collective(self, coll, nbytes, group_size=0, order=None, dep=0):
        sim_load_collective(self.ctx, coll, nbytes, group_size, order, dep)

    def set_credit(self, credit=None):
        """Per-link credit return delays [S*m] (None: all 1); load again after."""
        sim_set_credit(self.ctx, credit)

    def load_transactions(self, src, dst, pred_ptr, pred_idx):
        sim_load_transactions(self.ctx, src, dst, pred_ptr, pred_idx)

    def load_memcpy(self, mc):
        """GPU programs (fields of ``sim_inputs.noc.Memcpy``): plain memcpy
        programs, or copies, reduces, releases and acquires when ``kind``
        is set."""
        if mc.kind is None:
            sim_load_memcpy(self.ctx, mc.cu, mc.src_space, mc.dst_space, mc.src_line, mc.dst_line, mc.n_lines,
                            mc.space_channels, mc.n_ch, mc.unroll, mc.window)
        else:
            sim_load_gpu_ops(self.ctx, mc.kind, mc.cu, mc.src_ptr, mc.src_space, mc.src_line, mc.dst_space,
                             mc.dst_line, mc.n_lines, mc.space_channels, mc.n_ch, mc.unroll, mc.window)

    def sizes(self):
        return sim_sizes(self.ctx)

    def route(self, src, dst):
        return sim_route(self.ctx, src, dst)

    def txn_info(self, x):
        return sim_txn_info(self.ctx, x)

    def alloc_outputs(self, device="cuda"):
        import torch
        T, m, S, _ = self.sizes()
        return (torch.empty((S, max(T, 1)), dtype=torch.int32, device=device),
                torch.empty((S, m), dtype=torch.int64, device=device),
                torch.empty((S, m), dtype=torch.int64, device=device),
                torch.empty((S,), dtype=torch.int32, device=device))

    def enqueue(self, outs, stream=None, max_cycles=0):
        import torch
        s = stream if stream is not None else torch.cuda.current_stream()
        comp, tx, busy, mk = outs
        sim_run(self.ctx, s.cuda_stream, comp.data_ptr(), tx.data_ptr(), busy.data_ptr(),
                mk.data_ptr(), max_cycles)

    def run(self, max_cycles=0, outs=None) -> RunResult:
        import torch
        outs = outs if outs is not None else self.alloc_outputs()
        self.enqueue(outs, max_cycles=max_cycles)
        torch.cuda.current_stream().synchronize()
        rc, st, cyc = sim_status_after_sync(self.ctx, self.S)
        comp, tx, busy, mk = outs
        return RunResult(comp, tx, busy, mk, rc, st, cyc)

    def close(self):
        if self.ctx:
            sim_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
