"""Seeded mixed-feature parity cases: each draws a topology, a workload (a
collective in either dependency mode, a random DAG, or memcpy programs on a
small NoC), an arbitration setting (lowest id / round-robin, with or without
class-fair turns), optional credit delays and an engine (the default choice
or one forced at random; an engine that declines the case is skipped), and
compares every output with the CPU oracle.  Features that are rare in the
targeted tests meet here."""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from sim_inputs import noc
from tests.test_gpu_parity import ENGINES, check_engine, simmod, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

COLLS = [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE, si.COLL_ALLTOALL, si.COLL_RING_ALLGATHER,
         si.COLL_RING_REDUCESCATTER, si.COLL_DIRECT_ALLGATHER, si.COLL_DIRECT_REDUCESCATTER,
         si.COLL_RHD_ALLREDUCE, si.COLL_DBT_ALLREDUCE]


def draw(seed):
    rng = np.random.default_rng(50_000 + seed)
    kind = rng.choice(["torus", "mesh", "fat", "dag", "noc"], p=[0.3, 0.15, 0.15, 0.25, 0.15])
    txns = None
    if kind == "torus":
        X, Y = [(2, 2), (4, 2), (4, 4), (3, 3)][int(rng.integers(0, 4))]
        coll = int(rng.choice(COLLS))
        if coll == si.COLL_RHD_ALLREDUCE and (X * Y) & (X * Y - 1):
            coll = si.COLL_DBT_ALLREDUCE
        w = si.torus2d(X, Y, n_scenarios=int(rng.integers(1, 6)), seed=int(rng.integers(0, 1 << 30)),
                       bws=tuple(int(b) for b in rng.choice([1, 2, 3, 4, 8], size=2)), lat_lo=1,
                       lat_hi=int(rng.integers(2, 30)), depths=tuple(int(c) for c in rng.integers(1, 20, size=3)),
                       nbytes=128 * X * Y * int(rng.integers(1, 5)) * 2, coll=coll)
        w.dep = int(rng.integers(0, 2)) if coll != si.COLL_ALLTOALL else 0
        if coll == si.COLL_RHD_ALLREDUCE and rng.integers(0, 2) and (X, Y) == (4, 4):
            w.order = si.gray_torus_order(4, 4)
    elif kind == "mesh":
        p = int(rng.integers(2, 7))
        coll = int(rng.choice(COLLS))
        if coll == si.COLL_RHD_ALLREDUCE and p & (p - 1):
            coll = si.COLL_RING_ALLGATHER
        b = int(rng.integers(1, 5))
        L = int(rng.integers(1, 12))
        w = si.full_mesh(p, b=b, L=L, cap=int(rng.integers(1, b * (L + 1) + 2)), coll=coll,
                         nbytes=128 * p * 2 * int(rng.integers(1, 6)))
        w.dep = int(rng.integers(0, 2)) if coll != si.COLL_ALLTOALL else 0
    elif kind == "fat":
        w = si.fat_tree(4, nbytes=128 * 16 * int(rng.integers(1, 3)), cap=int(rng.integers(2, 9)), lat_lo=1,
                        lat_hi=int(rng.integers(2, 12)), coll=int(rng.choice([si.COLL_ALLTOALL, si.COLL_RING_ALLREDUCE,
                                                                              si.COLL_DBT_ALLREDUCE])))
    elif kind == "dag":
        n_end = int(rng.integers(2, 7))
        S = int(rng.integers(1, 4))
        n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 4)), int(rng.integers(0, 6)),
                                                  bmax=int(rng.choice([1, 2, 4, 8])), Lmax=5, capmax=9, S=S)
        txns = si.random_dag(rng, n_end, int(rng.integers(1, 250)), max_preds=3)
        w = si.Workload(f"dag{seed}", n, n_end, rp, ci, S, bw, lat, cap, 0, -1, 0)
    else:
        w0, lay = noc.gpu_noc(1, mesh=(2, 2), cus_per_router=2, ch_per_router=2, ports_per_router=1,
                              noc=(int(rng.integers(1, 5)), 1, 8), cu_out=(int(rng.integers(1, 3)), 1, 4),
                              mem=(1, int(rng.integers(1, 4)), 4))
        rows = [(int(rng.choice(lay.cus[0])), 0, 0, int(rng.integers(0, 20)), 40 + int(rng.integers(0, 20)),
                 int(rng.integers(0, 8))) for _ in range(int(rng.integers(1, 7)))]
        w = noc.memcpy_workload(w0, noc._ops(rows, lay, int(rng.integers(1, 5)), int(rng.integers(1, 9))))
    w.arb = int(rng.integers(0, 2)) | (si.ARB_FAIR_CLASSES if rng.random() < 0.2 else 0)
    if rng.random() < 0.3:
        w.credit = rng.integers(1, 8, size=len(w.bw)).astype(np.int32)
    engine = str(rng.choice(ENGINES)) if rng.random() < 0.6 else None
    return w, txns, engine


@pytest.mark.parametrize("seed", range(150))
def test_fuzz(simmod, oracle_lib, seed):
    w, txns, engine = draw(seed)
    check_engine(simmod, oracle_lib, w, engine or "", txns=txns)
