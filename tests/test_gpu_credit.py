"""GPU parity of the credit-delay flow-control variant against the CPU
oracle, through the C ABI (the workgroup engine simulates delays above 1;
the other engines decline them)."""
from __future__ import annotations

import numpy as np
import pytest

import sim_inputs as si
from tests.test_gpu_parity import ENGINES, check_engine, check_vs_oracle, simmod, torch_cuda, say  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("seed", range(16))
def test_credit_random_dags(simmod, oracle_lib, engine, seed):
    rng = np.random.default_rng(11000 + seed)
    n_end = int(rng.integers(2, 6))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 3)), int(rng.integers(0, 5)),
                                              bmax=3, Lmax=4, capmax=5, S=2)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 200)), max_preds=3)
    w = si.Workload("rand_credit", n, n_end, rp, ci, 2, bw, lat, cap, seed % 2, -1, 0)
    w.credit = rng.integers(1, 6, size=len(bw)).astype(np.int32)
    check_engine(simmod, oracle_lib, w, engine, txns=(src, dst, pptr, pidx))


@pytest.mark.parametrize("coll", [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE, si.COLL_RHD_ALLREDUCE,
                                  si.COLL_DBT_ALLREDUCE])
@pytest.mark.parametrize("dep", [0, 1])
def test_credit_torus(simmod, oracle_lib, coll, dep):
    w = si.torus2d(4, 4, n_scenarios=6, seed=150 + coll + 10 * dep, bws=(1, 2, 4), lat_lo=1, lat_hi=20,
                   depths=(2, 3, 7, 32), nbytes=128 * 16 * 4, coll=coll, arb=(coll + dep) % 2)
    w.dep = dep
    w.credit = np.random.default_rng(coll).integers(1, 12, size=len(w.bw)).astype(np.int32)
    # direct and RHD in rank order deadlock in most of these scenarios (two-hop
    # partners on small buffers), with or without delays; those are compared
    # up to the deadlock
    check_vs_oracle(simmod, oracle_lib, w, expect_ok=False)


def test_credit_equal_to_latency_full_size_sample(simmod, oracle_lib):
    """Full-size 4x4 torus scenarios with every credit delay equal to its
    link's latency (credits travel back over the link)."""
    w = si.take_scenarios(si.config("C5"), [0, 1, 2, 1000, 4095])
    w.credit = w.lat.copy()
    say("C5-sized, credit = latency: 5 scenarios")
    check_vs_oracle(simmod, oracle_lib, w)


def test_credit_reset_restores_base_model(simmod, oracle_lib):
    w = si.torus2d(4, 4, n_scenarios=3, seed=9, bws=(1, 2), lat_lo=1, lat_hi=9, depths=(2, 5), nbytes=128 * 16 * 2)
    s = simmod.Simulator(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb, w.n_scenarios)
    try:
        s.set_credit(np.full(len(w.bw), 3, np.int32))
        with pytest.raises(simmod.SimError) as e:
            s.run()
        assert e.value.status == simmod.SIM_ERR_STATE
        s.load_collective(w.coll, w.bytes)
        a = s.run()
        s.set_credit(None)
        s.load_collective(w.coll, w.bytes)
        b = s.run()
    finally:
        s.close()
    for k in range(w.n_scenarios):
        base = oracle_lib.simulate_workload(w, k)
        comp = b.completion[k, :len(base.completion)].cpu().numpy().view(np.uint32)
        assert np.array_equal(comp, base.completion)
    assert a.status == 0


@pytest.mark.parametrize("arb", [0, 1])
@pytest.mark.parametrize("bws", [(1,), (1, 2, 4), (8,), (2, 8)])
def test_credit_wave_torus(simmod, oracle_lib, arb, bws):
    """The wave engine's b = 1 loop and its general loop with delays."""
    w = si.torus2d(4, 4, n_scenarios=13, seed=170 + arb + len(bws), bws=bws, lat_lo=1, lat_hi=25,
                   depths=(1, 2, 3, 7, 32), nbytes=128 * 16 * 6, arb=arb)
    w.credit = np.random.default_rng(arb + 7 * len(bws)).integers(1, 14, size=len(w.bw)).astype(np.int32)
    check_engine(simmod, oracle_lib, w, "wave", must_run=True)


@pytest.mark.parametrize("engine", ["wave", "workgroup", "workgroup_scan", "resident"])
def test_credit_wave_full_size_sample(simmod, oracle_lib, engine):
    w = si.take_scenarios(si.config("C5"), [3, 7, 2048, 4000])
    w.credit = w.lat.copy()
    check_engine(simmod, oracle_lib, w, engine, must_run=True)


def test_credit_with_chunk_dependencies_not_on_wave(simmod, oracle_lib):
    # the wave engine has no instantiation for both: the workgroup engine runs it
    w = si.torus2d(4, 4, n_scenarios=3, seed=5, bws=(1, 2), lat_lo=1, lat_hi=9, depths=(2, 5), nbytes=128 * 16 * 2)
    w.dep = si.DEP_CHUNK
    w.credit = np.full(len(w.bw), 4, np.int32)
    check_vs_oracle(simmod, oracle_lib, w)
    with pytest.raises(pytest.skip.Exception):
        check_engine(simmod, oracle_lib, w, "wave")


@pytest.mark.parametrize("arb", [0, 1])
@pytest.mark.parametrize("seed", range(8))
def test_windowed_grid(simmod, oracle_lib, arb, seed):
    """The grid engine's windowed form: one-line-per-cycle graphs whose links
    all have latency and credit delay of at least 2 (a k = 4 fat tree, or a
    one-scenario torus), delays below, at and above the latency; every line,
    counter and the makespan against the oracle."""
    rng = np.random.default_rng(13000 + seed)
    if seed % 2 == 0:
        w = si.fat_tree(4, lat_seed=seed, lat_lo=2, lat_hi=int(rng.integers(3, 16)), cap=int(rng.integers(2, 9)),
                        nbytes=128 * 16 * int(rng.integers(1, 4)), arb=arb,
                        coll=int(rng.choice([si.COLL_ALLTOALL, si.COLL_ALLTOALL])))
    else:
        # shallow buffers deadlock this all-to-all (both sides must stop at the
        # same point); deep ones finish
        w = si.torus2d(4, 4, n_scenarios=1, seed=seed, bws=(1, 1), lat_lo=2, lat_hi=int(rng.integers(3, 12)),
                       depths=(2, 4, 9) if seed < 4 else (24, 32, 48), nbytes=128 * 16 * 2, coll=si.COLL_ALLTOALL,
                       arb=arb)
    lo = np.maximum(2, w.lat - 3)
    w.credit = rng.integers(lo, w.lat + 4).astype(np.int32)
    check_engine(simmod, oracle_lib, w, "grid", must_run=True)


@pytest.mark.parametrize("stride", [1, 8])
@pytest.mark.parametrize("seed", [0, 2])
def test_windowed_grid_placement(simmod, oracle_lib, stride, seed, monkeypatch):
    """The windowed form with its workgroups launched as consecutive blocks
    (spread over the dies) or every eighth block: the same bytes."""
    monkeypatch.setenv("SIMGPU_GRID_STRIDE", str(stride))
    monkeypatch.setenv("SIMGPU_GRID_WGS", "32")
    rng = np.random.default_rng(14000 + seed)
    w = si.fat_tree(4, lat_seed=seed, lat_lo=2, lat_hi=int(rng.integers(3, 16)), cap=int(rng.integers(2, 9)),
                    nbytes=128 * 16 * 3, arb=seed % 2, coll=si.COLL_ALLTOALL)
    w.credit = rng.integers(np.maximum(2, w.lat - 2), w.lat + 3).astype(np.int32)
    check_engine(simmod, oracle_lib, w, "grid", must_run=True)
