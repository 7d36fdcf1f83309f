"""GPU parity: libsimgpu (HIP kernels, called through the C ABI) against the
CPU oracle, bit for bit.

Small and scaled cases run the oracle in the test and compare every
completion cycle, tx_lines, busy_cycles and makespan.  The five full-size
workloads compare SHA-256 digests of the complete outputs (and a sample of
values) with ``tests/golden/*.json``, which tests/golden/make_golden.py
wrote by running the oracle alone.
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import sim_inputs as si

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


@pytest.fixture(scope="module")
def simmod(torch_cuda):
    from paper_2606_10440_amd import sim
    sim.lib()  # raises if the library was not built
    return sim


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def run_gpu(simmod, w, max_cycles=0, txns=None):
    s = simmod.Simulator(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb,
                         w.n_scenarios)
    if w.credit is not None:
        s.set_credit(w.credit)
    if txns is not None:
        s.load_transactions(*txns)
    elif w.meta.get("memcpy") is not None:
        s.load_memcpy(w.meta["memcpy"])
    else:
        s.load_collective(w.coll, w.bytes, w.group_size, w.order, w.dep)
    r = s.run(max_cycles=max_cycles)
    s.close()
    return r


def compare_scenario(r, s, want, T):
    assert want.status_name == "OK"
    assert r.scenario_status[s] == 0
    comp = r.completion[s, :T].cpu().numpy().view(np.uint32)
    bad = np.nonzero(comp != want.completion)[0]
    assert bad.size == 0, f"scenario {s}: {bad.size} completions differ, first id {bad[:5]} " \
                          f"gpu {comp[bad[:5]]} oracle {want.completion[bad[:5]]}"
    assert np.array_equal(r.tx_lines[s].cpu().numpy().astype(np.uint64), want.tx_lines)
    assert np.array_equal(r.busy_cycles[s].cpu().numpy().astype(np.uint64), want.busy_cycles)
    assert int(r.makespan[s].item()) == want.makespan


def compare_deadlocked(r, s, want):
    """Same status, same counters, same cycle for every line that completed."""
    assert r.scenario_status[s] == 7
    comp = r.completion[s, :len(want.completion)].cpu().numpy().view(np.uint32)
    done = want.completion != 0xFFFFFFFF
    assert np.array_equal(comp[done], want.completion[done])
    assert np.array_equal(r.tx_lines[s].cpu().numpy().astype(np.uint64), want.tx_lines)
    assert np.array_equal(r.busy_cycles[s].cpu().numpy().astype(np.uint64), want.busy_cycles)


def first_divergence(simmod, oracle_lib, w, s, txns=None):
    """Locate a mismatch: the smallest max_cycles bound at which the GPU and
    the oracle differ for scenario s (bisection), with the first lines and
    links that differ there."""
    m = w.n_links
    sl = slice(s * m, (s + 1) * m)

    def both(mc):
        r = run_gpu(simmod, w, max_cycles=mc, txns=txns)
        if txns is None:
            o = oracle_lib.simulate_workload(w, s, max_cycles=mc)
        else:
            o = oracle_lib.simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw[sl], w.lat[sl], w.cap[sl],
                                    w.arb, txns=txns, max_cycles=mc,
                                    credit=None if w.credit is None else w.credit[sl])
        comp = r.completion[s, :len(o.completion)].cpu().numpy().view(np.uint32)
        done = o.completion != 0xFFFFFFFF
        lines = np.nonzero(done & (comp != o.completion))[0]
        links = np.nonzero(r.tx_lines[s].cpu().numpy().astype(np.uint64) != o.tx_lines)[0]
        return lines, links

    full = oracle_lib.simulate_workload(w, s) if txns is None else None
    lo, hi = 0, (full.makespan + 2) if full is not None and full.makespan else 1 << 20
    lines, links = both(hi)
    if not len(lines) and not len(links):
        return "no divergence found below the makespan"
    while hi - lo > 1:
        mid = (lo + hi) // 2
        ln, lk = both(mid)
        if len(ln) or len(lk):
            hi, lines, links = mid, ln, lk
        else:
            lo = mid
    return f"first divergence at max_cycles={hi}: lines {lines[:8].tolist()}, links {links[:8].tolist()}"


def check_vs_oracle(simmod, oracle_lib, w, scenarios=None, expect_ok=True):
    r = run_gpu(simmod, w)
    if expect_ok:
        assert r.status == 0, simmod.STATUS_NAMES[r.status]
    n_ok = 0
    for s in (range(w.n_scenarios) if scenarios is None else scenarios):
        want = oracle_lib.simulate_workload(w, s)
        try:
            if want.status_name == "DEADLOCK":
                compare_deadlocked(r, s, want)
            else:
                compare_scenario(r, s, want, len(want.completion))
                n_ok += 1
        except AssertionError as e:
            want_code = {"OK": 0, "DEADLOCK": 7}.get(want.status_name, -100)
            if int(r.scenario_status[s]) != want_code:  # no GPU re-runs for an engine error
                raise AssertionError(f"{e}\nscenario {s}: GPU status {int(r.scenario_status[s])}, "
                                     f"oracle {want.status_name}") from None
            raise AssertionError(f"{e}\n{first_divergence(simmod, oracle_lib, w, s)}") from None
    return r, n_ok


# ----------------------------------------------------------------- small cases

def test_c1_full(simmod, oracle_lib):
    r, _ = check_vs_oracle(simmod, oracle_lib, si.config("C1"))
    assert int(r.makespan[0]) == 266


def test_c2_full(simmod, oracle_lib):
    w = si.config("C2")
    r, _ = check_vs_oracle(simmod, oracle_lib, w)
    ids = np.arange(r.completion.shape[1], dtype=np.int64)
    comp = r.completion[0].cpu().numpy().view(np.uint32)
    assert np.array_equal(comp, 16384 * (ids // (16384 * 8)) + ids % 16384 + 51)


@pytest.mark.parametrize("p,C,b,L,coll", [(3, 5, 1, 4, 0), (4, 8, 2, 3, 0), (5, 10, 1, 7, 1), (4, 6, 3, 2, 1),
                                          (2, 9, 1, 1, 0), (6, 12, 2, 20, 1)])
def test_mesh_collectives(simmod, oracle_lib, p, C, b, L, coll):
    w = si.full_mesh(p, b=b, L=L, cap=max(1, b * (L + 1) // 2), coll=coll, nbytes=128 * C * p)
    check_vs_oracle(simmod, oracle_lib, w)


@pytest.mark.parametrize("seed", range(60))
def test_random_dags(simmod, oracle_lib, seed):
    rng = np.random.default_rng(1000 + seed)
    n_end = int(rng.integers(2, 7))
    S = int(rng.integers(1, 4))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 4)), int(rng.integers(0, 6)),
                                              bmax=4, Lmax=5, capmax=6, S=S)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 300)), max_preds=3)
    arb = seed % 2
    w = si.Workload("rand", n, n_end, rp, ci, S, bw, lat, cap, arb, -1, 0)
    say(f"random dag seed={seed} n={n} E={n_end} S={S} T={len(src)} arb={arb}")
    r = run_gpu(simmod, w, txns=(src, dst, pptr, pidx))
    m = int(rp[-1])
    for s in range(S):
        want = oracle_lib.simulate(n, n_end, rp, ci, bw[s * m:(s + 1) * m], lat[s * m:(s + 1) * m],
                                   cap[s * m:(s + 1) * m], arb, txns=(src, dst, pptr, pidx))
        if want.status_name == "DEADLOCK":
            compare_deadlocked(r, s, want)
            continue
        compare_scenario(r, s, want, len(src))


@pytest.mark.parametrize("k,nbytes,cap,lo,hi", [(4, 128 * 16, 5, 2, 9), (6, 128 * 4, 8, 5, 30),
                                                (8, 128 * 2, 32, 100, 300)])
def test_small_fat_trees(simmod, oracle_lib, k, nbytes, cap, lo, hi):
    w = si.fat_tree(k, nbytes=nbytes, cap=cap, lat_lo=lo, lat_hi=hi)
    check_vs_oracle(simmod, oracle_lib, w)


def test_scaled_hierarchical(simmod, oracle_lib):
    w = si.scaled(si.config("C3"), bytes=128 * 64 * 8 * 3)
    check_vs_oracle(simmod, oracle_lib, w)


def test_scaled_hierarchical_small_domains(simmod, oracle_lib):
    w = si.domains_leaf_spine(G=3, M=4, n_leaf=3, n_spine=2, intra=(2, 3, 4), fabric=(1, 7, 6),
                              nbytes=128 * 12 * 5)
    check_vs_oracle(simmod, oracle_lib, w)


def test_batched_torus_subset(simmod, oracle_lib):
    w = si.take_scenarios(si.config("C5"), range(24))
    w = si.scaled(w, bytes=128 * 16 * 64)
    check_vs_oracle(simmod, oracle_lib, w)


def test_batched_more_waves_than_simds(simmod, oracle_lib):
    # 6000 scenarios of a 3x3 torus need more wavefronts than the device has
    # SIMDs, so the shortest share SIMDs in pairs; every bandwidth class and
    # ring size mixes in the placement.  A spread sample is checked line by
    # line, the rest by status.
    w = si.torus2d(3, 3, n_scenarios=6000, seed=23, bws=(1, 2, 4), lat_lo=1, lat_hi=24,
                   depths=(16, 32, 64), nbytes=128 * 9 * 6)
    sample = sorted({0, 1, 2, 5999, 5998} | set(range(7, 6000, 251)))
    say(f"6000-scenario torus: checking {len(sample)} scenarios against the oracle")
    r, n_ok = check_vs_oracle(simmod, oracle_lib, w, scenarios=sample)
    assert n_ok == len(sample)
    assert (r.scenario_status == 0).all()


@pytest.mark.parametrize("arb,coll,depths,nbytes", [(0, si.COLL_DIRECT_ALLREDUCE, (8, 13, 16, 32), 128 * 120),
                                                    (1, si.COLL_ALLTOALL, (8, 13, 16, 32), 128 * 3),
                                                    (1, si.COLL_ALLTOALL, (16, 32, 64), 128 * 8),
                                                    (1, si.COLL_DIRECT_ALLREDUCE, (1, 2, 3, 7, 16), 128 * 120),
                                                    (0, si.COLL_ALLTOALL, (1, 2, 3, 7, 16), 128 * 3)])
def test_torus_random_params(simmod, oracle_lib, arb, coll, depths, nbytes):
    # A torus with wrap links has cyclic buffer dependencies: with tiny
    # buffers many scenarios deadlock, which must be detected identically.
    w = si.torus2d(4, 3, n_scenarios=40, seed=11 + arb + 2 * coll, bws=(1, 2, 3, 4), lat_lo=1, lat_hi=12,
                   depths=depths, nbytes=nbytes, arb=arb, coll=coll)
    r, n_ok = check_vs_oracle(simmod, oracle_lib, w, expect_ok=False)
    if depths[0] >= 8:
        assert n_ok > 0


# ----------------------------------------------------------------- error paths

def test_deadlock_detected(simmod, oracle_lib):
    rp = np.array([0, 1, 2, 3], np.int32)
    ci = np.array([1, 2, 0], np.int32)
    one = np.ones(3, np.int32)
    src = np.array([0, 1, 2] * 4, np.int32)
    dst = np.array([2, 0, 1] * 4, np.int32)
    pptr = np.zeros(13, np.int64)
    w = si.Workload("ring3", 3, 3, rp, ci, 1, one, one, one, 0, -1, 0)
    want = oracle_lib.simulate(3, 3, rp, ci, one, one, one, 0, txns=(src, dst, pptr, np.zeros(0, np.int64)))
    assert want.status_name == "DEADLOCK"
    r = run_gpu(simmod, w, txns=(src, dst, pptr, np.zeros(0, np.int64)))
    assert r.status == simmod.SIM_ERR_DEADLOCK and r.scenario_status[0] == 7


def test_cyclic_predecessors_deadlock(simmod):
    rp = np.array([0, 1, 2, 3], np.int32)
    ci = np.array([1, 2, 0], np.int32)
    four = np.full(3, 4, np.int32)
    w = si.Workload("ring3", 3, 3, rp, ci, 1, four, four, four, 0, -1, 0)
    r = run_gpu(simmod, w, txns=(np.array([0, 1]), np.array([1, 2]), np.array([0, 1, 2]), np.array([1, 0])))
    assert r.status == simmod.SIM_ERR_DEADLOCK


def test_max_cycles_guard(simmod):
    w = si.config("C1")
    assert run_gpu(simmod, w, max_cycles=100).status == simmod.SIM_ERR_MAX_CYCLES
    r = run_gpu(simmod, w, max_cycles=265)
    assert r.status == 0 and int(r.makespan[0]) == 266


def test_empty_workload(simmod):
    w = si.config("C1")
    r = run_gpu(simmod, w, txns=(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(1, np.int64),
                                 np.zeros(0, np.int64)))
    assert r.status == 0 and int(r.makespan[0]) == 0
    assert int(r.tx_lines.sum()) == 0


def test_deterministic_repeat(simmod):
    w = si.take_scenarios(si.config("C5"), range(64))
    w = si.scaled(w, bytes=128 * 16 * 32)
    s = simmod.Simulator.from_workload(w)
    a = s.run()
    ca = a.completion.clone()
    b = s.run()
    s.close()
    assert a.status == b.status == 0
    assert bool((ca == b.completion).all())


@pytest.mark.parametrize("engine,threads", [("lane", (64, 256, 1024)), ("lanehbm", (64, 512)),
                                            ("wave", (None,)), ("workgroup", (None,))])
def test_launch_geometry_same_bytes(simmod, engine, threads):
    """One workload on every engine, and on the lane engines at several
    workgroup sizes: the outputs are the same bytes."""
    w = si.torus2d(4, 4, n_scenarios=6, seed=77, bws=(1, 2, 4), lat_lo=1, lat_hi=20, depths=(3, 16),
                   nbytes=128 * 16 * 8, arb=1)
    ref = run_engine(simmod, w, "workgroup")
    assert ref.status == 0
    want = [t.cpu().numpy() for t in (ref.completion, ref.tx_lines, ref.busy_cycles, ref.makespan)]
    for th in threads:
        old = os.environ.get("SIMGPU_LANE_THREADS")
        if th is not None:
            os.environ["SIMGPU_LANE_THREADS"] = str(th)
        try:
            r = run_engine(simmod, w, engine)
        finally:
            if old is None:
                os.environ.pop("SIMGPU_LANE_THREADS", None)
            else:
                os.environ["SIMGPU_LANE_THREADS"] = old
        assert r.status == 0
        got = [t.cpu().numpy() for t in (r.completion, r.tx_lines, r.busy_cycles, r.makespan)]
        for a, b in zip(want, got):
            assert a.tobytes() == b.tobytes(), (engine, th)


# ----------------------------------------------------------------- full size

def _digest(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def _golden(name):
    with open(os.path.join(HERE, "golden", f"{name}.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C1_chunk", "C2_chunk"])
def test_full_size_digest(simmod, torch_cuda, name):
    g = _golden(name)
    w = si.config(name)
    say(f"full-size {name}: running on GPU")
    r = run_gpu(simmod, w)
    assert r.status == 0
    comp = r.completion[0].cpu().numpy().view(np.uint32)
    idx = np.array(g["sample_idx"])
    assert np.array_equal(comp[idx].astype(np.int64), np.array(g["sample_completion"]))
    assert int(r.makespan[0]) == g["makespan"][0]
    assert _digest(comp.astype("<u4")) == g["completion_sha256"][0]
    assert _digest(r.tx_lines[0].cpu().numpy().astype("<u8")) == g["tx_lines_sha256"][0]
    assert _digest(r.busy_cycles[0].cpu().numpy().astype("<u8")) == g["busy_cycles_sha256"][0]


@pytest.mark.parametrize("name,engine", [("C5", None), ("C5_chunk", None), ("C5_rhd", None), ("C5_dbt", None),
                                         ("C5_ag", None), ("C5_credit", None), ("NOC2_ag", None),
                                         ("C5_credit", "resident"), ("C5_rhd", "resident"),
                                         ("NOC2_ag", "workgroup")])
def test_full_size_batched_digest(simmod, torch_cuda, name, engine, monkeypatch):
    """Every scenario of the batched workloads against the oracle's golden
    digests: on the engine the library picks, and on the LDS-resident and
    generic workgroup engines where another one is picked."""
    g = _golden(name)
    w = si.config(name)
    if engine:
        monkeypatch.setenv("SIMGPU_ENGINE", engine)
    say(f"full-size {name}: running {w.n_scenarios} scenarios on GPU ({engine or 'default engine'})")
    r = run_gpu(simmod, w)
    assert r.status == 0
    mk = r.makespan.cpu().numpy()
    assert np.array_equal(mk, np.array(g["makespan"]))
    tx = r.tx_lines.cpu().numpy().astype("<u8")
    busy = r.busy_cycles.cpu().numpy().astype("<u8")
    S = w.n_scenarios
    chunk = 256
    bad = []
    with ThreadPoolExecutor(16) as ex:
        for c0 in range(0, S, chunk):
            host = r.completion[c0:c0 + chunk].cpu().numpy().view(np.uint32)
            dig = list(ex.map(lambda i: _digest(host[i].astype("<u4")), range(host.shape[0])))
            for i, d in enumerate(dig):
                s = c0 + i
                if d != g["completion_sha256"][s] or _digest(tx[s]) != g["tx_lines_sha256"][s] or \
                        _digest(busy[s]) != g["busy_cycles_sha256"][s]:
                    bad.append(s)
    assert not bad, f"{len(bad)} scenarios differ, first {bad[:10]}"


# ----------------------------------------------------------------- every engine

ENGINES = ["workgroup", "workgroup_scan", "lane", "lanehbm", "b1", "wave", "grid", "resident"]


def run_engine(simmod, w, engine, txns=None, must_run=False):
    """Run with the engine forced; skip if the library refuses that engine
    for this workload (the wave engine's limits: at most 64 traffic links,
    four flows per link, three feeders per link), or fail if must_run (the
    engine is documented to take such workloads)."""
    old = os.environ.get("SIMGPU_ENGINE")
    if engine:
        os.environ["SIMGPU_ENGINE"] = engine
    else:  # the library's own choice
        os.environ.pop("SIMGPU_ENGINE", None)
    try:
        try:
            return run_gpu(simmod, w, txns=txns)
        except simmod.SimError as e:
            if e.status == simmod.SIM_ERR_INVALID_ARG and "SIMGPU_ENGINE" in str(e) and not must_run:
                pytest.skip(f"engine {engine} not usable for {w.name}")
            raise
    finally:
        if old is None:
            os.environ.pop("SIMGPU_ENGINE", None)
        else:
            os.environ["SIMGPU_ENGINE"] = old


def check_engine(simmod, oracle_lib, w, engine, txns=None, must_run=False):
    say(f"engine {engine}: {w.name} S={w.n_scenarios}")
    r = run_engine(simmod, w, engine, txns, must_run=must_run)
    m = w.n_links
    n_ok = 0
    for s in range(w.n_scenarios):
        sl = slice(s * m, (s + 1) * m)
        if txns is None:
            want = oracle_lib.simulate_workload(w, s)
        else:
            want = oracle_lib.simulate(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw[sl], w.lat[sl],
                                       w.cap[sl], w.arb, txns=txns,
                                       credit=None if w.credit is None else w.credit[sl])
        try:
            if want.status_name == "DEADLOCK":
                compare_deadlocked(r, s, want)
            else:
                compare_scenario(r, s, want, len(want.completion))
                n_ok += 1
        except AssertionError as e:
            # Bisect only when both sides ended the same way and only values
            # differ; an engine watchdog or internal error is reported as is
            # (its cause is found on the CPU, not by re-running the GPU case).
            want_code = {"OK": 0, "DEADLOCK": 7}.get(want.status_name, -100)
            if int(r.scenario_status[s]) != want_code:
                raise AssertionError(f"{e}\nscenario {s}: GPU status {int(r.scenario_status[s])}, "
                                     f"oracle {want.status_name}") from None
            old = os.environ.get("SIMGPU_ENGINE")
            if engine:
                os.environ["SIMGPU_ENGINE"] = engine
            else:
                os.environ.pop("SIMGPU_ENGINE", None)
            try:
                report = first_divergence(simmod, oracle_lib, w, s, txns)
            finally:
                if old is None:
                    os.environ.pop("SIMGPU_ENGINE", None)
                else:
                    os.environ["SIMGPU_ENGINE"] = old
            raise AssertionError(f"{e}\n{report}") from None
    return n_ok


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("arb", [0, 1])
def test_engines_fat_tree_b1(simmod, oracle_lib, engine, arb):
    w = si.fat_tree(4, nbytes=128 * 12, cap=5, lat_lo=2, lat_hi=9, arb=arb)
    assert check_engine(simmod, oracle_lib, w, engine) == 1


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("arb", [0, 1])
def test_engines_torus_ring_b1(simmod, oracle_lib, engine, arb):
    w = si.torus2d(4, 4, n_scenarios=6, seed=21 + arb, bws=(1,), lat_lo=1, lat_hi=30, depths=(2, 4, 32),
                   nbytes=128 * 16 * 20, arb=arb)
    check_engine(simmod, oracle_lib, w, engine)


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("seed", range(12))
def test_engines_random_dag_b1(simmod, oracle_lib, engine, seed):
    rng = np.random.default_rng(5000 + seed)
    n_end = int(rng.integers(2, 7))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 4)), int(rng.integers(0, 6)),
                                              bmax=1, Lmax=5, capmax=6, S=2)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 300)), max_preds=3)
    w = si.Workload("rand_b1", n, n_end, rp, ci, 2, bw, lat, cap, seed % 2, -1, 0)
    check_engine(simmod, oracle_lib, w, engine, txns=(src, dst, pptr, pidx))


@pytest.mark.parametrize("engine", ["workgroup", "workgroup_scan", "lane", "lanehbm", "wave", "resident"])
@pytest.mark.parametrize("seed", range(12))
def test_engines_random_dag_multirate(simmod, oracle_lib, engine, seed):
    rng = np.random.default_rng(6000 + seed)
    n_end = int(rng.integers(2, 7))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 4)), int(rng.integers(0, 6)),
                                              bmax=4, Lmax=5, capmax=6, S=2)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 300)), max_preds=3)
    w = si.Workload("rand_mr", n, n_end, rp, ci, 2, bw, lat, cap, seed % 2, -1, 0)
    check_engine(simmod, oracle_lib, w, engine, txns=(src, dst, pptr, pidx))


# ----------------------------------------------------------------- wave engine
# Several scenarios per wavefront, each with its own clock; scenarios are
# reordered across waves by expected length, so every scenario is compared.

@pytest.mark.parametrize("arb", [0, 1])
@pytest.mark.parametrize("coll", [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE])
@pytest.mark.parametrize("bws", [(1,), (1, 2, 4), (8,), (2, 8)])
def test_wave_torus_mixed(simmod, oracle_lib, arb, coll, bws):
    X = 4 if coll == si.COLL_RING_ALLREDUCE else 2  # direct on 4x4 puts more than four flows on a link
    w = si.torus2d(X, X, n_scenarios=13, seed=40 + arb + 2 * coll + len(bws), bws=bws, lat_lo=1, lat_hi=25,
                   depths=(1, 2, 3, 7, 32), nbytes=128 * X * X * 6, arb=arb, coll=coll)
    check_engine(simmod, oracle_lib, w, "wave")


@pytest.mark.parametrize("seed", range(24))
def test_wave_random_dags(simmod, oracle_lib, seed):
    """Small random graphs and DAGs, bandwidth up to 8, three scenarios."""
    rng = np.random.default_rng(7000 + seed)
    n_end = int(rng.integers(2, 5))
    n, rp, ci, bw, lat, cap = si.random_graph(rng, n_end, int(rng.integers(0, 3)), int(rng.integers(0, 4)),
                                              bmax=int(rng.choice([1, 2, 4, 8])), Lmax=4, capmax=9, S=3)
    src, dst, pptr, pidx = si.random_dag(rng, n_end, int(rng.integers(1, 250)), max_preds=3)
    w = si.Workload("rand_wave", n, n_end, rp, ci, 3, bw, lat, cap, seed % 2, -1, 0)
    check_engine(simmod, oracle_lib, w, "wave", txns=(src, dst, pptr, pidx))


# ----------------------------------------------------- per-chunk dependencies
# Every line of a step waits for the whole chunk of the step before (put +
# signal); the oracle releases them through per-chunk join counters, the
# engines through one delivered-count threshold per predecessor chunk.

@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("p,C,b,L,coll", [(3, 5, 1, 4, 0), (4, 8, 2, 3, 0), (5, 10, 1, 7, 1), (4, 6, 3, 2, 1),
                                          (2, 9, 1, 1, 0), (6, 12, 2, 20, 1), (5, 7, 1, 3, 3)])
def test_chunk_mesh(simmod, oracle_lib, engine, p, C, b, L, coll):
    w = si.full_mesh(p, b=b, L=L, cap=max(1, b * (L + 1) // 2), coll=coll, nbytes=128 * C * p)
    w.dep = si.DEP_CHUNK
    assert check_engine(simmod, oracle_lib, w, engine) == 1


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("arb", [0, 1])
@pytest.mark.parametrize("coll", [si.COLL_RING_ALLREDUCE, si.COLL_DIRECT_ALLREDUCE])
def test_chunk_torus(simmod, oracle_lib, engine, arb, coll):
    X = 4 if coll == si.COLL_RING_ALLREDUCE else 2
    bws = (1,) if engine == "b1" else (1, 2, 4)
    w = si.torus2d(X, X, n_scenarios=9, seed=80 + arb + 2 * coll, bws=bws, lat_lo=1, lat_hi=25,
                   depths=(1, 2, 3, 7, 32), nbytes=128 * X * X * 6, arb=arb, coll=coll)
    w.dep = si.DEP_CHUNK
    check_engine(simmod, oracle_lib, w, engine)


@pytest.mark.parametrize("engine", ENGINES)
def test_chunk_fat_tree(simmod, oracle_lib, engine):
    w = si.fat_tree(4, nbytes=128 * 16 * 3, cap=5, lat_lo=2, lat_hi=9, arb=1, coll=si.COLL_RING_ALLREDUCE)
    w.dep = si.DEP_CHUNK
    assert check_engine(simmod, oracle_lib, w, engine) == 1


def test_chunk_rejected_for_hierarchical(simmod):
    w = si.scaled(si.config("C3"), bytes=128 * 64 * 8)
    s = simmod.Simulator(w.n_nodes, w.n_endpoints, w.row_ptr, w.col_idx, w.bw, w.lat, w.cap, w.arb, 1)
    try:
        with pytest.raises(simmod.SimError) as e:
            s.load_collective(w.coll, w.bytes, w.group_size, None, si.DEP_CHUNK)
        assert e.value.status == simmod.SIM_ERR_INVALID_ARG
        with pytest.raises(simmod.SimError):
            s.load_collective(si.COLL_RING_ALLREDUCE, 128 * 64, 0, None, 2)
    finally:
        s.close()


# ------------------------------------------------------- further collectives
# Ring and direct all-gather / reduce-scatter, recursive halving-doubling and
# double binary tree all-reduce, per line and per message.

MORE = [si.COLL_RING_ALLGATHER, si.COLL_RING_REDUCESCATTER, si.COLL_DIRECT_ALLGATHER,
        si.COLL_DIRECT_REDUCESCATTER, si.COLL_RHD_ALLREDUCE, si.COLL_DBT_ALLREDUCE]


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("coll", MORE)
@pytest.mark.parametrize("dep", [0, 1])
def test_more_collectives_mesh(simmod, oracle_lib, engine, coll, dep):
    b = 1 if engine == "b1" else 2
    w = si.full_mesh(4, b=b, L=5, cap=b * 3, coll=coll, nbytes=128 * 4 * 6)
    w.dep = dep
    assert check_engine(simmod, oracle_lib, w, engine) == 1


@pytest.mark.parametrize("engine", ENGINES)
@pytest.mark.parametrize("coll", MORE)
@pytest.mark.parametrize("dep", [0, 1])
def test_more_collectives_torus(simmod, oracle_lib, engine, coll, dep):
    bws = (1,) if engine == "b1" else (1, 2, 4)
    w = si.torus2d(4, 4, n_scenarios=5, seed=90 + coll + 16 * dep, bws=bws, lat_lo=1, lat_hi=25,
                   depths=(1, 2, 3, 7, 32), nbytes=128 * 16 * 4, arb=(coll + dep) % 2, coll=coll)
    w.dep = dep
    check_engine(simmod, oracle_lib, w, engine)


@pytest.mark.parametrize("coll", MORE)
def test_more_collectives_fat_tree_ordered(simmod, oracle_lib, coll):
    w = si.fat_tree(4, nbytes=128 * 16 * 2, cap=5, lat_lo=2, lat_hi=9, arb=1, coll=coll)
    w.order = np.random.default_rng(coll).permutation(16).astype(np.int32)
    check_vs_oracle(simmod, oracle_lib, w)


def test_rhd_rank_order_torus_deadlocks_like_oracle(simmod, oracle_lib):
    """Full-size 4x4 torus sweep, RHD in rank order: two-hop partners close
    cyclic buffer dependencies and every scenario deadlocks.  The engine must
    stop where the oracle stops, with the same completed lines and counters."""
    w = si.take_scenarios(si.config("C5"), [0, 1, 2, 3, 1000, 4095])
    w.coll = si.COLL_RHD_ALLREDUCE
    say("C5-sized RHD in rank order: 6 scenarios")
    r, n_ok = check_vs_oracle(simmod, oracle_lib, w, expect_ok=False)
    assert n_ok == 0 and r.status == simmod.SIM_ERR_DEADLOCK


@pytest.mark.parametrize("dep", [0, 1])
@pytest.mark.parametrize("arb", [0, 1])
def test_wave_all_64_links(simmod, oracle_lib, dep, arb):
    """RHD on the 4x4 torus in Gray-code order uses all 64 links: one
    scenario per wavefront, every lane busy."""
    w = si.torus2d(4, 4, n_scenarios=7, seed=123 + arb + 2 * dep, bws=(1, 2, 4), lat_lo=1, lat_hi=30,
                   depths=(1, 2, 5, 16), nbytes=128 * 16 * 8, arb=arb, coll=si.COLL_RHD_ALLREDUCE)
    w.order = si.gray_torus_order(4, 4)
    w.dep = dep
    check_engine(simmod, oracle_lib, w, "wave")


# ------------------------------------------------ wave engine, ring graphs

@pytest.mark.parametrize("arb", [0, 1])
@pytest.mark.parametrize("coll", [si.COLL_RING_ALLGATHER, si.COLL_DIRECT_ALLREDUCE, si.COLL_ALLTOALL])
def test_wave_mesh_collectives_arb(simmod, oracle_lib, arb, coll):
    """Full mesh, both policies, b = 3: one-hop flows on links of their own
    (streams with many predecessors for the direct all-gather)."""
    w = si.full_mesh(6, b=3, L=4, cap=5, coll=coll, nbytes=128 * 6 * 5, arb=arb)
    assert check_engine(simmod, oracle_lib, w, "wave") == 1


@pytest.mark.parametrize("seed", range(16))
def test_wave_directed_ring_dags(simmod, oracle_lib, seed):
    """A directed ring whose flows go one or two hops: every link is fed by
    its predecessor link and by its own stream and sends lines on or out.
    Tiny buffers (the ring's buffers form a cycle, so some scenarios
    deadlock), mixed bandwidths, both policies, random predecessor DAGs."""
    rng = np.random.default_rng(9100 + seed)
    n = int(rng.integers(3, 7))
    rp = np.arange(n + 1, dtype=np.int32)
    ci = np.array([(v + 1) % n for v in range(n)], np.int32)
    S = 3
    bw = rng.choice([1, 2, 4, 8], size=S * n).astype(np.int32)
    lat = rng.integers(1, 6, size=S * n).astype(np.int32)
    cap = rng.integers(1, 9, size=S * n).astype(np.int32)
    T = int(rng.integers(20, 200))
    src = rng.integers(0, n, size=T).astype(np.int32)
    dst = ((src + rng.integers(1, 3, size=T)) % n).astype(np.int32)
    pptr = [0]
    pidx = []
    for x in range(T):
        k = int(rng.integers(0, 3)) if x else 0
        pidx += sorted(set(int(v) for v in rng.integers(0, x, size=k))) if x else []
        pptr.append(len(pidx))
    w = si.Workload("dir_ring", n, n, rp, ci, S, bw, lat, cap, seed % 2, -1, 0)
    check_engine(simmod, oracle_lib, w, "wave", txns=(src, dst, np.array(pptr, np.int64), np.array(pidx, np.int64)))


@pytest.mark.parametrize("name,general", [("C1", False), ("C2", False), ("C3", False), ("C1_chunk", False),
                                          ("C2_chunk", False), ("C4", False), ("C4_credit", False), ("C1", True),
                                          ("C2", True), ("C2_chunk", True)])
def test_full_size_digest_grid(simmod, torch_cuda, name, general):
    """The device-wide engine (one topology over many workgroups) on the
    single-topology benchmark workloads: the same bytes as the oracle's
    golden digests.  Graphs with every bandwidth 1 run its one-line form
    unless the general form is asked for; C4 with credit delays its
    windowed form."""
    g = _golden(name)
    w = si.config(name)
    say(f"full-size {name}: grid engine{' (general form)' if general else ''}")
    env = {"SIMGPU_ENGINE": "grid", "SIMGPU_GRID_GENERAL": "1" if general else None}
    old = {k: os.environ.get(k) for k in env}
    for k, v in env.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v
    try:
        r = run_gpu(simmod, w)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    assert r.status == 0, simmod.STATUS_NAMES[r.status]
    comp = r.completion[0].cpu().numpy().view(np.uint32)
    idx = np.array(g["sample_idx"])
    assert np.array_equal(comp[idx].astype(np.int64), np.array(g["sample_completion"]))
    assert int(r.makespan[0]) == g["makespan"][0]
    assert _digest(comp.astype("<u4")) == g["completion_sha256"][0]
    assert _digest(r.tx_lines[0].cpu().numpy().astype("<u8")) == g["tx_lines_sha256"][0]
    assert _digest(r.busy_cycles[0].cpu().numpy().astype("<u8")) == g["busy_cycles_sha256"][0]


@pytest.mark.parametrize("stride", [1, 8])
@pytest.mark.parametrize("name", ["C2", "C3"])
def test_grid_placement_same_bytes(simmod, torch_cuda, name, stride, monkeypatch):
    """The grid engine with its workgroups launched as consecutive blocks
    (spread over the dies) or every eighth block: the golden digests either
    way (C2: the one-line form, C3: the general form)."""
    monkeypatch.setenv("SIMGPU_ENGINE", "grid")
    monkeypatch.setenv("SIMGPU_GRID_STRIDE", str(stride))
    g = _golden(name)
    w = si.config(name)
    r = run_gpu(simmod, w)
    assert r.status == 0, simmod.STATUS_NAMES[r.status]
    comp = r.completion[0].cpu().numpy().view(np.uint32)
    assert _digest(comp.astype("<u4")) == g["completion_sha256"][0]
    assert _digest(r.tx_lines[0].cpu().numpy().astype("<u8")) == g["tx_lines_sha256"][0]
    assert _digest(r.busy_cycles[0].cpu().numpy().astype("<u8")) == g["busy_cycles_sha256"][0]
