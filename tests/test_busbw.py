"""Bus bandwidth (the paper's reporting measure) from simulated times."""
from __future__ import annotations

import pytest

import sim_inputs as si
from paper_2606_10440_amd.sim import bus_bandwidth


def test_paper_table_arithmetic():
    # All-reduce of 1 MiB over 8 GPUs completing in 165.98 us: the table of
    # Sec. 5.5 reports 88.45 Gbps; 2(p-1)/p * S / T = 88.44 Gbps.
    assert bus_bandwidth(si.COLL_RING_ALLREDUCE, 1 << 20, 8, 165.98e-6) / 1e9 == pytest.approx(88.44, abs=0.01)


def test_ring_reaches_link_bandwidth(oracle_lib):
    # C2's ring all-reduce is bandwidth bound: its bus bandwidth is within
    # (latency / time) of one line (1024 bits) per cycle per link.
    w = si.config("C2")
    r = oracle_lib.simulate_workload(w)
    bb = bus_bandwidth(w.coll, w.bytes, w.n_endpoints, r.makespan)
    assert 0.999 * 1024 < bb < 1024


def test_factors():
    assert bus_bandwidth(si.COLL_RING_ALLGATHER, 800, 8, 1.0) == pytest.approx(8 * 800 * 7 / 8)
    assert bus_bandwidth(si.COLL_ALLTOALL, 100, 4, 1.0) == pytest.approx(8 * 400 * 3 / 4)
