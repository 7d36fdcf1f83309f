"""The paper's GPU-architecture exploration (Sec. 5.3), reproduced in the
model at two GPUs (the paper uses 16 and 32): qualitative checks of the two
findings it draws, on the oracle.

* Loop unrolling (Fig. LoopUnrollingResult, all-to-all): more wavefront
  requests in flight per CU shortens a bandwidth-bound collective, the gain
  saturates, and a small latency-bound collective barely moves.
* Outstanding-request limit per CU (Fig. WFReqExploration, all-gather, a
  proxy for the register file): the same shape; the small collective is
  insensitive once a few requests may be outstanding.

These are statements about trends, not numbers: the paper prints none (its
values are only in the figures).  The exact makespans below are what the
model gives and are checked against the GPU path in test_gpu_memcpy.py.
"""
from __future__ import annotations

import pytest

from sim_inputs import noc


@pytest.fixture(scope="module")
def two_gpus():
    return noc.gpu_noc(2)


def makespan(oracle_lib, w0, mc):
    r = oracle_lib.simulate_workload(noc.memcpy_workload(w0, mc), 0)
    assert r.status_name == "OK"
    return r.makespan


def test_unrolling_helps_bandwidth_bound_all_to_all(oracle_lib, two_gpus):
    w0, lay = two_gpus
    big = [makespan(oracle_lib, w0, noc.alltoall_ops(lay, 4096, n_wg=32, unroll=u, window=64))
           for u in (1, 2, 4, 8, 16)]
    # each doubling of the unroll factor helps ...
    assert all(b < a for a, b in zip(big, big[1:])), big
    # ... a lot while requests are scarce, little once the CU's window binds
    assert big[0] / big[2] > 3.0, big
    assert big[3] / big[4] < 1.05, big


def test_unrolling_irrelevant_for_latency_bound_all_to_all(oracle_lib, two_gpus):
    w0, lay = two_gpus
    small = [makespan(oracle_lib, w0, noc.alltoall_ops(lay, 64, n_wg=32, unroll=u, window=64))
             for u in (1, 2, 4, 8, 16)]
    # two lines per workgroup: beyond unroll 2 nothing changes
    assert len(set(small[1:])) == 1, small
    assert small[0] / small[1] < 1.25, small


def test_outstanding_limit_saturates_all_gather(oracle_lib, two_gpus):
    w0, lay = two_gpus
    ws = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024)
    big = [makespan(oracle_lib, w0, noc.allgather_ops(lay, 16384, n_wg=32, unroll=16, window=w)) for w in ws]
    # up to the unrolled batch's worth the limit is the bound: halving the time
    # per doubling at first ...
    assert all(b < a for a, b in zip(big[:8], big[1:8])), big
    assert big[0] / big[3] > 6.0, big
    # ... and once 256 requests may be outstanding, more buys nothing
    assert max(big[8:]) / min(big[8:]) < 1.05, big
    assert big[-1] == big[-2], big


def test_outstanding_limit_irrelevant_for_latency_bound_all_gather(oracle_lib, two_gpus):
    w0, lay = two_gpus
    small = [makespan(oracle_lib, w0, noc.allgather_ops(lay, 128, n_wg=32, unroll=16, window=w))
             for w in (4, 8, 32, 128)]
    assert len(set(small)) == 1, small
