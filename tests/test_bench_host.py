"""Host-side parts of bench.py: the CPU-oracle sample, the counter-staleness
hash and the one-GPU guard (no GPU needed)."""
from __future__ import annotations

import os
import subprocess
import sys

import bench
import sim_inputs as si

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_baseline_whole_scenario(oracle_lib):
    # C1 finishes inside the first cycle guard: the sample is the whole run
    r = bench.cpu_baseline(si.config("C1"), 1.0)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["value"] > 0
    assert "whole scenario" in r["sample"] and "(3072 line-hops" in r["sample"]


def test_cpu_baseline_prefix_counts_admissions(oracle_lib):
    # a run stopped by the cycle guard counts the link admissions done so far
    w = si.config("C2")
    part = oracle_lib.simulate_workload(w, 0, max_cycles=1000)
    assert part.status == 8
    done = int(part.tx_lines.sum())
    assert 0 < done < part.line_hops
    # C2 is one ring step of 16384 lines per link over 8 links: by cycle 1000
    # every link has admitted one line per cycle from cycle 0
    assert done == 8 * 1001


def test_cpu_baseline_batched(oracle_lib):
    w = si.take_scenarios(si.config("C5"), [0, 1])
    r = bench.cpu_baseline(w, 0.01)
    assert r["sample"].startswith("1 of 2 scenario(s)")


def test_source_hash_follows_includes(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2606_10440_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "engine_a.hip").write_text('#include "common.h"\nA\n')
    (csrc / "engine_b.hip").write_text('#include "other.h"\nB\n')
    (csrc / "common.h").write_text('#include "base.h"\n')
    (csrc / "other.h").write_text("O\n")
    (csrc / "base.h").write_text("X\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    a0, b0 = bench.engine_source_hash("engine_a<1>"), bench.engine_source_hash("void engine_b(x)")
    (csrc / "base.h").write_text("Y\n")  # reached from engine_a only
    assert bench.engine_source_hash("engine_a<1>") != a0
    assert bench.engine_source_hash("void engine_b(x)") == b0


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2 and "one GPU" in p.stderr
