"""Host-side checks of bench.py: the one-GPU contract, the plan's byte
accounting against the paper's per-pass traffic, and the counter summaries it
reads its traffic figure from."""
import json
import os
import re
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("proxy", ["local", "global"])
def test_counter_summaries_are_well_formed(proxy):
    """The committed summaries carry the FETCH_SIZE / WRITE_SIZE calibration
    and a traffic figure within a few percent of the algorithmic bytes."""
    path = bench.COUNTERS_FILES[("headline", proxy)]
    m = re.search(r"```json\s*(\{.*?\})\s*```", open(path).read(), flags=re.S)
    d = json.loads(m.group(1))
    assert d["workload"] == "headline" and d["proxy"] == proxy
    assert d["fetch_scale"] == pytest.approx(2.0, rel=1e-3)
    assert d["write_scale"] == pytest.approx(1.0, rel=1e-3)
    assert 1.0 <= d["hbm_bytes_per_pass"] / d["alg_bytes_per_pass"] < 1.05
    # per-worker moments: P'(16 + 16 D) bytes a pass; shared moment: P'(24 + 8 D)
    P = 25_000_000
    per_elem = d["alg_bytes_per_pass"] / P
    D = (per_elem - 16) / 16 if proxy == "local" else (per_elem - 24) / 8
    assert 20 < D <= 32


def test_traffic_is_withheld_for_other_sources(monkeypatch):
    """The traffic figure is only reported while the kernel sources hash to the
    value recorded with the counters."""
    monkeypatch.setattr(bench, "kernel_hash", lambda: "0" * 16)
    assert bench.measured_traffic("headline", "local") is None
    assert bench.measured_traffic("headline", "global") is None
    assert bench.measured_traffic("resnet18", "local") is None


def test_headline_distinct_workers_per_pass_match_schedule():
    """The algorithmic bytes bench.py reports come from the library's pass plan;
    recompute D per pass of 32 from the schedule (host only) and compare with
    the per-pass figure recorded next to the counters, to a few percent (the
    plan occasionally ends a pass early)."""
    import oracle as O
    from paper_1805_08469_amd.workloads import WORKLOADS
    wl = WORKLOADS["headline"]
    worker, _ = O.schedule(wl.n, wl.T, wl.law, wl.law_p0, wl.law_p1, seed=wl.seed)
    d = [np.unique(worker[k:k + wl.K]).size for k in range(0, wl.T, wl.K)]
    mean_bytes = 25_000_000 * (16 + 16 * np.mean(d))
    path = bench.COUNTERS_FILES[("headline", "local")]
    m = re.search(r"```json\s*(\{.*?\})\s*```", open(path).read(), flags=re.S)
    rec = json.loads(m.group(1))["alg_bytes_per_pass"]
    assert rec == pytest.approx(mean_bytes, rel=0.03)
