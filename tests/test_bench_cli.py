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


def _summary(key):
    path = os.path.join(ROOT, "profiles", bench.COUNTERS_FILES[key])
    m = re.search(r"```json\s*(\{.*?\})\s*```", open(path).read(), flags=re.S)
    return json.loads(m.group(1))


@pytest.mark.parametrize("key", sorted(bench.COUNTERS_FILES), ids=lambda k: "-".join(k))
def test_counter_summaries_are_well_formed(key):
    """The committed summaries carry the FETCH_SIZE / WRITE_SIZE calibration
    and a traffic figure near the algorithmic bytes (a state that fits the
    Infinity Cache moves less HBM traffic than its algorithmic bytes)."""
    workload, proxy, scope = key
    d = _summary(key)
    assert (d["workload"], d["proxy"], d.get("pi_scope", "element")) == key
    assert d["fetch_scale"] == pytest.approx(2.0, rel=1e-3)
    assert d["write_scale"] == pytest.approx(1.0, rel=1e-3)
    ratio = d["hbm_bytes_per_pass"] / d["alg_bytes_per_pass"]
    assert (0.0 < ratio < 1.05) if workload == "small" else (0.98 <= ratio < 1.05)
    if key[:2] == ("headline", "local") and scope == "element":
        # per-worker moments: P'(16 + 16 D) bytes a pass
        D = (d["alg_bytes_per_pass"] / 25_000_000 - 16) / 16
        assert 20 < D <= 32
    if key == ("headline", "global", "element"):
        D = (d["alg_bytes_per_pass"] / 25_000_000 - 24) / 8   # shared moment: P'(24 + 8 D)
        assert 20 < D <= 32
    if scope == "segment":   # 32 bytes per element-commit with post-commit pulls
        assert d["alg_bytes_per_pass"] == pytest.approx(32 * 25_000_000, rel=1e-5)
    assert d["valu_instrs_per_pass"] > 0


def test_traffic_is_withheld_for_other_sources(monkeypatch):
    """The counter figures are only reported while the kernel sources hash to
    the value recorded with the counters."""
    monkeypatch.setattr(bench, "kernel_hash", lambda: "0" * 16)
    for key in bench.COUNTERS_FILES:
        assert bench.measured_counters(*key) is None
    assert bench.measured_counters("tiny", "local", "element") is None


def test_host_description():
    d = bench.host_description()
    assert d["logical_cores"] >= 1 and (d["usable_cores"] is None or d["usable_cores"] >= 1)


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
    rec = _summary(("headline", "local", "element"))["alg_bytes_per_pass"]
    assert rec == pytest.approx(mean_bytes, rel=0.03)
