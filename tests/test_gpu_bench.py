"""bench.py on the GPU: its JSON line for the tiny workload under each option
(histogram recording, a forced cache policy, the segment scope, the shared
moment), one timed step each."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CASES = [
    (["--pi-hist"], "Fast, recording"),
    (["--pi-hist", "--proxy", "global"], "FastGlobal, diagnostic, depth 2"),
    (["--cache", "stream"], "Fast, depth 1, streaming"),
    (["--pi-scope", "segment"], "seg_step_kernel + seg_blocks_kernel"),
    (["--proxy", "global", "--cache", "keep"], "FastGlobal, depth 1>"),
]


@pytest.mark.parametrize("extra,label", CASES, ids=[" ".join(c[0]) for c in CASES])
def test_bench_line(extra, label):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "tiny",
           "--steps", "1", "--warmup", "0", "--no-cpu-baseline", *extra]
    print("[bench]", " ".join(extra), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=100)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    assert d["value"] > 0 and d["n_gpus"] == 1 and d["steps"] == 1
    roof = d["roofline"]
    assert label in roof["kernel"]
    assert roof["traffic"] is None
    if roof["bound"] == "hbm":
        assert 0 < roof["frac"] < 1
    else:   # against the VALU ceiling; the instruction count needs counters
        assert roof["bound"] == "alu" and 0 < roof["frac_of_compute_floor"] <= 1.2
