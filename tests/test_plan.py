"""Host logic of the fused pass's routes, on the CPU: plan_driver.cpp plans
random, skewed, run-structured and adversarial commit sequences into passes
with the library's planner (paper_1805_08469_amd/csrc/gem_plan.hpp) at ring
depths 2 to 6, and replays each pass the way the pass kernel moves a
thread's (snapshot, moment) chunks -- ring, register slots, store before
prefetch -- checking that every commit sees its worker's latest chunk, that
memory ends with every worker's last version, and that passes are cut only
where no held chunk can be evicted.  Built with AddressSanitizer and
UndefinedBehaviorSanitizer."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
@pytest.mark.parametrize("seed", [1, 2018])
def test_planned_routes_replay_the_sequential_commits(tmp_path, seed):
    exe = tmp_path / "plan_driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-o", str(exe), os.path.join(HERE, "plan_driver.cpp")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), str(seed)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok")
    assert "runtime error" not in r.stderr, r.stderr
