"""Host logic of the fused pass's routes, on the CPU: plan_driver.cpp plans
random, skewed, run-structured and adversarial commit sequences into passes
with the library's planner (paper_1805_08469_amd/csrc/gem_plan.hpp) at ring
depths 2 to 6, and replays each pass the way the pass kernel moves a
thread's (snapshot, moment) chunks -- ring, register slots, store before
prefetch -- checking that every commit sees its worker's latest chunk, that
memory ends with every worker's last version, and that passes are cut only
where no held chunk can be evicted.  layout_driver.cpp checks the snapshot
and moment table's index (paper_1805_08469_amd/csrc/gem_layout.hpp): one
index per element, all inside the table, contiguous pieces per tile.  Both
are built with AddressSanitizer and UndefinedBehaviorSanitizer."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _build_and_run(tmp_path, source, *args):
    exe = tmp_path / os.path.splitext(source)[0]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-o", str(exe), os.path.join(HERE, source)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), *map(str, args)], capture_output=True, text=True, timeout=300,
                       env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok")
    assert "runtime error" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
@pytest.mark.parametrize("seed", [1, 2018])
def test_planned_routes_replay_the_sequential_commits(tmp_path, seed):
    _build_and_run(tmp_path, "plan_driver.cpp", seed)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_table_layout_gives_every_element_its_own_index(tmp_path):
    _build_and_run(tmp_path, "layout_driver.cpp")
