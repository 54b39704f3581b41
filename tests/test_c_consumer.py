"""The C ABI from plain C: include/gem.h compiles as strict C11 and a C program
links against libgem.so (CPU); the program's run on the GPU -- a simulated
schedule in fused passes, two single commits of a device update, a
checkpoint round trip into a second master, a rejected call -- ends with the
oracle's theta, bit for bit."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PKG = os.path.join(ROOT, "paper_1805_08469_amd")
ROCM_LIB = "/opt/rocm/lib"


def _build(out):
    if shutil.which("gcc") is None or not os.path.exists(os.path.join(PKG, "libgem.so")):
        pytest.skip("gcc or the built library is missing")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic", "-O1",
           "-o", str(out), os.path.join(HERE, "c_consumer.c"),
           "-L" + PKG, "-lgem", "-Wl,-rpath," + PKG,
           "-L" + ROCM_LIB, "-lamdhip64", "-Wl,-rpath," + ROCM_LIB]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    return out


def test_header_is_strict_c_and_links(tmp_path):
    _build(tmp_path / "c_consumer")


@pytest.mark.gpu
def test_c_program_matches_oracle(tmp_path):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = _build(tmp_path / "c_consumer")
    P, n, T, K = 3001, 4, 150, 16
    r = subprocess.run([str(exe), str(P), str(n), str(T), str(K), str(tmp_path / "ck.bin")],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    lines = r.stdout.split()
    assert int(lines[0]) == T + 2
    theta = np.array([int(x, 16) for x in lines[1:]], dtype=np.uint32).view(np.float32)

    i = np.arange(P)
    h = (np.float32(0.001) + (i % 97).astype(np.float32) / np.float32(97.0)).astype(np.float32)
    ts = ((i % 13).astype(np.float32) / np.float32(6.0) - np.float32(1.0)).astype(np.float32)
    upd = (((i * 7) % 11 - 5).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    worker, tau = O.schedule(n, T, O.LAW_EXP, 0, 0, seed=7)
    hp = O.Hyper(lr=0.01, sigma=0.1, seed=20180522)
    st = O.State.initial(n, P)
    O.run(hp, P, st, i, h, ts, worker, tau)
    O.commit_given(hp, st, np.array([0], np.int32), upd[None, :])
    O.commit_given(hp, st, np.array([n - 1], np.int32), upd[None, :])
    assert np.array_equal(theta.view(np.uint32), st.theta.view(np.uint32))
