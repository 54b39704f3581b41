"""The C ABI on the CPU: the library loads, exports every symbol include/gem.h
declares, and its host-side logic (the queuing schedule, argument checks
that precede any device work) behaves as specified.  No kernel is launched."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

import oracle as O
from paper_1805_08469_amd import gem as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gem.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gem_[a-z0-9_]+)\s*\(", text)))


def test_header_declarations_match_binding():
    assert _declared() == sorted(G.EXPORTED)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", G.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    missing = [s for s in _declared() if s not in exported]
    assert not missing, missing
    lib = C.CDLL(G.LIB_PATH)
    for s in _declared():
        assert hasattr(lib, s)


def test_defaults_are_alg1():
    hp = G.gem_hyperparams_default()
    assert hp.momentum == pytest.approx(0.9) and hp.eps == np.float32(1e-16) and hp.kappa == 1.0
    assert (hp.pi_mode, hp.kappa_mode, hp.pull_mode, hp.rule, hp.proxy_mode, hp.pi_scope) == (
        G.GEM_PI_CLAMP0, G.GEM_KAPPA_LINEAR, G.GEM_PULL_POST_COMMIT, G.GEM_RULE_GEM,
        G.GEM_PROXY_LOCAL, G.GEM_PI_ELEMENT)


def test_strerror_covers_codes():
    for code in range(0, -11, -1):
        assert G.gem_strerror(code) != "unknown error"
    assert G.gem_strerror(-99) == "unknown error"


@pytest.mark.parametrize("law,p0,p1", [(G.GEM_LAW_EXP, 0, 0), (G.GEM_LAW_EXP_UNIFORM_MEAN, 0.8, 1.2),
                                       (G.GEM_LAW_EXP_LOGNORMAL_MEAN, 0.0, 0.5),
                                       (G.GEM_LAW_PARETO, 1.5, 1 / 3)])
@pytest.mark.parametrize("pull", [G.GEM_PULL_POST_COMMIT, G.GEM_PULL_PRE_COMMIT])
def test_schedule_bit_exact_vs_oracle(law, p0, p1, pull):
    for n, T, seed in [(1, 50, 0), (4, 3000, 7), (100, 5000, 20180522)]:
        w, t = G.gem_schedule_make(n, T, law, p0, p1, seed=seed, pull_mode=pull)
        w2, t2 = O.schedule(n, T, law, p0, p1, seed=seed, pull_mode=pull)
        assert np.array_equal(w, w2) and np.array_equal(t, t2)


def test_schedule_rejects_bad_arguments():
    L = G.lib()
    w = np.zeros(4, np.int32)
    law = G.gem_schedule_law(law=G.GEM_LAW_EXP)
    p = w.ctypes.data_as(C.POINTER(C.c_int32))
    assert L.gem_schedule_make(0, 4, C.byref(law), 0, 0, p, p) == G.GEM_EINVAL
    assert L.gem_schedule_make(2, 4, None, 0, 0, p, p) == G.GEM_EINVAL
    assert L.gem_schedule_make(2, 4, C.byref(law), 0, 7, p, p) == G.GEM_EINVAL
    bad = G.gem_schedule_law(law=9)
    assert L.gem_schedule_make(2, 4, C.byref(bad), 0, 0, p, p) == G.GEM_EINVAL
    par = G.gem_schedule_law(law=G.GEM_LAW_PARETO, p0=0.0, p1=1.0)
    assert L.gem_schedule_make(2, 4, C.byref(par), 0, 0, p, p) == G.GEM_EINVAL
    assert L.gem_schedule_make(2, 0, C.byref(law), 0, 0, None, None) == G.GEM_OK


def test_create_rejects_bad_arguments_before_device_work():
    L = G.lib()
    out = C.c_void_p()
    assert L.gem_create(0, 4, None, None, C.byref(out)) == G.GEM_EINVAL
    assert L.gem_create(16, 0, None, None, C.byref(out)) == G.GEM_EINVAL
    assert L.gem_create(16, 4, None, None, None) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.pi_mode = 5
    assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.proxy_mode = 2
    assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.pi_scope = 2
    assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.pi_scope = G.GEM_PI_SEGMENT
    hp.rule = G.GEM_RULE_ADAPTIVE        # per-segment pi is a GEM-rule scope
    assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.kappa_mode = G.GEM_KAPPA_SQRT
    hp.kappa = -1.0
    assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    # kappa scales a positive proxy energy (appendix B), in either form
    for mode in (G.GEM_KAPPA_LINEAR, G.GEM_KAPPA_SQRT):
        for kappa in (0.0, -0.0, -2.0, float("nan")):
            hp = G.gem_hyperparams_default()
            hp.kappa_mode = mode
            hp.kappa = kappa
            assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    # eps keeps |dtheta| + eps away from zero (Alg. 1): with eps = 0 an update
    # of exactly zero would give pi = inf and theta = inf * 0 = NaN
    for eps in (0.0, -0.0, -1e-16, float("inf"), float("nan")):
        hp = G.gem_hyperparams_default()
        hp.eps = eps
        assert L.gem_create(16, 4, C.byref(hp), None, C.byref(out)) == G.GEM_EINVAL
    hp = G.gem_hyperparams_default()
    hp.eps = 1e-45                       # the smallest positive binary32 is accepted
    assert hp.eps > 0
    # sizes: P above the largest grid, and a table whose byte count wraps 64 bits
    assert L.gem_create(G.GEM_P_MAX + 1, 1, None, None, C.byref(out)) == G.GEM_EINVAL
    assert L.gem_create(G.GEM_P_MAX, 2**31 - 1, None, None, C.byref(out)) == G.GEM_ENOMEM
    assert out.value is None


def test_p_max_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define GEM_P_MAX \(INT64_C\(1\) << (\d+)\)", text)
    assert m and G.GEM_P_MAX == 1 << int(m.group(1))


def test_null_handle_calls_fail_cleanly():
    L = G.lib()
    assert L.gem_destroy(None) == G.GEM_EINVAL
    assert L.gem_sync(None) == G.GEM_EINVAL
    assert L.gem_commit(None, None, 0) == G.GEM_EINVAL
    assert L.gem_sim_run(None, None, None, 0, 1) == G.GEM_EINVAL
    assert L.gem_copy_f32(None, None, 4, None) == G.GEM_EINVAL
    P, n = C.c_int64(), C.c_int32()
    assert L.gem_dims(None, C.byref(P), C.byref(n)) == G.GEM_EINVAL


def test_one_hip_runtime_per_process():
    """The binding loads torch's HIP runtime before libgem, so libgem shares
    it instead of mapping a second runtime beside torch's."""
    code = ("import re, sys; sys.path.insert(0, %r); from paper_1805_08469_amd import gem; "
            "import torch; m = open('/proc/self/maps').read(); "
            "print(len(set(re.findall(r'/\\S*libamdhip64\\S*', m))))" % ROOT)
    out = subprocess.run([os.sys.executable, "-c", code], check=True, capture_output=True,
                         text=True).stdout.strip()
    assert out == "1"
