"""gem_gather_static, the allocation-free variant of gem_gather, through the
C ABI: bit for bit the outputs of gem_gather on the same state, on two calls
in a row (the second with fewer indices, so stale scratch contents from the
first would show), and a request beyond the fixed scratch refused with
GEM_ESCRATCH."""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_08469_amd import gem
    return gem


def _gather(L, fn, h, idx, n):
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    th = np.full(idx.size, np.nan, np.float32)
    S = np.full((n, idx.size), np.nan, np.float32)
    M = np.full((n, idx.size), np.nan, np.float32)
    rc = getattr(L, fn)(h, idx.ctypes.data_as(C.POINTER(C.c_int64)), idx.size,
                        th.ctypes.data, S.ctypes.data, M.ctypes.data)
    return rc, th, S, M


@pytest.mark.parametrize("P,n", [(5000, 4), (70_001, 100)])
def test_static_gather_equals_gather(G, P, n):
    from paper_1805_08469_amd.workloads import make_problem
    L = G.lib()
    h_, ts = make_problem(P, 1e-3, 1.0, 3)
    worker, tau = G.gem_schedule_make(n, 300, G.GEM_LAW_EXP, seed=5)
    per_index = 8 + 4 * (1 + 2 * n)
    cap = G.GEM_SCRATCH_BYTES // per_index
    rng = np.random.default_rng(P)
    with G.Gem(P, n) as g:
        g.set_quadratic(h_, ts, 0.01, 0.1, 7)
        g.sim_run(worker, tau, 16)
        first = rng.integers(0, P, size=min(cap, 3 * P)).astype(np.int64)   # a full scratch
        first[:3] = [0, P - 1, P // 2]
        second = rng.integers(0, P, size=max(1, first.size // 7)).astype(np.int64)
        for idx in (first, second):
            print(f"[static gather] P={P} n={n} count={idx.size} cap={cap}", flush=True)
            rc, th, S, M = _gather(L, "gem_gather_static", g.h, idx, n)
            assert rc == G.GEM_OK
            rc0, th0, S0, M0 = _gather(L, "gem_gather", g.h, idx, n)
            assert rc0 == G.GEM_OK
            for a, b in ((th, th0), (S, S0), (M, M0)):
                assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
        # outputs may be left out, as for gem_gather
        idx = second[:5]
        th = np.zeros(idx.size, np.float32)
        rc = L.gem_gather_static(g.h, idx.ctypes.data_as(C.POINTER(C.c_int64)), idx.size,
                                 th.ctypes.data, None, None)
        assert rc == G.GEM_OK and np.array_equal(th, G.gem_gather(g.h, idx, n)[0])
        # beyond the scratch, or out of range: refused, nothing written
        too_many = np.zeros(cap + 1, np.int64)
        rc, th, S, M = _gather(L, "gem_gather_static", g.h, too_many, n)
        assert rc == G.GEM_ESCRATCH and np.all(np.isnan(th))
        rc, th, S, M = _gather(L, "gem_gather_static", g.h, np.array([0, P], np.int64), n)
        assert rc == G.GEM_EINVAL and np.all(np.isnan(th))
        assert L.gem_gather_static(g.h, None, 0, None, None, None) == G.GEM_OK
