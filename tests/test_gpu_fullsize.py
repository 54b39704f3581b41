"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times (gem_sim_run over the whole schedule with the workload's K).

The GPU runs every element; the oracle runs a sample of element indices: one
index in every block of 1024 elements (the elements one 256-thread block of
the pass owns, whose tile base and row offsets are block-uniform), at a lane
position that rotates through all 1024 positions, both sides of every
8192-element table-tile edge, the first and last chunks, the ragged tail and
random indices.  Each element's trajectory depends only on its own inputs,
the schedule and the seed, so the oracle's subset run equals those entries of
a full run (pinned on the CPU by test_subset_run_equals_full_run)."""
import numpy as np
import pytest

import oracle as O
from gpu_util import assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_08469_amd import gem
    return gem


BLOCK_ELEMS = 1024    # elements of one pass-kernel block (256 threads x 4)
TILE_ELEMS = 8192     # elements of one table tile


def _sample(P, k=2048, seed=0):
    rng = np.random.default_rng(seed)
    fixed = np.array([0, 1, 2, 3, 4, 5, 6, 7, P // 2, P - 8, P - 7, P - 6, P - 5, P - 4, P - 3,
                      P - 2, P - 1])
    # one index per block; 389 is odd, so the offsets run through every lane
    # position (and every element of a 16-byte chunk) once per 1024 blocks
    blocks = np.arange(-(-P // BLOCK_ELEMS), dtype=np.int64)
    per_block = blocks * BLOCK_ELEMS + (blocks * 389) % BLOCK_ELEMS
    edges = np.arange(1, -(-P // TILE_ELEMS), dtype=np.int64) * TILE_ELEMS
    idx = np.concatenate([fixed, per_block, edges - 1, edges, rng.integers(0, P, size=k)])
    return np.unique(idx[(idx >= 0) & (idx < P)]).astype(np.int64)



def _free_bytes():
    import torch
    free, _ = torch.cuda.mem_get_info()
    return free


def _workload_parity(G, name, T=None, proxy=0):
    from paper_1805_08469_amd.workloads import WORKLOADS, problem
    wl = WORKLOADS[name]
    if T is not None:
        wl = wl.with_(T=T)
    need = 4 * wl.P * (2 * wl.n + 3) * 1.05
    if _free_bytes() < need:
        pytest.skip(f"{name} needs {need / 2**30:.1f} GiB of device memory")
    h, ts = problem(wl)
    worker, tau = G.gem_schedule_make(wl.n, wl.T, wl.law, wl.law_p0, wl.law_p1, seed=wl.seed)
    idx = _sample(wl.P, seed=wl.P)
    print(f"[{name}] P={wl.P} n={wl.n} T={wl.T} K={wl.K} bf16={wl.bf16} proxy={proxy} "
          f"sample={idx.size}", flush=True)
    ghp = G.gem_hyperparams_default()
    ghp.proxy_mode = proxy
    with G.Gem(wl.P, wl.n, ghp) as g:
        g.set_quadratic(h, ts, wl.lr, wl.sigma, wl.seed, bf16=wl.bf16)
        g.sim_run(worker, tau, wl.K)
        theta, S, M = g.gather(idx)
        pc = g.pull_clocks()
        stats = g.stats()
    hp = O.Hyper(lr=wl.lr, sigma=wl.sigma, momentum=wl.momentum, bf16=wl.bf16, seed=wl.seed,
                 proxy=proxy)
    st = O.State.initial(wl.n, idx.size)
    O.run(hp, wl.P, st, idx, h[idx], ts[idx], worker, tau)
    assert np.array_equal(pc, st.pc)
    assert_parity(f"{name} theta", theta, st.theta)
    assert_parity(f"{name} S", S, st.S)
    assert_parity(f"{name} M", M, st.M)
    return stats


def test_small(G):
    s = _workload_parity(G, "small")
    assert s.passes == 10_000


def test_resnet18(G):
    _workload_parity(G, "resnet18")


def test_headline(G):
    s = _workload_parity(G, "headline")
    assert -(-5000 // 32) <= s.passes <= 1.1 * -(-5000 // 32)


def test_headline_global_proxy(G):
    """The shared-moment mode at the headline size, as bench.py --proxy global
    runs it.  The shared moment is row 0 of M; the other rows stay zero."""
    _workload_parity(G, "headline", proxy=1)


def test_large(G):
    _workload_parity(G, "large")
