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


def test_largest_vector(G):
    """The largest P the library takes, less 3 (ragged: not a multiple of the
    16-byte chunk, the 1024-element block or the 8192-element tile), two
    workers, 33 commits in passes of 32 and 1.  Element indices near 2^31 and
    table offsets past 2^33 bytes must reach the right elements.  The oracle
    runs one index per block of the top 2^24 elements, both sides of every
    tile edge there, the last 16 elements, indices around 2^29 and 2^30 and
    random indices over the whole vector.  h and theta* repeat a random
    pattern every 2^20 elements, scaled and shifted per 2^20-element span, so
    no two spans hold the same values."""
    P = G.GEM_P_MAX - 3
    n, T, K = 2, 33, 32
    need = 4 * P * (2 * n + 3) * 1.05
    if _free_bytes() < need:
        pytest.skip(f"needs {need / 2**30:.1f} GiB of device memory")
    rng = np.random.default_rng(11)
    span = 1 << 20
    base_h = np.exp(rng.uniform(np.log(1e-4), 0.0, span)).astype(np.float32)
    base_t = rng.standard_normal(span).astype(np.float32)
    h = np.empty(P, dtype=np.float32)
    ts = np.empty(P, dtype=np.float32)
    for c in range(-(-P // span)):
        a, b = c * span, min(P, (c + 1) * span)
        h[a:b] = base_h[:b - a] * np.float32(1.0 + c * 2.0 ** -12)
        ts[a:b] = base_t[:b - a] + np.float32(c * 2.0 ** -10)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=3)
    top = P - (1 << 24)
    blocks = np.arange(top // BLOCK_ELEMS, -(-P // BLOCK_ELEMS), dtype=np.int64)
    per_block = blocks * BLOCK_ELEMS + (blocks * 389) % BLOCK_ELEMS
    edges = np.arange(top // TILE_ELEMS + 1, -(-P // TILE_ELEMS), dtype=np.int64) * TILE_ELEMS
    fixed = np.array([0, 1, 2, 3, (1 << 29) - 1, 1 << 29, (1 << 30) - 1, 1 << 30,
                      (1 << 31) - 1024], dtype=np.int64)
    idx = np.concatenate([fixed, per_block, edges - 1, edges, np.arange(P - 16, P),
                          rng.integers(0, P, size=20_000)])
    idx = np.unique(idx[(idx >= 0) & (idx < P)]).astype(np.int64)
    print(f"[largest] P={P} n={n} T={T} K={K} sample={idx.size}", flush=True)
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.02, 5)
        g.sim_run(worker, tau, K)
        theta, S, M = g.gather(idx)
        stats = g.stats()
    assert stats.passes == 2 and stats.commits == T
    hp = O.Hyper(lr=0.01, sigma=0.02, momentum=0.9, seed=5)
    st = O.State.initial(n, idx.size)
    O.run(hp, P, st, idx, h[idx], ts[idx], worker, tau)
    del h, ts
    assert_parity("largest theta", theta, st.theta)
    assert_parity("largest S", S, st.S)
    assert_parity("largest M", M, st.M)
