"""GPU parity of whole simulated runs (gem_sim_run) against the oracle:
theta, every worker's snapshot S[w] and moment M[w], element by element, on
the same seeded schedules and noise.  Covers the tiny workload end to end,
fusion of K commits per pass (with workers repeating inside a pass at every
distance), ragged parameter counts, every commit-rule mode,
bfloat16 updates, diagnostics, checkpoint resume and worker restarts."""
import os
import tempfile

import numpy as np
import pytest

import oracle as O
from gpu_util import assert_parity, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_08469_amd import gem
    return gem


def _hp(G, pi_mode=0, kappa=1.0, kappa_mode=0, pull=0, rule=0, momentum=0.9, proxy=0):
    hp = G.gem_hyperparams_default()
    hp.momentum, hp.kappa = momentum, kappa
    hp.pi_mode, hp.kappa_mode, hp.pull_mode, hp.rule = pi_mode, kappa_mode, pull, rule
    hp.proxy_mode = proxy
    return hp


def _ohp(hp, lr, sigma, seed, bf16=False):
    return O.Hyper(lr=lr, sigma=sigma, momentum=hp.momentum, eps=1e-16, kappa=hp.kappa,
                   pi_mode=hp.pi_mode, kappa_mode=hp.kappa_mode, pull_mode=hp.pull_mode,
                   rule=hp.rule, bf16=bf16, proxy=hp.proxy_mode, seed=seed)


def _run_both(G, P, n, worker, tau, K, hp, lr=0.01, sigma=0.1, seed=7, bf16=False,
              h_lo=1e-3, pseed=1):
    from paper_1805_08469_amd.workloads import make_problem
    h, ts = make_problem(P, h_lo, 1.0, pseed)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, lr, sigma, seed, bf16=bf16)
        g.sim_run(worker, tau, K)
        out = (g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, g.stats())
    st = O.State.initial(n, P)
    O.run(_ohp(hp, lr, sigma, seed, bf16), P, st, np.arange(P), h, ts, worker, tau)
    return out, st


def _check(out, st, tag=""):
    theta, S, M, pc, clock, _ = out
    assert clock == st.t
    assert np.array_equal(pc, st.pc), f"{tag} pull clocks"
    assert_parity(f"{tag} theta", theta, st.theta)
    assert_parity(f"{tag} S", S, st.S)
    assert_parity(f"{tag} M", M, st.M)


def test_tiny_workload_full(G):
    from paper_1805_08469_amd.workloads import WORKLOADS
    wl = WORKLOADS["tiny"]
    worker, tau = G.gem_schedule_make(wl.n, wl.T, wl.law, wl.law_p0, wl.law_p1, seed=wl.seed)
    out, st = _run_both(G, wl.P, wl.n, worker, tau, wl.K, _hp(G), wl.lr, wl.sigma, wl.seed,
                        h_lo=wl.h_lo, pseed=wl.seed)
    _check(out, st, "tiny")
    assert out[5].passes == wl.T       # K = 1: one pass per commit


@pytest.mark.parametrize("K", [1, 2, 3, 8, 16, 32])
def test_fusion_is_invisible(G, K):
    """K commits per pass equal K single commits, bit for bit, including
    workers that commit several times inside one pass."""
    P, n, T = 3000, 3, 300
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=5)
    out, st = _run_both(G, P, n, worker, tau, K, _hp(G))
    _check(out, st, f"K={K}")
    assert out[5].passes == -(-T // K)      # three workers never fill four slots


def _taus(worker, n):
    pc = np.zeros(n, dtype=np.int64)
    tau = []
    for t, w in enumerate(worker):
        tau.append(t - pc[w])
        pc[w] = t + 1
    return np.array(tau, dtype=np.int32)


@pytest.mark.parametrize("pattern", ["same_worker_runs", "distance_two", "round_robin_12",
                                     "mixed"])
@pytest.mark.parametrize("K", [2, 3, 32])
def test_repeats_inside_a_pass(G, pattern, K):
    """A worker that commits again inside a pass must see the snapshot and
    moment its previous commit left: at distance 1 (taken from registers), at
    distance 2 (re-read right after the store) and farther (re-read from
    memory), with passes of every parity."""
    rng = np.random.default_rng(K)
    if pattern == "same_worker_runs":
        worker = np.repeat(np.array([0, 1, 2, 1, 0, 3, 3, 2], np.int32), 5)
        n = 4
    elif pattern == "distance_two":
        worker = np.tile(np.array([0, 1, 0, 1, 2, 3, 2, 3, 2], np.int32), 6)
        n = 4
    elif pattern == "round_robin_12":
        n = 12
        worker = np.tile(np.arange(n, dtype=np.int32), 20)
    else:
        n = 5
        worker = rng.integers(0, n, size=200).astype(np.int32)
    out, st = _run_both(G, 2048 + 5, n, worker, _taus(worker, n), K, _hp(G))
    _check(out, st, pattern)
    # a pass ends early when an immediate repeat finds every register slot busy
    assert out[5].passes >= -(-worker.size // K)
    if pattern == "round_robin_12":
        assert out[5].passes == -(-worker.size // K)


@pytest.mark.parametrize("P", [1, 3, 63, 64, 65, 1000, 4133, 70001])
def test_ragged_sizes(G, P):
    n, T = 5, 60
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=P)
    out, st = _run_both(G, P, n, worker, tau, 8, _hp(G))
    _check(out, st, f"P={P}")


MODES = {
    "literal": dict(pi_mode=1),
    "kappa2_linear": dict(kappa=2.0),
    "kappa3_sqrt": dict(kappa=3.0, kappa_mode=1),
    "kappa_half": dict(kappa=0.5),
    "pre_commit_pull": dict(pull=1),
    "downpour": dict(rule=1),
    "adaptive": dict(rule=2),
    "mu0": dict(momentum=0.0),
    "global_proxy": dict(proxy=1),
    "global_proxy_kappa2_pre_pull": dict(proxy=1, kappa=2.0, pull=1),
}


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("K", [1, 16])
def test_modes(G, mode, K):
    P, n, T = 4096 + 17, 6, 80
    hp = _hp(G, **MODES[mode])
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=3, pull_mode=hp.pull_mode)
    out, st = _run_both(G, P, n, worker, tau, K, hp)
    _check(out, st, mode)


@pytest.mark.parametrize("mode", sorted(MODES))
def test_modes_with_extreme_update_magnitudes(G, mode):
    """Every mode with caller updates of every magnitude (subnormal, huge,
    infinite, NaN) mixed into ordinary ones: the general division where an
    operand leaves the core range, overflow to infinity, NaN from inf - inf;
    the state equals the oracle's (NaN compares equal to NaN)."""
    import torch
    P, n, T, K = 4133, 3, 24, 8
    rng = np.random.default_rng(57)
    d = (rng.standard_normal((T, P)) * 0.01).astype(np.float32)
    ext = np.array([0.0, -0.0, 1e-45, -1e-40, 1e-30, -1e-20, 1e-10, -1e10, 1e20, -1e30, 3e38,
                    np.inf, -np.inf, np.nan], dtype=np.float32)
    pick = rng.random((T, P)) < 0.03
    d[pick] = rng.choice(ext, size=int(pick.sum()))
    hp = _hp(G, **MODES[mode])
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=57, pull_mode=hp.pull_mode)
    pad = np.zeros((T, -(-P // 8) * 8), dtype=np.float32)   # rows 16-byte aligned
    pad[:, :P] = d
    dev = torch.from_numpy(pad).cuda()
    with G.Gem(P, n, hp) as g:
        for b in range(0, T, K):
            g.commit_batch([dev[j].data_ptr() for j in range(b, b + K)], G.GEM_F32,
                           worker[b:b + K], tau[b:b + K])
        torch.cuda.synchronize()
        out = (g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, g.stats())
    st = O.State.initial(n, P)
    with np.errstate(all="ignore"):
        O.commit_given(_ohp(hp, 0.0, 0.0, 0), st, worker, d, tau=tau)
    _check(out, st, f"{mode} extremes")


POLICY_CASES = [
    ("default_depth4", {}, 32, False),    # Fast, ring depth 4
    ("default_depth2", {}, 8, False),     # Fast, ring depth 2 (short passes)
    ("global_proxy", dict(proxy=1), 32, False),
    ("kappa2_linear", dict(kappa=2.0), 32, False),
    ("default_bf16", {}, 16, True),
    # passes of one commit: the kernels compiled for a single commit
    ("default_k1", {}, 1, False),
    ("global_proxy_k1", dict(proxy=1), 1, False),
    ("kappa2_linear_k1", dict(kappa=2.0), 1, False),
    ("default_bf16_k1", {}, 1, True),
]


@pytest.mark.parametrize("case,mode,K,bf16", POLICY_CASES, ids=[c[0] for c in POLICY_CASES])
def test_cache_policies_give_the_same_bits(G, case, mode, K, bf16):
    """Streaming (non-temporal) and default-policy passes give the same state,
    bit for bit, equal to the oracle -- every pass variant and ring depth, with
    repeats and evictions inside passes (a small state, where AUTO keeps the
    default policy and STREAM is forced)."""
    P, n, T = 8192 * 2 + 77, 5, 160
    hp = _hp(G, **mode)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=31, pull_mode=hp.pull_mode)
    from paper_1805_08469_amd.workloads import make_problem
    h, ts = make_problem(P, 1e-3, 1.0, 31)
    states = {}
    for policy in (G.GEM_CACHE_KEEP, G.GEM_CACHE_STREAM, G.GEM_CACHE_AUTO):
        with G.Gem(P, n, hp) as g:
            g.set_cache_policy(policy)
            g.set_quadratic(h, ts, 0.01, 0.1, 9, bf16=bf16)
            g.sim_run(worker, tau, K)
            states[policy] = (g.theta(), g.S(), g.M())
    for policy in (G.GEM_CACHE_STREAM, G.GEM_CACHE_AUTO):
        for a, b in zip(states[G.GEM_CACHE_KEEP], states[policy]):
            assert np.array_equal(a, b), f"{case}: policy {policy} differs"
    st = O.State.initial(n, P)
    O.run(_ohp(hp, 0.01, 0.1, 9, bf16), P, st, np.arange(P), h, ts, worker, tau)
    assert_parity(f"{case} theta", states[G.GEM_CACHE_STREAM][0], st.theta)
    assert_parity(f"{case} S", states[G.GEM_CACHE_STREAM][1], st.S)
    assert_parity(f"{case} M", states[G.GEM_CACHE_STREAM][2], st.M)


@pytest.mark.parametrize("mode", [{}, dict(proxy=1)], ids=["default", "global_proxy"])
def test_single_commit_tail_pass(G, mode):
    """A run whose last pass holds one commit (T = 2K + 1) switches to the
    single-commit kernel for it; the state still equals the oracle's."""
    P, n, K = 8192 + 129, 6, 32
    T = 2 * K + 1
    hp = _hp(G, **mode)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=5, pull_mode=hp.pull_mode)
    from paper_1805_08469_amd.workloads import make_problem
    h, ts = make_problem(P, 1e-3, 1.0, 5)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 4)
        g.sim_run(worker, tau, K)
        out = (g.theta(), g.S(), g.M(), g.clock)
    assert out[3] == T
    st = O.State.initial(n, P)
    O.run(_ohp(hp, 0.01, 0.1, 4), P, st, np.arange(P), h, ts, worker, tau)
    assert_parity("theta", out[0], st.theta)
    assert_parity("S", out[1], st.S)
    assert_parity("M", out[2], st.M)


def test_cache_policy_rejects_unknown_values(G):
    with G.Gem(100, 2) as g:
        assert G.lib().gem_set_cache_policy(g.h, 3) == G.GEM_EINVAL
        assert G.lib().gem_set_cache_policy(g.h, -1) == G.GEM_EINVAL
        assert G.lib().gem_set_cache_policy(g.h, G.GEM_CACHE_STREAM) == G.GEM_OK


@pytest.mark.parametrize("K", [1, 16])
def test_bf16_updates(G, K):
    P, n, T = 5000, 10, 120
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_PARETO, 1.5, 1 / 3, seed=11)
    out, st = _run_both(G, P, n, worker, tau, K, _hp(G), sigma=0.02, bf16=True)
    _check(out, st, "bf16")


def test_literal_diverges_on_gpu_like_oracle(G):
    """The LITERAL pi blows up on the tiny workload (reading R8); the GPU follows the
    oracle into the blow-up as long as values stay finite."""
    from paper_1805_08469_amd.workloads import WORKLOADS
    wl = WORKLOADS["tiny"]
    T = 150
    worker, tau = G.gem_schedule_make(wl.n, T, wl.law, seed=wl.seed)
    out, st = _run_both(G, wl.P, wl.n, worker, tau, 1, _hp(G, pi_mode=1), wl.lr, wl.sigma,
                        wl.seed, h_lo=wl.h_lo, pseed=wl.seed)
    _check(out, st, "literal")
    assert np.nanmax(np.abs(st.theta)) > 1e6


@pytest.mark.parametrize("proxy", [0, 1], ids=["local", "global"])
def test_diagnostics_match_oracle(G, proxy):
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T, K = 10_000 + 3, 8, 200, 8
    h, ts = make_problem(P, 1e-3, 1.0, 2)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=2)
    hp = _hp(G, proxy=proxy)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 4)
        G.gem_diag_enable(g.h, True)
        g.sim_run(worker, tau, K)
        d = G.gem_diag(g.h)
    st = O.State.initial(n, P)
    dg, _ = O.run(_ohp(hp, 0.01, 0.1, 4), P, st, np.arange(P), h, ts, worker, tau, diag=True)
    assert d.n_commits == T
    assert d.n_elem_commits == P * T
    assert d.n_clamped == int(dg["n_clamped"].sum())
    assert d.sum_ek == pytest.approx(float(dg["sum_ek"].sum()), rel=1e-9)
    assert d.sum_proxy == pytest.approx(float(dg["sum_proxy"].sum()), rel=1e-9)
    assert d.loss == pytest.approx(O.loss(st.theta, h, ts), rel=1e-10)


def test_checkpoint_resume_is_bit_exact(G):
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T, K = 3000, 7, 200, 16
    h, ts = make_problem(P, 1e-3, 1.0, 5)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=8)
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 6)
        g.sim_run(worker, tau, K)
        straight = (g.theta(), g.S(), g.M())
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "ck.bin")
        with G.Gem(P, n) as g:
            g.set_quadratic(h, ts, 0.01, 0.1, 6)
            g.sim_run(worker[:77], tau[:77], K)
            assert G.gem_save(g.h, path) == G.GEM_OK
        with G.Gem(P, n) as g:
            assert G.gem_load(g.h, path) == G.GEM_OK
            assert g.clock == 77
            g.sim_run(worker[77:], tau[77:], K)
            resumed = (g.theta(), g.S(), g.M())
        with G.Gem(P + 1, n) as g:
            assert G.gem_load(g.h, path) == G.GEM_EIO
    for a, b in zip(straight, resumed):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("proxy,w", [(0, 2), (1, 0)])
def test_reset_worker_matches_oracle(G, proxy, w):
    """A worker that fails and restarts: m_w = 0, it pulls theta now (Alg. 1 Worker
    start-up).  With the shared moment (row 0 of M) only the pull happens."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 2000, 4
    h, ts = make_problem(P, 1e-3, 1.0, 9)
    worker, tau = G.gem_schedule_make(n, 100, G.GEM_LAW_EXP, seed=9)
    st = O.State.initial(n, P)
    ohp = O.Hyper(lr=0.01, sigma=0.1, momentum=0.9, seed=3, proxy=proxy)
    with G.Gem(P, n, _hp(G, proxy=proxy)) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 3)
        g.sim_run(worker[:50], tau[:50], 8)
        O.run(ohp, P, st, np.arange(P), h, ts, worker[:50], tau[:50])
        assert G.gem_reset_worker(g.h, w) == G.GEM_OK
        st.S[w] = st.theta
        if proxy == 0:
            st.M[w] = 0
        st.pc[w] = st.t
        w2 = worker[50:]
        pc = st.pc.copy()
        tau2 = []
        for j, w in enumerate(w2):
            tau2.append(st.t + j - pc[w])
            pc[w] = st.t + j + 1
        g.sim_run(w2, np.array(tau2, np.int32), 8)
        O.run(ohp, P, st, np.arange(P), h, ts, w2, tau2)
        _check((g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, None), st, "reset")


@pytest.mark.parametrize("mode", ["default", "downpour", "adaptive", "literal", "global_proxy"])
def test_pi_histograms_match_oracle(G, mode):
    """Per-commit histograms of the applied scale factor (Sec. 4's per-parameter
    pi), counted exactly; recorded alongside the energy diagnostics and cut
    at the recording capacity."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T, K, cap = 6000 + 7, 5, 150, 16, 120
    kw = {"default": {}, "downpour": dict(rule=1), "adaptive": dict(rule=2),
          "literal": dict(pi_mode=1), "global_proxy": dict(proxy=1)}[mode]
    hp = _hp(G, **kw)
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=7)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 2)
        G.gem_diag_enable(g.h, mode == "default")
        G.gem_pi_hist_start(g.h, cap)
        g.sim_run(worker, tau, K)
        got = G.gem_pi_hist_read(g.h, T)
        theta = g.theta()
    st = O.State.initial(n, P)
    _, _, hist = O.run(_ohp(hp, 0.01, 0.1, 2), P, st, np.arange(P), h, ts, worker, tau,
                       pi_hist=True)
    assert got.shape == (cap, G.GEM_PI_BINS)
    assert np.array_equal(got, hist[:cap])
    assert_parity("theta", theta, st.theta)


@pytest.mark.parametrize("K,bf16,cap", [(16, False, 120), (32, False, 150), (8, False, 77),
                                        (32, True, 100)])
def test_pi_histograms_recording_pass_match_oracle(G, K, bf16, cap):
    """The default rule without energy diagnostics records through its own
    pass (one LDS histogram per commit for the whole pass, flushed once):
    counts exact against the oracle, in deep (K >= 16) and shallow passes, with
    bf16 updates, a ragged tail and the capacity reached inside a pass."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 6000 + 7, 5, 150
    hp = _hp(G)
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=7)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 2, bf16=bf16)
        G.gem_pi_hist_start(g.h, cap)
        g.sim_run(worker, tau, K)
        got = G.gem_pi_hist_read(g.h, T)
        theta, S, M = g.theta(), g.S(), g.M()
    st = O.State.initial(n, P)
    _, _, hist = O.run(_ohp(hp, 0.01, 0.1, 2, bf16=bf16), P, st, np.arange(P), h, ts, worker, tau, pi_hist=True)
    assert got.shape == (min(cap, T), G.GEM_PI_BINS)
    assert np.array_equal(got, hist[:cap])
    assert got.sum(axis=1).tolist() == [P] * min(cap, T)
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)


# Partitions for per-segment histograms: one segment; tensors inside and across
# the 1024-element blocks; a block holding more segments than it keeps
# block-local histograms for (the rest count straight into memory).
HIST_PARTITIONS = {
    "one": lambda P: [0, P],
    "tensors": lambda P: [0, 17, 1024, 1100, 3000, 3001, P],
    "many_small": lambda P: sorted(set(list(range(0, 1024, 37)) + [2048, 2049, 4095, P])),
}


@pytest.mark.parametrize("mode", ["default", "downpour", "global_proxy"])
@pytest.mark.parametrize("part", sorted(HIST_PARTITIONS))
def test_pi_histograms_per_segment_match_oracle(G, mode, part):
    """One histogram per segment (per tensor) and commit, counted exactly, in
    the same run as the per-commit recording's oracle."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T, K, cap = 6000 + 7, 5, 60, 16, 50
    seg = np.array(HIST_PARTITIONS[part](P), dtype=np.int64)
    kw = {"default": {}, "downpour": dict(rule=1), "global_proxy": dict(proxy=1)}[mode]
    hp = _hp(G, **kw)
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=7)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 2)
        g.set_segments(seg)
        G.gem_pi_hist_start_segments(g.h, cap)
        with pytest.raises(G.GemError):      # the partition is fixed while recording
            g.set_segments([0, P])
        g.sim_run(worker, tau, K)
        got = G.gem_pi_hist_read(g.h, T, segments=seg.size - 1)
        theta = g.theta()
    st = O.State.initial(n, P)
    _, _, hist = O.run(_ohp(hp, 0.01, 0.1, 2), P, st, np.arange(P), h, ts, worker, tau,
                       pi_hist=True, hist_segments=seg)
    assert got.shape == (cap, seg.size - 1, G.GEM_PI_BINS)
    assert np.array_equal(got, hist[:cap])
    assert_parity("theta", theta, st.theta)
