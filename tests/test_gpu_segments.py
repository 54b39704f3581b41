"""GPU parity of the segment-norm scale factors (one pi per segment of the
parameter vector, from Euclidean norms) against the oracle: theta, every S[w]
and M[w], bit for bit, for generated and given updates, ragged sizes and
partitions (one global segment, segments inside and across the 1024-index
groups of the sums, one-element segments), every mode the scope supports,
sums spanning several 2^18-index blocks, and a headline-sized vector."""
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


def _hp(G, **kw):
    hp = G.gem_hyperparams_default()
    hp.pi_scope = G.GEM_PI_SEGMENT
    for k, v in kw.items():
        setattr(hp, k, v)
    return hp


def _ohp(hp, lr, sigma, seed, bf16=False):
    return O.Hyper(lr=lr, sigma=sigma, momentum=hp.momentum, eps=hp.eps, kappa=hp.kappa,
                   pi_mode=hp.pi_mode, kappa_mode=hp.kappa_mode, pull_mode=hp.pull_mode,
                   rule=hp.rule, bf16=bf16, proxy=hp.proxy_mode, seed=seed)


def _partition(kind, P):
    if kind == "global":
        return np.array([0, P], dtype=np.int64)
    if kind == "unit":
        return np.arange(P + 1, dtype=np.int64)
    if kind == "ragged":
        cuts = [c for c in (17, 1024, 1100, 2053, 2054, 4096, 4097, 262_143, 262_145, 524_288)
                if c < P]
        return np.array([0, *cuts, P], dtype=np.int64)
    if kind == "tensors":
        # a model-like mix: large weight tensors with small bias/scale vectors between them
        rng = np.random.default_rng(P)
        sizes = []
        while sum(sizes) < P:
            sizes.append(int(rng.choice([64, 128, 3 * 3 * 64 * 64, 7, 1, 512, 5000])))
        off = np.concatenate([[0], np.cumsum(sizes)])
        off = off[off < P]
        return np.concatenate([off, [P]]).astype(np.int64)
    raise ValueError(kind)


def _run_both(G, P, n, worker, tau, hp, seg, lr=0.01, sigma=0.1, seed=7, bf16=False):
    from paper_1805_08469_amd.workloads import make_problem
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, lr, sigma, seed, bf16=bf16)
        if seg is not None:
            g.set_segments(seg)
        g.sim_run(worker, tau, 8)
        out = (g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, g.stats())
    st = O.State.initial(n, P)
    O.run_segments(_ohp(hp, lr, sigma, seed, bf16), st,
                   seg if seg is not None else [0, P], worker, tau, h=h, ts=ts)
    return out, st


def _check(out, st, tag):
    theta, S, M, pc, clock, _ = out
    assert clock == st.t
    assert np.array_equal(pc, st.pc), f"{tag} pull clocks"
    assert_parity(f"{tag} theta", theta, st.theta)
    assert_parity(f"{tag} S", S, st.S)
    assert_parity(f"{tag} M", M, st.M)


# one-element segments only at the smaller sizes (one reduction block per element)
PARTITIONS = [(k, P) for P in (300, 5003, 20_000, 600_001)
              for k in ("global", "ragged", "tensors", "unit") if k != "unit" or P <= 5003]


@pytest.mark.parametrize("kind,P", PARTITIONS)
def test_partitions(G, kind, P):
    n, T = 5, 40
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=P)
    print(f"[segments {kind}] P={P} n={n} T={T}", flush=True)
    out, st = _run_both(G, P, n, worker, tau, _hp(G), _partition(kind, P))
    _check(out, st, f"{kind} P={P}")
    assert out[5].passes == T


def test_default_is_one_global_segment(G):
    P, n, T = 4099, 3, 30
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=1)
    out, st = _run_both(G, P, n, worker, tau, _hp(G), None)
    _check(out, st, "default")


MODES = {
    "literal": dict(pi_mode=1),
    "kappa2": dict(kappa=2.0),
    "kappa3_sqrt": dict(kappa=3.0, kappa_mode=1),
    "pre_pull": dict(pull_mode=1),
    "global_proxy": dict(proxy_mode=1),
    "mu0": dict(momentum=0.0),
}


@pytest.mark.parametrize("mode", sorted(MODES))
def test_modes(G, mode):
    P, n, T = 6000, 4, 50
    hp = _hp(G, **MODES[mode])
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=9, pull_mode=hp.pull_mode)
    out, st = _run_both(G, P, n, worker, tau, hp, _partition("ragged", P))
    _check(out, st, mode)


def test_bf16_updates(G):
    P, n, T = 5000, 6, 40
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_PARETO, 1.5, 1 / 3, seed=4)
    out, st = _run_both(G, P, n, worker, tau, _hp(G), _partition("tensors", P), sigma=0.02,
                        bf16=True)
    _check(out, st, "bf16")


def test_same_worker_back_to_back(G):
    """A worker committing twice in a row reads the snapshot its first commit
    just pulled (taken from registers in the step that applies it)."""
    n = 3
    worker = np.array([0, 0, 0, 1, 1, 2, 0, 0, 2, 2, 2, 1], dtype=np.int32)
    pc = np.zeros(n, dtype=np.int64)
    tau = []
    for t, w in enumerate(worker):
        tau.append(t - pc[w])
        pc[w] = t + 1
    tau = np.array(tau, dtype=np.int32)
    for kind in ("global", "ragged"):
        out, st = _run_both(G, 4500, n, worker, tau, _hp(G), _partition(kind, 4500))
        _check(out, st, f"back-to-back {kind}")


def test_unit_segments_equal_element_scope(G):
    """One-element segments are element-wise GEM: the two GPU paths agree bit
    for bit."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 2500, 4, 60
    h, ts = make_problem(P, 1e-3, 1.0, 5)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=5)
    res = []
    for scope in (G.GEM_PI_ELEMENT, G.GEM_PI_SEGMENT):
        hp = G.gem_hyperparams_default()
        hp.pi_scope = scope
        with G.Gem(P, n, hp) as g:
            g.set_quadratic(h, ts, 0.01, 0.1, 6)
            g.set_segments(np.arange(P + 1))
            g.sim_run(worker, tau, 16)
            res.append((g.theta(), g.S(), g.M()))
    for a, b, name in zip(res[0], res[1], ("theta", "S", "M")):
        assert_parity(name, b, a)


def _device_rows(torch, arr):
    """Device copies of update rows, each 16-byte aligned."""
    K, P = arr.shape
    stride = (P + 7) // 8 * 8
    buf = torch.zeros((K, stride), dtype=torch.float32 if arr.dtype == np.float32 else torch.int16,
                      device="cuda")
    buf[:, :P] = torch.from_numpy(arr.view(np.int16) if arr.dtype == np.uint16 else arr).cuda()
    return buf, [buf[j].data_ptr() for j in range(K)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_given_updates(G, dtype):
    import torch
    P, n, K = 3001, 4, 30
    rng = np.random.default_rng(8)
    d = (rng.standard_normal((K, P)) * 0.01).astype(np.float32)
    if dtype == "bf16":
        d = (O.round_bf16(d).view(np.uint32) >> 16).astype(np.uint16)
    worker, tau = G.gem_schedule_make(n, K, G.GEM_LAW_EXP, seed=2)
    seg = _partition("ragged", P)
    buf, ptrs = _device_rows(torch, d)
    hp = _hp(G)
    with G.Gem(P, n, hp) as g:
        g.set_segments(seg)
        g.commit_batch(ptrs[:10], G.GEM_F32 if dtype == "f32" else G.GEM_BF16, worker[:10],
                       tau[:10])
        for j in range(10, K):   # one by one through the batch entry point
            g.commit_batch(ptrs[j:j + 1], G.GEM_F32 if dtype == "f32" else G.GEM_BF16,
                           worker[j:j + 1], tau[j:j + 1])
        torch.cuda.synchronize()
        out = (g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, g.stats())
    st = O.State.initial(n, P)
    O.run_segments(_ohp(hp, 0.0, 0.0, 0), st, seg, worker, tau, d=d)
    _check(out, st, f"given {dtype}")


@pytest.mark.parametrize("per_segment", [False, True])
def test_pi_histograms(G, per_segment):
    """Histograms under the segment scope: each commit counts every element of
    a segment in the bin of that segment's factor (the oracle's pi per segment
    and commit, binned by the oracle)."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T, cap = 7000, 4, 30, 25
    seg = _partition("tensors", P)
    nseg = seg.size - 1
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=3)
    hp = _hp(G)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 7)
        g.set_segments(seg)
        if per_segment:
            G.gem_pi_hist_start_segments(g.h, cap)
        else:
            G.gem_pi_hist_start(g.h, cap)
        g.sim_run(worker, tau, 8)
        got = G.gem_pi_hist_read(g.h, T, segments=nseg if per_segment else 0)
    st = O.State.initial(n, P)
    pi, _ = O.run_segments(_ohp(hp, 0.01, 0.1, 7), st, seg, worker, tau, h=h, ts=ts, pi=True)
    bins = O.pi_bin(pi)                                   # [T, nseg]
    size = np.diff(seg)
    want = np.zeros((cap, nseg if per_segment else 1, G.GEM_PI_BINS), dtype=np.uint32)
    for j in range(cap):
        for k in range(nseg):
            want[j, k if per_segment else 0, bins[j, k]] += size[k]
    assert np.array_equal(got, want if per_segment else want[:, 0])


@pytest.mark.parametrize("mode", ["default", "pre_pull", "global_proxy", "kappa3_sqrt"])
def test_diagnostics(G, mode):
    """The energy sums (eqs. 11 and 22) and the clamp count under the segment
    scope, against the oracle's per-commit diagnostics."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 9001, 4, 40
    kw = {"default": {}, "pre_pull": dict(pull_mode=1), "global_proxy": dict(proxy_mode=1),
          "kappa3_sqrt": dict(kappa=3.0, kappa_mode=1)}[mode]
    hp = _hp(G, **kw)
    seg = _partition("tensors", P)
    h, ts = make_problem(P, 1e-3, 1.0, 5)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=5, pull_mode=hp.pull_mode)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 9)
        g.set_segments(seg)
        G.gem_diag_enable(g.h, True)
        g.sim_run(worker[:15], tau[:15], 8)
        G.gem_diag_reset(g.h)
        g.sim_run(worker[15:], tau[15:], 8)
        d = G.gem_diag(g.h)
        theta = g.theta()
    st = O.State.initial(n, P)
    _, _, dg = O.run_segments(_ohp(hp, 0.01, 0.1, 9), st, seg, worker, tau, h=h, ts=ts, diag=True)
    later = dg[15:]
    assert d.n_commits == T - 15
    assert d.n_elem_commits == P * (T - 15)
    assert d.n_clamped == int(later["n_clamped"].sum())
    assert d.sum_ek == pytest.approx(float(later["sum_ek"].sum()), rel=1e-9)
    assert d.sum_proxy == pytest.approx(float(later["sum_proxy"].sum()), rel=1e-9)
    assert d.loss == pytest.approx(O.loss(st.theta, h, ts), rel=1e-10)
    assert_parity("theta", theta, st.theta)


def test_rejections(G):
    P, n = 1000, 2
    hp = _hp(G)
    hp.rule = G.GEM_RULE_DOWNPOUR
    with pytest.raises(G.GemError):
        G.Gem(P, n, hp)
    with G.Gem(P, n, _hp(G)) as g:
        for seg in ([0, 500], [1, P], [0, 500, 500, P], [0, 600, 400, P]):
            with pytest.raises(G.GemError):
                g.set_segments(seg)
        worker, tau = G.gem_schedule_make(n, 4, G.GEM_LAW_EXP, seed=1)
        with pytest.raises(G.GemError):      # no problem set
            g.sim_run(worker, tau, 4)
        assert g.clock == 0


def test_segment_factors_repeat_bit_for_bit(G):
    """The last block of each segment's index-block sums forms its factor, found
    by a device-scope counter between fences: whichever block that is, every
    sum keeps its order.  Five runs of the same schedule on fresh handles, with
    segments of many index blocks and segments inside one, give identical
    state and factor histograms, equal to the oracle."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 5 * 262_144 + 777, 3, 60
    seg = np.array([0, 100, 262_144 + 5, 262_144 + 6, 3 * 262_144 + 11, P], dtype=np.int64)
    h, ts = make_problem(P, 1e-3, 1.0, 21)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=21)
    hp = _hp(G)
    runs = []
    for r in range(5):
        print(f"[segments repeat] run {r} P={P} nseg={seg.size - 1}", flush=True)
        with G.Gem(P, n, hp) as g:
            g.set_quadratic(h, ts, 0.01, 0.1, 5)
            g.set_segments(seg)
            G.gem_pi_hist_start_segments(g.h, T)
            g.sim_run(worker, tau, 8)
            runs.append((g.theta(), g.S(), g.M(),
                         G.gem_pi_hist_read(g.h, T, segments=seg.size - 1)))
    for r in range(1, 5):
        for a, b in zip(runs[0], runs[r]):
            assert np.array_equal(a, b), f"run {r} differs from run 0"
    st = O.State.initial(n, P)
    O.run_segments(_ohp(hp, 0.01, 0.1, 5), st, seg, worker, tau, h=h, ts=ts)
    assert_parity("repeat theta", runs[0][0], st.theta)
    assert_parity("repeat S", runs[0][1], st.S)
    assert_parity("repeat M", runs[0][2], st.M)


@pytest.mark.parametrize("bf16", [False, True])
def test_cache_policies_give_the_same_bits(G, bf16):
    """Streaming (non-temporal) and default-policy step kernels give the same
    state, bit for bit, equal to the oracle (a small state, where AUTO keeps
    the default policy and STREAM is forced)."""
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 3 * 1024 + 333, 4, 50
    seg = _partition("ragged", P)
    h, ts = make_problem(P, 1e-3, 1.0, 13)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=13)
    hp = _hp(G)
    states = {}
    for policy in (G.GEM_CACHE_KEEP, G.GEM_CACHE_STREAM):
        with G.Gem(P, n, hp) as g:
            g.set_cache_policy(policy)
            g.set_quadratic(h, ts, 0.01, 0.1, 3, bf16=bf16)
            g.set_segments(seg)
            g.sim_run(worker, tau, 8)
            states[policy] = (g.theta(), g.S(), g.M())
    for a, b in zip(states[G.GEM_CACHE_KEEP], states[G.GEM_CACHE_STREAM]):
        assert np.array_equal(a, b)
    st = O.State.initial(n, P)
    O.run_segments(_ohp(hp, 0.01, 0.1, 3, bf16), st, seg, worker, tau, h=h, ts=ts)
    assert_parity("stream theta", states[G.GEM_CACHE_STREAM][0], st.theta)
    assert_parity("stream S", states[G.GEM_CACHE_STREAM][1], st.S)
    assert_parity("stream M", states[G.GEM_CACHE_STREAM][2], st.M)


def test_extreme_update_magnitudes(G):
    """Caller updates of every magnitude (subnormal, huge, infinite, NaN)
    under per-segment factors: the binary64 sums of squares overflow, turn
    infinite or NaN in some segments and not in others, and the state stays
    equal to the oracle's (NaN compares equal to NaN)."""
    import torch
    P, n, T = 3000, 3, 24
    rng = np.random.default_rng(41)
    d = (rng.standard_normal((T, P)) * 0.01).astype(np.float32)
    ext = np.array([0.0, -0.0, 1e-45, -1e-40, 1e-30, 1e20, -1e30, 3e38, np.inf, -np.inf, np.nan],
                   dtype=np.float32)
    pick = rng.random((T, P)) < 0.002
    d[pick] = rng.choice(ext, size=int(pick.sum()))
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=41)
    seg = _partition("ragged", P)
    buf, ptrs = _device_rows(torch, d)
    hp = _hp(G)
    with G.Gem(P, n, hp) as g:
        g.set_segments(seg)
        g.commit_batch(ptrs, G.GEM_F32, worker, tau)
        torch.cuda.synchronize()
        out = (g.theta(), g.S(), g.M(), g.pull_clocks(), g.clock, g.stats())
    st = O.State.initial(n, P)
    with np.errstate(all="ignore"):
        O.run_segments(_ohp(hp, 0.0, 0.0, 0), st, seg, worker, tau, d=d)
    assert np.isfinite(st.theta).any() and not np.isfinite(st.theta).all()
    _check(out, st, "extremes")


def test_headline_size_global_norm(G):
    """A 25M-parameter vector (the headline size) with four workers: one global
    segment and a model-like partition, a few commits, against the oracle on
    every element of theta and sampled elements of S and M."""
    import torch
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 25_000_000, 4, 3
    free, _ = torch.cuda.mem_get_info()
    if free < 4 * P * (3 * n + 6):
        pytest.skip("not enough device memory")
    h, ts = make_problem(P, 1e-4, 1.0, 11)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=11)
    idx = np.unique(np.concatenate([[0, 1, 1023, 1024, P // 2, P - 2, P - 1],
                                    np.random.default_rng(1).integers(0, P, 2000)]))
    for kind in ("global", "tensors"):
        seg = _partition(kind, P)
        print(f"[segments headline {kind}] P={P} nseg={seg.size - 1}", flush=True)
        hp = _hp(G)
        with G.Gem(P, n, hp) as g:
            g.set_quadratic(h, ts, 0.01, 0.02, 20180522)
            g.set_segments(seg)
            g.sim_run(worker, tau, 8)
            theta = g.theta()
            _, S, M = g.gather(idx)
        st = O.State.initial(n, P)
        O.run_segments(_ohp(hp, 0.01, 0.02, 20180522), st, seg, worker, tau, h=h, ts=ts)
        assert_parity(f"headline {kind} theta", theta, st.theta)
        assert_parity(f"headline {kind} S", S, st.S[:, idx])
        assert_parity(f"headline {kind} M", M, st.M[:, idx])
