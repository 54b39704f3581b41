"""Pins of the oracle's segment-norm scale factors (eq. 18 with Euclidean norms
over segments of the parameter vector: per tensor, or one global norm).

* Segments of one element turn the norms into absolute values, so the run must
  equal the element-wise oracle bit for bit, in every mode and for generated
  and given updates.
* The sum of squares that defines a norm: exact where every partial sum is
  exact (integer-valued terms), and within its error bound of an exactly
  rounded sum (math.fsum) otherwise, over ragged segment bounds and across
  the aligned 2^18-index blocks of its tree.
* One worker, no staleness: a single global segment with mu = 0 is plain SGD
  bit for bit; with momentum the committed update has exactly the proxy's norm
  (the compliance of eq. 13, in norm).
* The triangle inequality behind eqs. (11)-(13): with the clamped factor, the
  drift after a commit never exceeds the larger of the proxy's norm and the
  drift before it, segment by segment.
"""
import math

import numpy as np
import pytest

import oracle as O
from paper_1805_08469_amd.workloads import make_problem

UNIT_MODES = {
    "default": {},
    "literal": dict(pi_mode=O.PI_LITERAL),
    "kappa2": dict(kappa=2.0),
    "kappa3_sqrt": dict(kappa=3.0, kappa_mode=O.KAPPA_SQRT),
    "pre_pull": dict(pull_mode=O.PULL_PRE),
    "global_proxy": dict(proxy=O.PROXY_GLOBAL),
    "bf16": dict(bf16=True),
    "mu0": dict(momentum=0.0),
}


def _problem(P, seed=4):
    return make_problem(P, 1e-3, 1.0, seed)


@pytest.mark.parametrize("mode", sorted(UNIT_MODES))
def test_unit_segments_equal_elementwise(mode):
    P, n, T = 1500, 4, 60
    h, ts = _problem(P)
    hp = O.Hyper(lr=0.01, sigma=0.1, seed=3, **UNIT_MODES[mode])
    w, tau = O.schedule(n, T, O.LAW_EXP, 0, 0, seed=2, pull_mode=hp.pull_mode)
    st, st2 = O.State.initial(n, P), O.State.initial(n, P)
    O.run(hp, P, st, np.arange(P), h, ts, w, tau)
    O.run_segments(hp, st2, np.arange(P + 1), w, tau, h=h, ts=ts)
    for a, b in ((st.theta, st2.theta), (st.S, st2.S), (st.M, st2.M)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(st.pc, st2.pc)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unit_segments_equal_elementwise_given(dtype):
    P, n, K = 700, 3, 25
    rng = np.random.default_rng(5)
    d = (rng.standard_normal((K, P)) * 0.01).astype(np.float32)
    if dtype == "bf16":
        d = (O.round_bf16(d).view(np.uint32) >> 16).astype(np.uint16)
    w, tau = O.schedule(n, K, O.LAW_EXP, 0, 0, seed=6)
    hp = O.Hyper(momentum=0.9)
    st, st2 = O.State.initial(n, P), O.State.initial(n, P)
    O.commit_given(hp, st, w, d, tau)
    O.run_segments(hp, st2, np.arange(P + 1), w, tau, d=d)
    for a, b in ((st.theta, st2.theta), (st.S, st2.S), (st.M, st2.M)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("lo,hi", [(0, 1), (0, 1024), (3, 1025), (1000, 5000), (2047, 2049),
                                   (0, 9000), (5, 5), (262_000, 262_200), (1, 600_000)])
def test_sumsq_exact_on_integer_terms(lo, hi):
    """Integer terms below 2^10 keep every partial sum an integer below 2^53, so
    any order gives the exact sum: a dropped, repeated or misplaced term fails."""
    rng = np.random.default_rng(lo * 7 + hi)
    x = rng.integers(-1000, 1000, size=600_000).astype(np.float32)
    exact = sum(int(v) * int(v) for v in x[lo:hi])
    assert O.sumsq(x, lo, hi) == float(exact)


@pytest.mark.parametrize("size,seed", [(1, 0), (1023, 1), (1025, 2), (50_000, 3),
                                       (600_001, 4)])
def test_sumsq_within_error_bound(size, seed):
    """Against the exactly rounded sum: each of the (log2 2^18 + blocks) levels
    of additions contributes at most one rounding of relative 2^-53."""
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(size) * np.exp(rng.uniform(-20, 20, size))).astype(np.float32)
    lo, hi = size // 7, size
    ref = math.fsum(float(v) * float(v) for v in x[lo:hi])
    levels = 18 + (hi - 1) // 2 ** 18 - lo // 2 ** 18 + 1
    got = O.sumsq(x, lo, hi)
    assert abs(got - ref) <= levels * 2.0 ** -53 * ref


def test_global_norm_n1_mu0_is_sgd_bitwise():
    """One worker without staleness and mu = 0: m = dtheta and theta = s, so the
    global factor is ||d|| / (||d|| + eps) = 1 once eps is absorbed, and
    every commit is theta + dtheta."""
    P, T = 3000, 40
    h, ts = _problem(P, 8)
    hp = O.Hyper(lr=0.05, sigma=0.1, momentum=0.0, seed=11)
    w = np.zeros(T, dtype=np.int32)
    st = O.State.initial(1, P)
    pi, tr = O.run_segments(hp, st, [0, P], w, h=h, ts=ts, pi=True, trace=True)
    assert np.all(pi == 1.0)
    theta = np.zeros(P, dtype=np.float32)
    for j in range(T):
        theta = (theta + tr[j, :, 1]).astype(np.float32)
    assert np.array_equal(theta, st.theta)


@pytest.mark.parametrize("kappa", [1.0, 2.0])
def test_global_norm_n1_update_has_the_proxy_norm(kappa):
    """One worker without staleness: theta_t = s_t, so pi = k ||m|| / (||d|| + eps)
    and the committed update pi d has norm k ||m|| (eq. 13 with norms), up to
    the roundings of the norms and of pi."""
    P, T = 2000, 30
    h, ts = _problem(P, 9)
    hp = O.Hyper(lr=0.02, sigma=0.1, momentum=0.9, kappa=kappa, seed=12)
    w = np.zeros(T, dtype=np.int32)
    st = O.State.initial(1, P)
    pi, tr = O.run_segments(hp, st, [0, P], w, h=h, ts=ts, pi=True, trace=True)
    for j in range(T):
        a, d, m = (tr[j, :, k].astype(np.float64) for k in range(3))
        assert np.all(a == 0.0)
        psi = float(pi[j, 0]) * np.linalg.norm(d)
        assert psi == pytest.approx(kappa * np.linalg.norm(m), rel=2e-6)


@pytest.mark.parametrize("n", [4, 20])
def test_segment_drift_bound(n):
    """Triangle inequality: for pi >= 0, ||a + pi d|| <= ||a|| + pi ||d||, and pi ||d||
    <= k ||m|| - ||a|| when pi > 0, so the drift after a commit is at most
    max(k ||m||, ||a||) per segment (evaluated in binary64 on the step's
    binary32 operands; relative slack for the roundings of pi and the norms)."""
    P, T = 2500, 200
    h, ts = _problem(P, 10)
    hp = O.Hyper(lr=0.01, sigma=0.1, momentum=0.9, seed=13)
    w, tau = O.schedule(n, T, O.LAW_EXP, 0, 0, seed=n)
    seg = [0, 17, 1024, 1100, 2048, P]
    st = O.State.initial(n, P)
    pi, tr = O.run_segments(hp, st, seg, w, tau, h=h, ts=ts, pi=True, trace=True)
    assert np.all(pi >= 0.0)
    clamped = 0
    for j in range(T):
        for k in range(len(seg) - 1):
            sl = slice(seg[k], seg[k + 1])
            a, d, m = (tr[j, sl, q].astype(np.float64) for q in range(3))
            after = np.linalg.norm(a + float(pi[j, k]) * d)
            bound = max(np.linalg.norm(m), np.linalg.norm(a))
            assert after <= bound * (1 + 1e-6) + 1e-30, (j, k, after, bound)
            clamped += int(pi[j, k] == 0.0)
    assert 0 < clamped < T * (len(seg) - 1)


def test_bad_segments_rejected():
    P, n = 100, 2
    w = np.zeros(1, dtype=np.int32)
    h, ts = _problem(P)
    for seg in ([0, 50], [1, P], [0, 50, 50, P], [0, 60, 40, P]):
        with pytest.raises(O.OracleError):
            O.run_segments(O.Hyper(), O.State.initial(n, P), seg, w, h=h, ts=ts)
    with pytest.raises(O.OracleError):
        O.run_segments(O.Hyper(rule=O.RULE_DOWNPOUR), O.State.initial(n, P), [0, P], w,
                       h=h, ts=ts)


def test_unit_segments_diagnostics_equal_elementwise():
    """The energy diagnostics of a one-element-segment run equal the
    element-wise run's, commit by commit (same terms, same order)."""
    P, n, T = 1200, 4, 50
    h, ts = _problem(P, 21)
    hp = O.Hyper(lr=0.01, sigma=0.1, seed=4)
    w, tau = O.schedule(n, T, O.LAW_EXP, 0, 0, seed=21)
    dg, _ = O.run(hp, P, O.State.initial(n, P), np.arange(P), h, ts, w, tau, diag=True)
    _, _, dgs = O.run_segments(hp, O.State.initial(n, P), np.arange(P + 1), w, tau, h=h, ts=ts,
                               diag=True)
    assert np.array_equal(dg, dgs)
    assert dg["n_clamped"].sum() > 0
