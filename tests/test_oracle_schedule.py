"""Pins of the oracle's queuing schedule (Sec. 1, eq. 2).

With homogeneous exponential compute times the system is memoryless: every
commit belongs to a uniformly random worker, independently, so the staleness
tau (the number of other commits between a worker's pull and its commit) is
Geometric(1/n) with mean n - 1 -- the expected staleness the paper quotes for
a homogeneous queue.  Heterogeneous laws are checked against their own
means; the structural identity tau_t = t - (previous commit of w_t + 1) holds
for every law.
"""
import numpy as np
import pytest
from scipy import stats

import oracle as O


@pytest.mark.parametrize("n", [4, 20, 100])
def test_homogeneous_queue_mean_staleness(n):
    T = 60_000
    w, tau = O.schedule(n, T, O.LAW_EXP, seed=n)
    # workers iid uniform: chi-square on counts
    counts = np.bincount(w, minlength=n)
    assert stats.chisquare(counts).pvalue > 1e-4
    # staleness after each worker's first commit ~ Geometric(1/n) - 1, mean n-1
    first = np.zeros(T, bool)
    seen = set()
    for t, ww in enumerate(w):
        if ww not in seen:
            first[t] = True
            seen.add(ww)
    x = tau[~first].astype(np.float64)
    se = np.sqrt((n - 1) * n / x.size)  # sd of Geometric failures = sqrt(n(n-1))
    assert abs(x.mean() - (n - 1)) < 5 * se
    # distribution: P(tau = k) = (1/n)(1-1/n)^k, binned
    p = 1.0 / n
    edges = np.unique(np.round(np.quantile(x, np.linspace(0, 1, 21))).astype(int))
    obs = np.histogram(x, bins=np.append(edges, np.inf))[0]
    cdf = lambda k: 1 - (1 - p) ** np.asarray(k, dtype=np.float64)
    exp_p = np.diff(np.append(cdf(edges), 1.0))
    exp_p[0] += cdf(edges[0])
    exp_c = exp_p * x.size
    keep = exp_c > 20
    chi2 = ((obs[keep] - exp_c[keep]) ** 2 / exp_c[keep]).sum()
    assert stats.chi2.sf(chi2, keep.sum() - 1) > 1e-4


@pytest.mark.parametrize("law,p0,p1,pull", [
    (O.LAW_EXP, 0, 0, O.PULL_POST), (O.LAW_EXP_UNIFORM_MEAN, 0.8, 1.2, O.PULL_POST),
    (O.LAW_EXP_LOGNORMAL_MEAN, 0.0, 0.5, O.PULL_POST), (O.LAW_PARETO, 1.5, 1 / 3, O.PULL_POST),
    (O.LAW_EXP, 0, 0, O.PULL_PRE)])
def test_structural_tau_identity(law, p0, p1, pull):
    n, T = 17, 5000
    w, tau = O.schedule(n, T, law, p0, p1, seed=5, pull_mode=pull)
    last = np.full(n, -1)
    for t in range(T):
        ww = w[t]
        prev_pull = 0 if last[ww] < 0 else (last[ww] + (1 if pull == O.PULL_POST else 0))
        assert tau[t] == t - prev_pull
        last[ww] = t
    assert np.all(tau >= 0)


def test_heterogeneous_speeds_shift_commit_shares():
    """Per-worker exponential means: the long-run commit share of worker w is
    proportional to its rate 1/mean_w."""
    n, T, seed = 10, 80_000, 3
    w, _ = O.schedule(n, T, O.LAW_EXP_LOGNORMAL_MEAN, 0.0, 0.5, seed=seed)
    means = np.array([O.worker_mean(O.LAW_EXP_LOGNORMAL_MEAN, 0.0, 0.5, seed, k) for k in range(n)])
    share = np.bincount(w, minlength=n) / T
    expect = (1 / means) / (1 / means).sum()
    assert np.allclose(share, expect, rtol=0.05)
    means_u = np.array([O.worker_mean(O.LAW_EXP_UNIFORM_MEAN, 0.8, 1.2, 1, k) for k in range(1000)])
    assert means_u.min() >= 0.8 and means_u.max() < 1.2 and abs(means_u.mean() - 1.0) < 0.02


def test_pareto_job_times():
    """Pareto(alpha = 1.5, x_m = 1/3): support [x_m, inf), mean alpha x_m/(alpha-1) = 1,
    survival (x_m/x)^alpha."""
    x = np.array([O.job_time(O.LAW_PARETO, 1.5, 1 / 3, 1.0, 4, w, k)
                  for w in range(20) for k in range(2000)])
    assert x.min() >= 1 / 3
    for q in (1.0, 3.0, 10.0):
        emp = (x > q).mean()
        assert emp == pytest.approx((1 / 3 / q) ** 1.5, rel=0.1)


def test_exponential_job_times():
    x = np.array([O.job_time(O.LAW_EXP, 0, 0, 2.0, 4, w, k) for w in range(10) for k in range(4000)])
    assert stats.kstest(x, "expon", args=(0, 2.0)).pvalue > 1e-3
