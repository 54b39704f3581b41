"""Seeded synthetic workloads for the GEM commit pipeline.

This module only describes workloads and draws their fixed inputs (the
diagonal quadratic's curvatures h and minimiser theta*); it holds none of
the method's arithmetic.  The library, the benchmark and the test suite all
take their inputs from here.

The five workloads mirror the sizes the method is exercised at: a tiny
parity case, a small-CNN-sized parameter vector, a ResNet-18-sized one, the
headline 25M-parameter / 100-worker case, and a 124M-parameter case with
bfloat16 worker updates.  Hyper-parameters default to Alg. 1's eta = 0.01,
mu = 0.9, eps = 1e-16 unless a workload states otherwise.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

# Compute-time laws of the simulated workers (values match the C-ABI enum).
LAW_EXP = 0               # exponential, mean 1 for every worker
LAW_EXP_UNIFORM_MEAN = 1  # exponential, per-worker mean ~ U[p0, p1]
LAW_EXP_LOGNORMAL_MEAN = 2  # exponential, per-worker mean ~ LogNormal(p0, p1)
LAW_PARETO = 3            # Pareto, shape p0, scale p1 (same law for every worker)


@dataclass(frozen=True)
class Workload:
    name: str
    P: int            # parameters
    n: int            # asynchronous workers
    T: int            # commits
    K: int            # commits fused per pass
    h_lo: float       # curvature h_i ~ LogUniform[h_lo, h_hi]
    h_hi: float
    sigma: float      # gradient noise N(0, sigma^2)
    lr: float         # eta
    momentum: float   # mu
    law: int
    law_p0: float
    law_p1: float
    bf16: bool = False  # workers send bfloat16 updates
    seed: int = 20180522

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", P=4096, n=4, T=2000, K=1, h_lo=1e-3, h_hi=1.0, sigma=0.1,
                     lr=0.01, momentum=0.9, law=LAW_EXP, law_p0=0.0, law_p1=0.0),
    "small": Workload("small", P=1_200_000, n=20, T=10_000, K=1, h_lo=1e-4, h_hi=1.0,
                      sigma=0.05, lr=0.005, momentum=0.9, law=LAW_EXP_UNIFORM_MEAN,
                      law_p0=0.8, law_p1=1.2),
    "resnet18": Workload("resnet18", P=11_700_000, n=50, T=5000, K=8, h_lo=1e-4, h_hi=1.0,
                         sigma=0.05, lr=0.01, momentum=0.9, law=LAW_EXP, law_p0=0.0,
                         law_p1=0.0),
    "headline": Workload("headline", P=25_000_000, n=100, T=5000, K=32, h_lo=1e-4, h_hi=1.0,
                         sigma=0.02, lr=0.01, momentum=0.9, law=LAW_EXP_LOGNORMAL_MEAN,
                         law_p0=0.0, law_p1=0.5),
    "large": Workload("large", P=124_000_000, n=100, T=1000, K=16, h_lo=1e-4, h_hi=1.0,
                      sigma=0.02, lr=0.01, momentum=0.9, law=LAW_PARETO, law_p0=1.5,
                      law_p1=1.0 / 3.0, bf16=True),
}


def make_problem(P: int, h_lo: float, h_hi: float, seed: int,
                 chunk: int = 1 << 24) -> tuple[np.ndarray, np.ndarray]:
    """Curvatures h ~ LogUniform[h_lo, h_hi] and minimiser theta* ~ N(0, 1).

    Drawn in binary64 from two independent PCG64 streams and rounded to
    binary32; generated in chunks so that a prefix of a larger problem equals
    the smaller problem.
    """
    rng_h = np.random.default_rng([seed, 1])
    rng_t = np.random.default_rng([seed, 2])
    h = np.empty(P, dtype=np.float32)
    ts = np.empty(P, dtype=np.float32)
    lo, hi = np.log(h_lo), np.log(h_hi)
    for i0 in range(0, P, chunk):
        m = min(chunk, P - i0)
        u = rng_h.random(m)
        h[i0:i0 + m] = np.exp(lo + (hi - lo) * u)
        ts[i0:i0 + m] = rng_t.standard_normal(m)
    return h, ts


def problem(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    return make_problem(w.P, w.h_lo, w.h_hi, w.seed)
