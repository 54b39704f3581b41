"""CPU oracle for Gradient Energy Matching -- TEST INFRASTRUCTURE ONLY.

A ctypes view of ``libgem_oracle.so`` (plain single-threaded C, built from
``gem_oracle.c`` by ``oracle/build.py``).  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import this package; the HIP
library never does, and the two share no code.

Every function documents the passage of Hermans & Louppe (arXiv 1805.08469)
that it follows; see ``gem_oracle.c`` for the binary32 operation order.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgem_oracle.so")

PI_CLAMP0, PI_LITERAL = 0, 1
KAPPA_LINEAR, KAPPA_SQRT = 0, 1
PULL_POST, PULL_PRE = 0, 1
RULE_GEM, RULE_DOWNPOUR, RULE_ADAPTIVE = 0, 1, 2
PROXY_LOCAL, PROXY_GLOBAL = 0, 1
LAW_EXP, LAW_EXP_UNIFORM_MEAN, LAW_EXP_LOGNORMAL_MEAN, LAW_PARETO = 0, 1, 2, 3

OK, EINVAL, ENOMEM, EWORKER, ESTALE = 0, -1, -2, -3, -4
PI_BINS = 643


class OracleConfig(C.Structure):
    _fields_ = [
        ("P", C.c_int64),
        ("n", C.c_int32),
        ("lr", C.c_float),
        ("sigma", C.c_float),
        ("momentum", C.c_float),
        ("eps", C.c_float),
        ("kappa", C.c_float),
        ("pi_mode", C.c_int32),
        ("kappa_mode", C.c_int32),
        ("pull_mode", C.c_int32),
        ("rule", C.c_int32),
        ("bf16", C.c_int32),
        ("proxy", C.c_int32),
        ("seed", C.c_uint64),
    ]


COMMIT_DIAG_DTYPE = np.dtype([("sum_ek", np.float64), ("sum_proxy", np.float64),
                              ("n_clamped", np.int64), ("pad", np.int64)])


def _ptr(a, ctype):
    return a.ctypes.data_as(C.POINTER(ctype)) if a is not None else None


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(_LIB_PATH)
        u32p, u64p = C.POINTER(C.c_uint32), C.POINTER(C.c_uint64)
        f32p, i32p, i64p = C.POINTER(C.c_float), C.POINTER(C.c_int32), C.POINTER(C.c_int64)
        L.or_philox4x32.argtypes = [u32p, u32p, C.c_int, u32p]
        L.or_philox4x64.argtypes = [u64p, u64p, C.c_int, u64p]
        L.or_philox_weyl32.restype = C.c_uint32
        L.or_philox_weyl32.argtypes = [C.c_int]
        L.or_philox_weyl64.restype = C.c_uint64
        L.or_philox_weyl64.argtypes = [C.c_int]
        L.or_ln2_lo.restype = C.c_float
        L.or_log_unit_array.argtypes = [f32p, f32p, C.c_int64]
        L.or_sincos_turn24_array.argtypes = [u32p, f32p, f32p, C.c_int64]
        L.or_round_bf16_array.argtypes = [f32p, f32p, C.c_int64]
        L.or_normals.argtypes = [C.c_uint64, C.c_uint32, C.c_int64, C.c_int64, f32p]
        L.or_normals_at.argtypes = [C.c_uint64, C.c_uint32, i64p, C.c_int64, f32p]
        L.or_worker_mean.restype = C.c_double
        L.or_worker_mean.argtypes = [C.c_int32, C.c_double, C.c_double, C.c_uint64, C.c_int32]
        L.or_job_time.restype = C.c_double
        L.or_job_time.argtypes = [C.c_int32, C.c_double, C.c_double, C.c_double, C.c_uint64,
                                  C.c_int32, C.c_int64]
        L.or_schedule.restype = C.c_int
        L.or_schedule.argtypes = [C.c_int32, C.c_int64, C.c_int32, C.c_double, C.c_double,
                                  C.c_uint64, C.c_int32, i32p, i32p]
        L.or_run.restype = C.c_int
        L.or_run.argtypes = [C.POINTER(OracleConfig), i64p, C.c_int64, f32p, f32p,
                             f32p, f32p, f32p, i64p, C.c_int64, i32p, i32p, C.c_int64,
                             C.c_void_p, f32p, C.POINTER(C.c_uint32), C.c_int32, i64p]
        L.or_commit_given.restype = C.c_int
        L.or_commit_given.argtypes = [C.POINTER(OracleConfig), C.c_int64, f32p, f32p, f32p,
                                      i64p, C.c_int64, i32p, i32p, C.c_int64, f32p,
                                      C.POINTER(C.c_uint16), C.c_void_p, f32p,
                                      C.POINTER(C.c_uint32)]
        L.or_sumsq.restype = C.c_double
        L.or_sumsq.argtypes = [f32p, C.c_int64, C.c_int64]
        L.or_run_segments.restype = C.c_int
        L.or_run_segments.argtypes = [C.POINTER(OracleConfig), C.c_int32, i64p, f32p, f32p,
                                      f32p, f32p, f32p, i64p, C.c_int64, i32p, i32p, C.c_int64,
                                      f32p, C.POINTER(C.c_uint16), f32p, f32p, C.c_void_p]
        L.or_pi_bin.restype = C.c_int
        L.or_pi_bin.argtypes = [C.c_float]
        L.or_pi_bin_array.argtypes = [f32p, i32p, C.c_int64]
        L.or_loss.restype = C.c_double
        L.or_loss.argtypes = [f32p, f32p, f32p, C.c_int64]
        _lib = L
    return _lib


# --------------------------------------------------------------------------
# Random numbers (Philox4x32-10, Salmon et al. SC'11; Box & Muller 1958)
# --------------------------------------------------------------------------
def philox4x32(ctr, key, rounds: int = 10) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().or_philox4x32(_ptr(c, C.c_uint32), _ptr(k, C.c_uint32), rounds, _ptr(out, C.c_uint32))
    return out


def philox4x64(ctr, key, rounds: int = 10) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().or_philox4x64(_ptr(c, C.c_uint64), _ptr(k, C.c_uint64), rounds, _ptr(out, C.c_uint64))
    return out


def philox_weyl32(which: int) -> int:
    return int(lib().or_philox_weyl32(which))


def philox_weyl64(which: int) -> int:
    return int(lib().or_philox_weyl64(which))


def ln2_lo() -> float:
    return float(lib().or_ln2_lo())


def log_unit(u) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.float32)
    out = np.empty_like(u)
    lib().or_log_unit_array(_ptr(u, C.c_float), _ptr(out, C.c_float), u.size)
    return out


def sincos_turn24(k) -> tuple[np.ndarray, np.ndarray]:
    k = np.ascontiguousarray(k, dtype=np.uint32)
    s = np.empty(k.shape, dtype=np.float32)
    c = np.empty(k.shape, dtype=np.float32)
    lib().or_sincos_turn24_array(_ptr(k, C.c_uint32), _ptr(s, C.c_float), _ptr(c, C.c_float), k.size)
    return s, c


def round_bf16(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().or_round_bf16_array(_ptr(x, C.c_float), _ptr(out, C.c_float), x.size)
    return out


def normals(seed: int, t: int, i0: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.float32)
    lib().or_normals(seed, t, i0, count, _ptr(out, C.c_float))
    return out


def normals_at(seed: int, t: int, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float32)
    lib().or_normals_at(seed, t, _ptr(idx, C.c_int64), idx.size, _ptr(out, C.c_float))
    return out


# --------------------------------------------------------------------------
# Queuing schedule (Sec. 1 and eq. 2)
# --------------------------------------------------------------------------
def schedule(n: int, T: int, law: int = LAW_EXP, p0: float = 0.0, p1: float = 0.0,
             seed: int = 0, pull_mode: int = PULL_POST) -> tuple[np.ndarray, np.ndarray]:
    worker = np.zeros(T, dtype=np.int32)
    tau = np.zeros(T, dtype=np.int32)
    rc = lib().or_schedule(n, T, law, p0, p1, seed, pull_mode,
                           _ptr(worker, C.c_int32), _ptr(tau, C.c_int32))
    if rc != 0:
        raise RuntimeError(f"or_schedule failed: {rc}")
    return worker, tau


def worker_mean(law: int, p0: float, p1: float, seed: int, w: int) -> float:
    return float(lib().or_worker_mean(law, p0, p1, seed, w))


def job_time(law: int, p0: float, p1: float, mean_w: float, seed: int, w: int, k: int) -> float:
    return float(lib().or_job_time(law, p0, p1, mean_w, seed, w, k))


# --------------------------------------------------------------------------
# GEM state and commits (Alg. 1, eqs. 2, 3, 16-18, 22-23)
# --------------------------------------------------------------------------
@dataclass
class State:
    """theta[cnt], S[n, cnt], M[n, cnt], pull clocks pc[n], global clock t."""
    theta: np.ndarray
    S: np.ndarray
    M: np.ndarray
    pc: np.ndarray
    t: int = 0

    @staticmethod
    def initial(n: int, cnt: int, theta0=None) -> "State":
        """All workers pull theta_0 at clock 0 with m = 0 (Alg. 1, Worker start-up)."""
        th = np.zeros(cnt, dtype=np.float32) if theta0 is None else np.array(theta0, dtype=np.float32)
        return State(theta=th.copy(), S=np.tile(th, (n, 1)).astype(np.float32),
                     M=np.zeros((n, cnt), dtype=np.float32), pc=np.zeros(n, dtype=np.int64), t=0)

    def copy(self) -> "State":
        return State(self.theta.copy(), self.S.copy(), self.M.copy(), self.pc.copy(), self.t)


@dataclass
class Hyper:
    lr: float = 0.01
    sigma: float = 0.0
    momentum: float = 0.9
    eps: float = 1e-16
    kappa: float = 1.0
    pi_mode: int = PI_CLAMP0
    kappa_mode: int = KAPPA_LINEAR
    pull_mode: int = PULL_POST
    rule: int = RULE_GEM
    bf16: bool = False
    proxy: int = PROXY_LOCAL
    seed: int = 0

    def cfg(self, P: int, n: int) -> OracleConfig:
        return OracleConfig(P=P, n=n, lr=self.lr, sigma=self.sigma, momentum=self.momentum,
                            eps=self.eps, kappa=self.kappa, pi_mode=self.pi_mode,
                            kappa_mode=self.kappa_mode, pull_mode=self.pull_mode,
                            rule=self.rule, bf16=int(self.bf16), proxy=self.proxy,
                            seed=self.seed)


class OracleError(RuntimeError):
    def __init__(self, rc: int):
        super().__init__(f"oracle error {rc}")
        self.rc = rc


def run(hp: Hyper, P: int, st: State, idx, h, ts, worker, tau=None,
        diag: bool = False, trace: bool = False, pi_hist: bool = False, hist_segments=None):
    """Simulated run of len(worker) commits on the element subset ``idx``.

    The state ``st`` (theta, S, M restricted to ``idx``) is updated in place.
    Returns (diag array or None, trace array [T, cnt, 4] of (a, pi, d, m) or None),
    plus the per-commit histograms of the applied scale factor [T, PI_BINS]
    as a third item when ``pi_hist`` is set -- [T, nseg, PI_BINS] with one
    histogram per segment of the global index when ``hist_segments`` (the
    nseg + 1 offsets) is given.
    """
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    cnt = idx.size
    n = st.S.shape[0]
    h = np.ascontiguousarray(h, dtype=np.float32)
    ts = np.ascontiguousarray(ts, dtype=np.float32)
    worker = np.ascontiguousarray(worker, dtype=np.int32)
    T = worker.size
    tau_a = None if tau is None else np.ascontiguousarray(tau, dtype=np.int32)
    for a in (st.theta, st.S, st.M):
        assert a.dtype == np.float32 and a.flags.c_contiguous
    assert st.theta.size == cnt and st.S.shape == (n, cnt) and h.size == cnt and ts.size == cnt
    dg = np.zeros(T, dtype=COMMIT_DIAG_DTYPE) if diag else None
    tr = np.zeros((T, cnt, 4), dtype=np.float32) if trace else None
    seg = None if hist_segments is None else np.ascontiguousarray(hist_segments, dtype=np.int64)
    nseg = 0 if seg is None else seg.size - 1
    if pi_hist:
        shape = (T, PI_BINS) if seg is None else (T, nseg, PI_BINS)
        ph = np.zeros(shape, dtype=np.uint32)
    else:
        ph = None
    cfg = hp.cfg(P, n)
    rc = lib().or_run(C.byref(cfg), _ptr(idx, C.c_int64), cnt, _ptr(h, C.c_float),
                      _ptr(ts, C.c_float), _ptr(st.theta, C.c_float), _ptr(st.S, C.c_float),
                      _ptr(st.M, C.c_float), _ptr(st.pc, C.c_int64), st.t,
                      _ptr(worker, C.c_int32), _ptr(tau_a, C.c_int32), T,
                      dg.ctypes.data if dg is not None else None,
                      _ptr(tr, C.c_float), _ptr(ph, C.c_uint32), nseg, _ptr(seg, C.c_int64))
    if rc != 0:
        raise OracleError(rc)
    st.t += T
    return (dg, tr, ph) if pi_hist else (dg, tr)


def commit_given(hp: Hyper, st: State, worker, d, tau=None, diag: bool = False,
                 trace: bool = False):
    """Commits of caller-supplied updates d[K, P] (float32, or uint16 bf16 bit patterns).

    Returns (diag array or None, trace array [K, P, 4] of (a, pi, d, m) or None).
    """
    n, P = st.S.shape
    worker = np.ascontiguousarray(worker, dtype=np.int32)
    K = worker.size
    d = np.ascontiguousarray(d)
    assert d.shape == (K, P)
    tau_a = None if tau is None else np.ascontiguousarray(tau, dtype=np.int32)
    dg = np.zeros(K, dtype=COMMIT_DIAG_DTYPE) if diag else None
    tr = np.zeros((K, P, 4), dtype=np.float32) if trace else None
    cfg = hp.cfg(P, n)
    if d.dtype == np.float32:
        df, db = _ptr(d, C.c_float), None
    elif d.dtype == np.uint16:
        df, db = None, _ptr(d, C.c_uint16)
    else:
        raise TypeError("updates must be float32 or uint16 (bfloat16 bits)")
    rc = lib().or_commit_given(C.byref(cfg), P, _ptr(st.theta, C.c_float), _ptr(st.S, C.c_float),
                               _ptr(st.M, C.c_float), _ptr(st.pc, C.c_int64), st.t,
                               _ptr(worker, C.c_int32), _ptr(tau_a, C.c_int32), K, df, db,
                               dg.ctypes.data if dg is not None else None,
                               _ptr(tr, C.c_float), None)
    if rc != 0:
        raise OracleError(rc)
    st.t += K
    return dg, tr


def sumsq(x, lo: int = 0, hi: int | None = None) -> float:
    """Sum of squares of x[lo:hi] in binary64, in the order that defines the
    segment norms (see or_sumsq): every term the exact binary64 square; the
    adjacent-pairs tree within each aligned block of 2^18 indices (terms
    outside [lo, hi) are zero), then the block values added in increasing
    block order to a running total starting at zero."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    hi = x.size if hi is None else hi
    return float(lib().or_sumsq(_ptr(x, C.c_float), lo, hi))


def run_segments(hp: Hyper, st: State, seg_off, worker, tau=None, h=None, ts=None, d=None,
                 pi: bool = False, trace: bool = False, diag: bool = False):
    """Commits with one scale factor per segment [seg_off[k], seg_off[k+1]) of the
    parameter vector (norms over the segment in eq. 18; see or_run_segments).

    Updates are generated at the snapshots from (h, ts) as in ``run`` (on all P
    elements) when ``d`` is None, else given as d[T, P] (float32, or uint16
    bf16 bit patterns).  Returns (pi [T, nseg] or None, trace [T, P, 3] of
    (a, d, m) or None), plus the per-commit energy diagnostics as a third
    item when ``diag`` is set.
    """
    n, P = st.S.shape
    seg_off = np.ascontiguousarray(seg_off, dtype=np.int64)
    nseg = seg_off.size - 1
    worker = np.ascontiguousarray(worker, dtype=np.int32)
    T = worker.size
    tau_a = None if tau is None else np.ascontiguousarray(tau, dtype=np.int32)
    df = db = None
    if d is not None:
        d = np.ascontiguousarray(d)
        assert d.shape == (T, P)
        if d.dtype == np.float32:
            df = _ptr(d, C.c_float)
        elif d.dtype == np.uint16:
            db = _ptr(d, C.c_uint16)
        else:
            raise TypeError("updates must be float32 or uint16 (bfloat16 bits)")
    else:
        h = np.ascontiguousarray(h, dtype=np.float32)
        ts = np.ascontiguousarray(ts, dtype=np.float32)
        assert h.size == P and ts.size == P
    po = np.zeros((T, nseg), dtype=np.float32) if pi else None
    tr = np.zeros((T, P, 3), dtype=np.float32) if trace else None
    dg = np.zeros(T, dtype=COMMIT_DIAG_DTYPE) if diag else None
    cfg = hp.cfg(P, n)
    rc = lib().or_run_segments(C.byref(cfg), nseg, _ptr(seg_off, C.c_int64), _ptr(h, C.c_float),
                               _ptr(ts, C.c_float), _ptr(st.theta, C.c_float),
                               _ptr(st.S, C.c_float), _ptr(st.M, C.c_float),
                               _ptr(st.pc, C.c_int64), st.t, _ptr(worker, C.c_int32),
                               _ptr(tau_a, C.c_int32), T, df, db, _ptr(po, C.c_float),
                               _ptr(tr, C.c_float), dg.ctypes.data if dg is not None else None)
    if rc != 0:
        raise OracleError(rc)
    st.t += T
    return (po, tr, dg) if diag else (po, tr)


def loss(theta, h, ts) -> float:
    """1/2 sum h (theta - theta*)^2 in binary64 (the diagonal quadratic)."""
    theta = np.ascontiguousarray(theta, dtype=np.float32)
    h = np.ascontiguousarray(h, dtype=np.float32)
    ts = np.ascontiguousarray(ts, dtype=np.float32)
    return float(lib().or_loss(_ptr(theta, C.c_float), _ptr(h, C.c_float), _ptr(ts, C.c_float),
                               theta.size))


def pi_bin(pi) -> np.ndarray:
    """Histogram bin of each applied scale factor (see or_pi_bin)."""
    pi = np.ascontiguousarray(pi, dtype=np.float32)
    out = np.empty(pi.shape, dtype=np.int32)
    lib().or_pi_bin_array(_ptr(pi, C.c_float), _ptr(out, C.c_int32), pi.size)
    return out
