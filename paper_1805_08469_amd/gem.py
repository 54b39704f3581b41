"""Python binding of the libgem C ABI (``include/gem.h``).

Argument marshalling only: every step of the commit pipeline runs in the HIP
library ``libgem.so`` built in this package directory.  Device buffers are
passed as integer addresses (``tensor.data_ptr()``) and streams as
``torch.cuda.current_stream().cuda_stream``; nothing here computes on data.
Importing this module fails loudly if the library has not been built.

The wrappers of the commit-path calls (gem_commit, gem_commit_batch,
gem_generate, gem_sim_run, gem_reset_worker, gem_save, gem_load,
gem_copy_f32) return the library's GEM_* code as is; the others raise
GemError on a failed call.  The owning ``Gem`` class raises everywhere.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# The in-tree build; LIBGEM_PATH may name another build of the same sources.
LIB_PATH = os.environ.get("LIBGEM_PATH") or os.path.join(_HERE, "libgem.so")

GEM_OK, GEM_EINVAL, GEM_ENOMEM, GEM_EWORKER, GEM_ESTALE = 0, -1, -2, -3, -4
GEM_EDTYPE, GEM_EHIP, GEM_ESTATE, GEM_EIO, GEM_EALIGN = -5, -6, -7, -8, -9
GEM_ESCRATCH = -10
GEM_SCRATCH_BYTES = 4 << 20
GEM_F32, GEM_BF16 = 0, 1
GEM_PI_CLAMP0, GEM_PI_LITERAL = 0, 1
GEM_KAPPA_LINEAR, GEM_KAPPA_SQRT = 0, 1
GEM_PULL_POST_COMMIT, GEM_PULL_PRE_COMMIT = 0, 1
GEM_RULE_GEM, GEM_RULE_DOWNPOUR, GEM_RULE_ADAPTIVE = 0, 1, 2
GEM_PROXY_LOCAL, GEM_PROXY_GLOBAL = 0, 1
GEM_PI_ELEMENT, GEM_PI_SEGMENT = 0, 1
GEM_CACHE_AUTO, GEM_CACHE_KEEP, GEM_CACHE_STREAM = 0, 1, 2
GEM_LAW_EXP, GEM_LAW_EXP_UNIFORM_MEAN, GEM_LAW_EXP_LOGNORMAL_MEAN, GEM_LAW_PARETO = 0, 1, 2, 3
GEM_SNAPSHOT, GEM_MOMENT = 0, 1
GEM_K_MAX = 32
GEM_P_MAX = 1 << 31
GEM_PI_BINS = 643

# Every symbol include/gem.h declares.
EXPORTED = (
    "gem_strerror", "gem_last_error", "gem_hyperparams_default", "gem_create", "gem_destroy", "gem_set_theta",
    "gem_set_quadratic", "gem_commit", "gem_commit_batch", "gem_generate", "gem_schedule_make",
    "gem_sim_run", "gem_read_theta", "gem_read_state", "gem_gather", "gem_clock",
    "gem_pull_clocks", "gem_reset_worker", "gem_diag_enable", "gem_diag_reset", "gem_diag",
    "gem_stats", "gem_stats_reset", "gem_save", "gem_load", "gem_sync", "gem_copy_f32",
    "gem_pi_hist_start", "gem_pi_hist_start_segments", "gem_pi_hist_read", "gem_set_segments",
    "gem_set_cache_policy", "gem_dims", "gem_gather_static",
)


class gem_hyperparams(C.Structure):
    _fields_ = [("momentum", C.c_float), ("eps", C.c_float), ("kappa", C.c_float),
                ("pi_mode", C.c_int32), ("kappa_mode", C.c_int32), ("pull_mode", C.c_int32),
                ("rule", C.c_int32), ("proxy_mode", C.c_int32), ("pi_scope", C.c_int32)]


class gem_sim_params(C.Structure):
    _fields_ = [("lr", C.c_float), ("sigma", C.c_float), ("seed", C.c_uint64),
                ("update_dtype", C.c_int32), ("reserved", C.c_int32)]


class gem_schedule_law(C.Structure):
    _fields_ = [("law", C.c_int32), ("reserved", C.c_int32), ("p0", C.c_double),
                ("p1", C.c_double)]


class gem_diag_t(C.Structure):
    _fields_ = [("loss", C.c_double), ("sum_ek", C.c_double), ("sum_proxy", C.c_double),
                ("n_clamped", C.c_int64), ("n_elem_commits", C.c_int64), ("n_commits", C.c_int64)]


class gem_stats_t(C.Structure):
    _fields_ = [("commits", C.c_int64), ("passes", C.c_int64), ("alg_bytes", C.c_double)]


class GemError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        detail = f" [{gem_last_error()}]" if code == GEM_EHIP else ""
        super().__init__(f"{what}: {gem_strerror(code)} ({code}){detail}")
        self.code = code


def _load():
    # One HIP runtime per process: torch ships its own libamdhip64 under the
    # same soname as the system one.  Loading torch first makes libgem bind to
    # the runtime that owns torch's allocations and streams; loading libgem
    # first would bring in a second runtime beside torch's.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libgem HIP library not built: {LIB_PATH} is missing "
                          "(run __graft_entry__.build() or paper_1805_08469_amd/build.py)")
    L = C.CDLL(LIB_PATH)
    vp, i32p, i64p, f32p = C.c_void_p, C.POINTER(C.c_int32), C.POINTER(C.c_int64), C.c_void_p
    sig = {
        "gem_strerror": (C.c_char_p, [C.c_int]),
        "gem_last_error": (C.c_char_p, []),
        "gem_hyperparams_default": (C.c_int, [C.POINTER(gem_hyperparams)]),
        "gem_create": (C.c_int, [C.c_int64, C.c_int32, C.POINTER(gem_hyperparams), vp,
                                 C.POINTER(vp)]),
        "gem_destroy": (C.c_int, [vp]),
        "gem_set_theta": (C.c_int, [vp, f32p, C.c_int32]),
        "gem_set_quadratic": (C.c_int, [vp, f32p, f32p, C.POINTER(gem_sim_params)]),
        "gem_commit": (C.c_int, [vp, vp, C.c_int32]),
        "gem_commit_batch": (C.c_int, [vp, C.c_int32, C.POINTER(vp), C.c_int32, i32p, i32p]),
        "gem_generate": (C.c_int, [vp, C.c_int32, vp, C.c_int32]),
        "gem_schedule_make": (C.c_int, [C.c_int32, C.c_int64, C.POINTER(gem_schedule_law),
                                        C.c_uint64, C.c_int32, i32p, i32p]),
        "gem_sim_run": (C.c_int, [vp, i32p, i32p, C.c_int64, C.c_int32]),
        "gem_read_theta": (C.c_int, [vp, vp, C.c_int32]),
        "gem_read_state": (C.c_int, [vp, C.c_int32, C.c_int32, vp, C.c_int32]),
        "gem_gather": (C.c_int, [vp, i64p, C.c_int64, vp, vp, vp]),
        "gem_gather_static": (C.c_int, [vp, i64p, C.c_int64, vp, vp, vp]),
        "gem_clock": (C.c_int, [vp, i64p]),
        "gem_dims": (C.c_int, [vp, i64p, i32p]),
        "gem_pull_clocks": (C.c_int, [vp, i64p]),
        "gem_reset_worker": (C.c_int, [vp, C.c_int32]),
        "gem_diag_enable": (C.c_int, [vp, C.c_int32]),
        "gem_diag_reset": (C.c_int, [vp]),
        "gem_diag": (C.c_int, [vp, C.POINTER(gem_diag_t)]),
        "gem_stats": (C.c_int, [vp, C.POINTER(gem_stats_t)]),
        "gem_stats_reset": (C.c_int, [vp]),
        "gem_save": (C.c_int, [vp, C.c_char_p]),
        "gem_load": (C.c_int, [vp, C.c_char_p]),
        "gem_sync": (C.c_int, [vp]),
        "gem_set_cache_policy": (C.c_int, [vp, C.c_int32]),
        "gem_copy_f32": (C.c_int, [vp, vp, C.c_int64, vp]),
        "gem_pi_hist_start": (C.c_int, [vp, C.c_int64]),
        "gem_pi_hist_start_segments": (C.c_int, [vp, C.c_int64]),
        "gem_set_segments": (C.c_int, [vp, i64p, C.c_int32]),
        "gem_pi_hist_read": (C.c_int, [vp, C.POINTER(C.c_uint32), C.c_int64, i64p]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


_L = _load()


def lib():
    return _L


def _check(rc: int, what: str):
    if rc != GEM_OK:
        raise GemError(rc, what)


def _i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _p(a, ct):
    return None if a is None else a.ctypes.data_as(C.POINTER(ct))


# ---- the C ABI, name for name -------------------------------------------------
def gem_strerror(code: int) -> str:
    return _L.gem_strerror(code).decode()


def gem_last_error() -> str:
    return _L.gem_last_error().decode()


def gem_hyperparams_default() -> gem_hyperparams:
    hp = gem_hyperparams()
    _check(_L.gem_hyperparams_default(C.byref(hp)), "gem_hyperparams_default")
    return hp


def gem_create(P: int, n: int, hp: gem_hyperparams | None = None, stream: int | None = None) -> int:
    out = C.c_void_p()
    _check(_L.gem_create(P, n, C.byref(hp) if hp is not None else None, stream or None,
                         C.byref(out)), "gem_create")
    return out.value


def gem_destroy(g: int) -> None:
    _check(_L.gem_destroy(g), "gem_destroy")


def gem_dims(g: int) -> tuple[int, int]:
    """(P, n) of the handle."""
    P, n = C.c_int64(), C.c_int32()
    _check(_L.gem_dims(g, C.byref(P), C.byref(n)), "gem_dims")
    return P.value, n.value


def _host_f32(a, size: int, what: str) -> np.ndarray:
    """A contiguous binary32 copy of a host array that must hold `size`
    elements: the library reads or writes exactly that many."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if a.size != size:
        raise ValueError(f"{what}: {a.size} elements, the handle needs {size}")
    return a


def _same_size(g: int, P: int, what: str) -> None:
    if P != gem_dims(g)[0]:
        raise ValueError(f"{what}: P = {P}, the handle has P = {gem_dims(g)[0]}")


def gem_set_theta(g: int, theta0, in_is_device: bool = False) -> None:
    if in_is_device:
        _check(_L.gem_set_theta(g, theta0, 1), "gem_set_theta")
    else:
        a = _host_f32(theta0, gem_dims(g)[0], "gem_set_theta")
        _check(_L.gem_set_theta(g, a.ctypes.data, 0), "gem_set_theta")


def gem_set_quadratic(g: int, h, theta_star, sp: gem_sim_params) -> None:
    P = gem_dims(g)[0]
    h = _host_f32(h, P, "gem_set_quadratic (h)")
    ts = _host_f32(theta_star, P, "gem_set_quadratic (theta_star)")
    _check(_L.gem_set_quadratic(g, h.ctypes.data, ts.ctypes.data, C.byref(sp)), "gem_set_quadratic")


def gem_commit(g: int, dtheta_dev: int, worker_id: int) -> int:
    return _L.gem_commit(g, dtheta_dev, worker_id)


def gem_commit_batch(g: int, dthetas_dev, dtype: int, worker_ids, staleness=None) -> int:
    K = len(dthetas_dev)
    ptrs = (C.c_void_p * max(K, 1))(*[int(p) for p in dthetas_dev])
    w = _i32(worker_ids)
    s = _i32(staleness)
    return _L.gem_commit_batch(g, K, ptrs, dtype, _p(w, C.c_int32), _p(s, C.c_int32))


def gem_generate(g: int, worker_id: int, out_dev: int, dtype: int) -> int:
    return _L.gem_generate(g, worker_id, out_dev, dtype)


def gem_schedule_make(n: int, T: int, law: int, p0: float = 0.0, p1: float = 0.0, seed: int = 0,
                      pull_mode: int = GEM_PULL_POST_COMMIT):
    worker = np.zeros(T, dtype=np.int32)
    tau = np.zeros(T, dtype=np.int32)
    L = gem_schedule_law(law=law, p0=p0, p1=p1)
    _check(_L.gem_schedule_make(n, T, C.byref(L), seed, pull_mode, _p(worker, C.c_int32),
                                _p(tau, C.c_int32)), "gem_schedule_make")
    return worker, tau


def gem_sim_run(g: int, worker, tau, K: int) -> int:
    w = _i32(worker)
    t = _i32(tau)
    return _L.gem_sim_run(g, _p(w, C.c_int32), _p(t, C.c_int32), w.size, K)


def gem_read_theta(g: int, P: int) -> np.ndarray:
    _same_size(g, P, "gem_read_theta")
    out = np.empty(P, dtype=np.float32)
    _check(_L.gem_read_theta(g, out.ctypes.data, 0), "gem_read_theta")
    return out


def gem_read_state(g: int, w: int, which: int, P: int) -> np.ndarray:
    _same_size(g, P, "gem_read_state")
    out = np.empty(P, dtype=np.float32)
    _check(_L.gem_read_state(g, w, which, out.ctypes.data, 0), "gem_read_state")
    return out


def gem_gather(g: int, idx, n: int):
    if n != gem_dims(g)[1]:
        raise ValueError(f"gem_gather: n = {n}, the handle has n = {gem_dims(g)[1]}")
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    th = np.empty(idx.size, dtype=np.float32)
    S = np.empty((n, idx.size), dtype=np.float32)
    M = np.empty((n, idx.size), dtype=np.float32)
    _check(_L.gem_gather(g, _p(idx, C.c_int64), idx.size, th.ctypes.data, S.ctypes.data,
                         M.ctypes.data), "gem_gather")
    return th, S, M


def gem_gather_static(g: int, idx, n: int):
    """gem_gather through the library's fixed device scratch (no allocation
    in the library); raises GemError(GEM_ESCRATCH) for a request that does
    not fit it."""
    if n != gem_dims(g)[1]:
        raise ValueError(f"gem_gather_static: n = {n}, the handle has n = {gem_dims(g)[1]}")
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    th = np.empty(idx.size, dtype=np.float32)
    S = np.empty((n, idx.size), dtype=np.float32)
    M = np.empty((n, idx.size), dtype=np.float32)
    _check(_L.gem_gather_static(g, _p(idx, C.c_int64), idx.size, th.ctypes.data, S.ctypes.data,
                                M.ctypes.data), "gem_gather_static")
    return th, S, M


def gem_clock(g: int) -> int:
    t = C.c_int64()
    _check(_L.gem_clock(g, C.byref(t)), "gem_clock")
    return t.value


def gem_pull_clocks(g: int, n: int) -> np.ndarray:
    if n != gem_dims(g)[1]:
        raise ValueError(f"gem_pull_clocks: n = {n}, the handle has n = {gem_dims(g)[1]}")
    out = np.zeros(n, dtype=np.int64)
    _check(_L.gem_pull_clocks(g, _p(out, C.c_int64)), "gem_pull_clocks")
    return out


def gem_reset_worker(g: int, w: int) -> int:
    return _L.gem_reset_worker(g, w)


def gem_diag_enable(g: int, on: bool) -> None:
    _check(_L.gem_diag_enable(g, int(on)), "gem_diag_enable")


def gem_diag_reset(g: int) -> None:
    _check(_L.gem_diag_reset(g), "gem_diag_reset")


def gem_diag(g: int) -> gem_diag_t:
    d = gem_diag_t()
    _check(_L.gem_diag(g, C.byref(d)), "gem_diag")
    return d


def gem_stats(g: int) -> gem_stats_t:
    s = gem_stats_t()
    _check(_L.gem_stats(g, C.byref(s)), "gem_stats")
    return s


def gem_stats_reset(g: int) -> None:
    _check(_L.gem_stats_reset(g), "gem_stats_reset")


def gem_save(g: int, path: str) -> int:
    return _L.gem_save(g, path.encode())


def gem_load(g: int, path: str) -> int:
    return _L.gem_load(g, path.encode())


def gem_set_segments(g: int, offsets) -> None:
    """Segments [offsets[k], offsets[k+1]) for the segment-norm scale factors."""
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    _check(_L.gem_set_segments(g, _p(off, C.c_int64), off.size - 1), "gem_set_segments")


def gem_pi_hist_start(g: int, capacity: int) -> None:
    _check(_L.gem_pi_hist_start(g, capacity), "gem_pi_hist_start")


def gem_pi_hist_start_segments(g: int, capacity: int) -> None:
    _check(_L.gem_pi_hist_start_segments(g, capacity), "gem_pi_hist_start_segments")


def gem_pi_hist_read(g: int, max_commits: int, segments: int = 0) -> np.ndarray:
    """Recorded histograms: [commits, GEM_PI_BINS], or [commits, segments,
    GEM_PI_BINS] for a per-segment recording of that many segments."""
    rows = max(segments, 1)
    out = np.zeros((max(max_commits, 0), rows, GEM_PI_BINS), dtype=np.uint32)
    n = C.c_int64()
    _check(_L.gem_pi_hist_read(g, _p(out, C.c_uint32), max_commits, C.byref(n)), "gem_pi_hist_read")
    out = out[:min(n.value, max_commits)]
    return out if segments else out[:, 0]


def gem_sync(g: int) -> None:
    _check(_L.gem_sync(g), "gem_sync")


def gem_set_cache_policy(g: int, policy: int) -> None:
    _check(_L.gem_set_cache_policy(g, policy), "gem_set_cache_policy")


def gem_copy_f32(src_dev: int, dst_dev: int, count: int, stream: int | None = None) -> int:
    return _L.gem_copy_f32(src_dev, dst_dev, count, stream or None)


# ---- a small owning wrapper used by the tests and the benchmark ----------------
class Gem:
    """Owns one libgem handle.  ``stream`` is a hipStream_t address or None."""

    def __init__(self, P: int, n: int, hp: gem_hyperparams | None = None, stream: int | None = None):
        self.P, self.n = P, n
        self.h = gem_create(P, n, hp, stream)

    def close(self):
        if self.h:
            gem_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_quadratic(self, h, ts, lr, sigma, seed, bf16=False):
        sp = gem_sim_params(lr=lr, sigma=sigma, seed=seed,
                            update_dtype=GEM_BF16 if bf16 else GEM_F32)
        gem_set_quadratic(self.h, h, ts, sp)

    def set_segments(self, offsets):
        gem_set_segments(self.h, offsets)

    def set_cache_policy(self, policy: int):
        gem_set_cache_policy(self.h, policy)

    def sim_run(self, worker, tau, K):
        _check(gem_sim_run(self.h, worker, tau, K), "gem_sim_run")

    def commit(self, dtheta_dev: int, w: int):
        _check(gem_commit(self.h, dtheta_dev, w), "gem_commit")

    def commit_batch(self, ptrs, dtype, workers, staleness=None):
        _check(gem_commit_batch(self.h, ptrs, dtype, workers, staleness), "gem_commit_batch")

    def theta(self):
        return gem_read_theta(self.h, self.P)

    def state(self, w, which):
        return gem_read_state(self.h, w, which, self.P)

    def S(self):
        return np.stack([self.state(w, GEM_SNAPSHOT) for w in range(self.n)])

    def M(self):
        return np.stack([self.state(w, GEM_MOMENT) for w in range(self.n)])

    def gather(self, idx):
        return gem_gather(self.h, idx, self.n)

    @property
    def clock(self):
        return gem_clock(self.h)

    def pull_clocks(self):
        return gem_pull_clocks(self.h, self.n)

    def stats(self):
        return gem_stats(self.h)

    def sync(self):
        gem_sync(self.h)
