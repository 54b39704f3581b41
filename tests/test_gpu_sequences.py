"""GPU parity of longer call sequences and of the schedule extremes, against the
oracle: one worker (every commit of a pass repeats the previous worker), as
many workers as commits in a pass (no repeats), a seeded mix of the entry
points (simulated runs with varying K, given f32 and bf16 updates, worker
restarts, checkpoint and resume in a new handle), and checkpoints of the
per-segment scope, which carry the partition."""
import os
import tempfile

import numpy as np
import pytest

import oracle as O
from gpu_util import assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_08469_amd import gem
    return torch, gem


def _taus(worker, pc, t0):
    pc = pc.copy()
    tau = np.empty(len(worker), dtype=np.int32)
    for j, w in enumerate(worker):
        tau[j] = t0 + j - pc[w]
        pc[w] = t0 + j + 1
    return tau


def _check(g, st, tag):
    assert g.clock == st.t, tag
    assert np.array_equal(g.pull_clocks(), st.pc), f"{tag} pull clocks"
    assert_parity(f"{tag} theta", g.theta(), st.theta)
    assert_parity(f"{tag} S", g.S(), st.S)
    assert_parity(f"{tag} M", g.M(), st.M)


@pytest.mark.parametrize("K", [2, 32])
def test_single_worker(env, K):
    """n = 1: zero staleness, and every commit after the first in a pass takes
    the worker's rows from registers."""
    _, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, T = 5000, 200
    h, ts = make_problem(P, 1e-3, 1.0, 2)
    worker = np.zeros(T, dtype=np.int32)
    tau = np.zeros(T, dtype=np.int32)
    st = O.State.initial(1, P)
    with G.Gem(P, 1) as g:
        g.set_quadratic(h, ts, 0.02, 0.1, 4)
        g.sim_run(worker, tau, K)
        O.run(O.Hyper(lr=0.02, sigma=0.1, seed=4), P, st, np.arange(P), h, ts, worker, tau)
        _check(g, st, f"n=1 K={K}")
        assert g.stats().passes == -(-T // K)


@pytest.mark.parametrize("proxy", ["local", "global"])
def test_near_repeats_evict_far_held_rows(env, proxy):
    """Four workers held in the register slots for a far repeat, then workers
    that commit twice in a row: each near repeat takes the slot of the held
    chunk used furthest ahead, which goes back to memory and is read again
    through the ring.  No pass is cut, and the state equals the oracle."""
    _, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 4133, 8
    block = np.array([0, 1, 2, 3, 4, 4, 5, 5, 6, 6, 7, 7, 0, 1, 2, 3], np.int32)
    worker = np.tile(block, 8)
    tau = _taus(worker, np.zeros(n, np.int64), 0)
    h, ts = make_problem(P, 1e-3, 1.0, 9)
    hp = G.gem_hyperparams_default()
    hp.proxy_mode = G.GEM_PROXY_GLOBAL if proxy == "global" else G.GEM_PROXY_LOCAL
    st = O.State.initial(n, P)
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 6)
        g.sim_run(worker, tau, 32)
        O.run(O.Hyper(lr=0.01, sigma=0.1, seed=6, proxy=int(hp.proxy_mode)), P, st,
              np.arange(P), h, ts, worker, tau)
        _check(g, st, f"evictions ({proxy} proxy)")
        assert g.stats().passes == worker.size // 32


def test_no_repeats_in_a_pass(env):
    """n = 320 workers in a permuted round robin: every pass of 32 commits moves
    32 distinct workers' rows (no register slot is ever used)."""
    _, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 3001, 320
    rng = np.random.default_rng(7)
    worker = np.concatenate([rng.permutation(n) for _ in range(2)]).astype(np.int32)
    tau = _taus(worker, np.zeros(n, np.int64), 0)
    h, ts = make_problem(P, 1e-3, 1.0, 3)
    st = O.State.initial(n, P)
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 5)
        g.sim_run(worker, tau, 32)
        O.run(O.Hyper(lr=0.01, sigma=0.1, seed=5), P, st, np.arange(P), h, ts, worker, tau)
        _check(g, st, "no repeats")
        assert g.stats().passes == worker.size // 32


def _device_rows(torch, arr):
    K, P = arr.shape
    stride = (P + 7) // 8 * 8
    dt = torch.float32 if arr.dtype == np.float32 else torch.int16
    buf = torch.zeros((K, stride), dtype=dt, device="cuda")
    buf[:, :P] = torch.from_numpy(arr.view(np.int16) if arr.dtype == np.uint16 else arr).cuda()
    return buf, [buf[j].data_ptr() for j in range(K)]


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_mixed_call_sequence(env, seed):
    """A seeded sequence of the entry points on one master, and the same
    sequence on the oracle."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    rng = np.random.default_rng(seed)
    P, n = 2000 + seed * 37, 5
    lr, sigma, nseed = 0.01, 0.1, 100 + seed
    h, ts = make_problem(P, 1e-3, 1.0, seed)
    ohp = O.Hyper(lr=lr, sigma=sigma, seed=nseed)
    st = O.State.initial(n, P)
    g = G.Gem(P, n)
    g.set_quadratic(h, ts, lr, sigma, nseed)
    with tempfile.TemporaryDirectory() as tmp:
        for step in range(14):
            op = rng.choice(["sim", "sim", "given_f32", "given_bf16", "reset", "checkpoint"])
            print(f"[sequence seed={seed}] step {step}: {op}", flush=True)
            if op == "sim":
                T, K = int(rng.integers(1, 90)), int(rng.integers(1, 33))
                worker = rng.integers(0, n, size=T).astype(np.int32)
                tau = _taus(worker, st.pc, st.t)
                g.sim_run(worker, tau, K)
                O.run(ohp, P, st, np.arange(P), h, ts, worker, tau)
            elif op in ("given_f32", "given_bf16"):
                K = int(rng.integers(1, 40))
                worker = rng.integers(0, n, size=K).astype(np.int32)
                d = (rng.standard_normal((K, P)) * 0.01).astype(np.float32)
                dtype = G.GEM_F32
                if op == "given_bf16":
                    d = (O.round_bf16(d).view(np.uint32) >> 16).astype(np.uint16)
                    dtype = G.GEM_BF16
                buf, ptrs = _device_rows(torch, d)
                g.commit_batch(ptrs, dtype, worker, None)
                torch.cuda.synchronize()
                O.commit_given(ohp, st, worker, d)
            elif op == "reset":
                w = int(rng.integers(0, n))
                assert G.gem_reset_worker(g.h, w) == G.GEM_OK
                st.S[w] = st.theta
                st.M[w] = 0
                st.pc[w] = st.t
            else:
                path = os.path.join(tmp, f"ck{step}.bin")
                assert G.gem_save(g.h, path) == G.GEM_OK
                g.close()
                g = G.Gem(P, n)
                assert G.gem_load(g.h, path) == G.GEM_OK
        _check(g, st, f"sequence seed={seed}")
    g.close()


def test_segment_checkpoint_carries_the_partition(env):
    """Save under the per-segment scope with a partition, load into a fresh
    handle (no partition set), continue: equal to the straight run and to the
    oracle, bit for bit."""
    _, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 6000, 4, 60
    h, ts = make_problem(P, 1e-3, 1.0, 8)
    seg = np.array([0, 100, 1500, 1501, 4096, P], dtype=np.int64)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=8)
    hp = G.gem_hyperparams_default()
    hp.pi_scope = G.GEM_PI_SEGMENT
    with G.Gem(P, n, hp) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 9)
        g.set_segments(seg)
        g.sim_run(worker, tau, 8)
        straight = (g.theta(), g.S(), g.M())
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, "seg.bin")
        with G.Gem(P, n, hp) as g:
            g.set_quadratic(h, ts, 0.01, 0.1, 9)
            g.set_segments(seg)
            g.sim_run(worker[:25], tau[:25], 8)
            assert G.gem_save(g.h, path) == G.GEM_OK
        with G.Gem(P, n, hp) as g:
            assert G.gem_load(g.h, path) == G.GEM_OK
            g.sim_run(worker[25:], tau[25:], 8)
            resumed = (g.theta(), g.S(), g.M())
        # a truncated file is refused and leaves the handle as it was
        with open(path, "rb") as f:
            blob = f.read()
        with open(path, "wb") as f:
            f.write(blob[:-8])
        with G.Gem(P, n, hp) as g:
            assert G.gem_load(g.h, path) == G.GEM_EIO
            assert g.clock == 0 and np.all(g.theta() == 0)
    for a, b, name in zip(straight, resumed, ("theta", "S", "M")):
        assert_parity(f"segment resume {name}", b, a)
    st = O.State.initial(n, P)
    O.run_segments(O.Hyper(lr=0.01, sigma=0.1, seed=9), st, seg, worker, tau, h=h, ts=ts)
    assert_parity("segment resume vs oracle", resumed[0], st.theta)
