"""GPU tests of the commit entry points that take caller updates
(gem_commit, gem_commit_batch in fp32 and bf16), of the generator-then-commit
pipeline, and of the error paths: a rejected call must leave the state and
the clock untouched."""
import ctypes as C

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


def _updates(rng, K, P, scale=1e-2):
    return (rng.standard_normal((K, P)) * scale).astype(np.float32)


def _device_rows(torch, a):
    """Upload a [K, P] array with its row stride padded to 8 elements, so each
    row starts 16-byte aligned (fp32) / 8-byte aligned (bf16) as gem.h requires."""
    K, P = a.shape
    stride = -(-P // 8) * 8
    pad = np.zeros((K, stride), dtype=a.dtype)
    pad[:, :P] = a
    return torch.from_numpy(pad).cuda()


def _to_bf16_bits(x):
    b = O.round_bf16(x).view(np.uint32)
    return (b >> 16).astype(np.uint16)


@pytest.mark.parametrize("P", [7, 4096, 100_003])
def test_commit_one_by_one(env, P):
    torch, G = env
    n, T = 4, 40
    rng = np.random.default_rng(P)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=1)
    d = _updates(rng, T, P)
    dev = _device_rows(torch, d)
    with G.Gem(P, n) as g:
        for j in range(T):
            g.commit(dev[j].data_ptr(), int(worker[j]))
        theta, S, M = g.theta(), g.S(), g.M()
    st = O.State.initial(n, P)
    O.commit_given(O.Hyper(), st, worker, d, tau=tau)
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)


@pytest.mark.parametrize("policy", ["keep", "stream"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [1, 5, 32, 45])
def test_commit_batch(env, dtype, K, policy):
    torch, G = env
    P, n = 10_007, 3                      # n = 3: workers repeat inside every batch
    rng = np.random.default_rng(K)
    worker, tau = G.gem_schedule_make(n, 3 * K, G.GEM_LAW_EXP, seed=K)
    d = _updates(rng, 3 * K, P)
    if dtype == "bf16":
        bits = _to_bf16_bits(d)
        dev = _device_rows(torch, bits.view(np.int16))
        code = G.GEM_BF16
        ref_upd = bits
    else:
        dev = _device_rows(torch, d)
        code = G.GEM_F32
        ref_upd = d
    with G.Gem(P, n) as g:
        g.set_cache_policy(G.GEM_CACHE_STREAM if policy == "stream" else G.GEM_CACHE_KEEP)
        for b in range(3):
            rows = range(b * K, (b + 1) * K)
            g.commit_batch([dev[j].data_ptr() for j in rows], code, worker[b * K:(b + 1) * K],
                           tau[b * K:(b + 1) * K])
        theta, S, M, clock = g.theta(), g.S(), g.M(), g.clock
    st = O.State.initial(n, P)
    O.commit_given(O.Hyper(), st, worker, ref_upd, tau=tau)
    assert clock == 3 * K
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)


EXTREMES = np.array([0.0, -0.0, 1e-45, -1e-40, 1e-30, -1e-20, 1e-10, 1.0, -1e10, 1e20, -1e30,
                     3e38, np.inf, -np.inf, np.nan], dtype=np.float32)


@pytest.mark.parametrize("proxy", [0, 1])
def test_extreme_update_magnitudes(env, proxy):
    """Caller updates of every magnitude -- zeros of both signs, subnormals,
    values near the ends of the exponent range, infinities and NaN, mixed with
    ordinary ones -- through the default rule's variants (per-worker and
    shared moment): quotients outside the range of the core division take the
    general one, element by element, and the state stays equal to the
    oracle's (NaN compares equal to NaN)."""
    torch, G = env
    P, n, T, K = 8192 + 77, 3, 24, 8
    rng = np.random.default_rng(100 + proxy)
    d = (rng.standard_normal((T, P)) * 0.01).astype(np.float32)
    pick = rng.random((T, P)) < 0.03
    d[pick] = rng.choice(EXTREMES, size=int(pick.sum()))
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=7)
    dev = _device_rows(torch, d)
    hp = G.gem_hyperparams_default()
    hp.proxy_mode = G.GEM_PROXY_GLOBAL if proxy else G.GEM_PROXY_LOCAL
    with G.Gem(P, n, hp) as g:
        for b in range(0, T, K):
            g.commit_batch([dev[j].data_ptr() for j in range(b, b + K)], G.GEM_F32,
                           worker[b:b + K], tau[b:b + K])
        theta, S, M = g.theta(), g.S(), g.M()
    st = O.State.initial(n, P)
    O.commit_given(O.Hyper(proxy=proxy), st, worker, d, tau=tau)
    assert np.isnan(st.theta).any() and np.isinf(st.theta).any()   # the cases are reached
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)


@pytest.mark.parametrize("K", [1, 32])
def test_commit_batch_global_proxy(env, K):
    """Caller updates committed with the shared moment (Sec. 6): row 0 of M."""
    torch, G = env
    P, n = 5003, 4
    rng = np.random.default_rng(K + 100)
    worker, tau = G.gem_schedule_make(n, 2 * K, G.GEM_LAW_EXP, seed=K + 1)
    d = _updates(rng, 2 * K, P)
    dev = _device_rows(torch, d)
    hp = G.gem_hyperparams_default()
    hp.proxy_mode = G.GEM_PROXY_GLOBAL
    with G.Gem(P, n, hp) as g:
        for b in range(2):
            g.commit_batch([dev[j].data_ptr() for j in range(b * K, (b + 1) * K)], G.GEM_F32,
                           worker[b * K:(b + 1) * K], tau[b * K:(b + 1) * K])
        theta, S, M = g.theta(), g.S(), g.M()
    st = O.State.initial(n, P)
    O.commit_given(O.Hyper(proxy=O.PROXY_GLOBAL), st, worker, d, tau=tau)
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)
    assert np.all(M[1:] == 0)


@pytest.mark.parametrize("bf16", [False, True])
def test_generate_then_commit_equals_fused_run(env, bf16):
    """The unfused pipeline (generator kernel writes dtheta, commit kernel reads
    it) equals the fused simulated run."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 6000, 5, 64
    h, ts = make_problem(P, 1e-4, 1.0, 4)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=4)
    code = G.GEM_BF16 if bf16 else G.GEM_F32
    buf = torch.empty(P, dtype=torch.int16 if bf16 else torch.float32, device="cuda")
    with G.Gem(P, n) as a, G.Gem(P, n) as b:
        a.set_quadratic(h, ts, 0.01, 0.02, 8, bf16=bf16)
        b.set_quadratic(h, ts, 0.01, 0.02, 8, bf16=bf16)
        a.sim_run(worker, tau, 16)
        for j in range(T):
            assert G.gem_generate(b.h, int(worker[j]), buf.data_ptr(), code) == G.GEM_OK
            b.commit_batch([buf.data_ptr()], code, worker[j:j + 1], tau[j:j + 1])
        for x, y in ((a.theta(), b.theta()), (a.S(), b.S()), (a.M(), b.M())):
            assert np.array_equal(x, y)


def test_rejected_calls_change_nothing(env):
    torch, G = env
    P, n = 1000, 3
    d = torch.ones(P + 8, dtype=torch.float32, device="cuda")
    with G.Gem(P, n) as g:
        g.commit(d.data_ptr(), 0)
        before = (g.theta(), g.S(), g.M(), g.clock, g.pull_clocks())
        assert G.gem_commit(g.h, d.data_ptr(), 3) == G.GEM_EWORKER
        assert G.gem_commit(g.h, d.data_ptr(), -1) == G.GEM_EWORKER
        assert G.gem_commit(g.h, d.data_ptr() + 4, 0) == G.GEM_EALIGN
        assert G.gem_commit(g.h, 0, 0) == G.GEM_EINVAL
        # worker 1's staleness at t=1 is 1; a batch with a wrong value in its
        # second entry must not apply its first entry either
        assert G.gem_commit_batch(g.h, [d.data_ptr()] * 2, G.GEM_F32, [1, 2], [1, 0]) == G.GEM_ESTALE
        assert G.gem_commit_batch(g.h, [d.data_ptr()], 7, [1], None) == G.GEM_EDTYPE
        assert G.gem_commit_batch(g.h, [d.data_ptr() + 2], G.GEM_BF16, [1], None) == G.GEM_EALIGN
        assert G.gem_sim_run(g.h, [0], [0], 1) == G.GEM_ESTATE        # no problem set
        assert G.gem_generate(g.h, 0, d.data_ptr(), G.GEM_F32) == G.GEM_ESTATE
        g.set_quadratic(np.ones(P, np.float32), np.zeros(P, np.float32), 0.01, 0.0, 0)
        assert G.gem_sim_run(g.h, [0], [0], 0) == G.GEM_EINVAL          # K = 0
        assert G.gem_sim_run(g.h, [0], [0], 33) == G.GEM_EINVAL         # K > GEM_K_MAX
        assert G.gem_sim_run(g.h, [0, 9], None, 4) == G.GEM_EWORKER
        assert G.gem_reset_worker(g.h, 5) == G.GEM_EWORKER
        # sizes whose byte counts would wrap: refused before any allocation
        L = G.lib()
        assert L.gem_pi_hist_start(g.h, 2**62) == G.GEM_EINVAL
        assert L.gem_pi_hist_start_segments(g.h, 2**62) == G.GEM_EINVAL
        idx = np.zeros(4, np.int64)
        assert L.gem_gather(g.h, idx.ctypes.data_as(C.POINTER(C.c_int64)), G.GEM_P_MAX + 1,
                            None, None, None) == G.GEM_EINVAL
        # host buffers of the wrong length are refused by the binding before
        # the library could read or write past their ends
        assert G.gem_dims(g.h) == (P, n)
        with pytest.raises(ValueError):
            G.gem_set_quadratic(g.h, np.ones(P - 1, np.float32), np.zeros(P, np.float32),
                                G.gem_sim_params(lr=0.01))
        with pytest.raises(ValueError):
            G.gem_set_theta(g.h, np.zeros(P - 3, np.float32))
        with pytest.raises(ValueError):
            G.gem_read_theta(g.h, P + 1)
        with pytest.raises(ValueError):
            G.gem_read_state(g.h, 0, G.GEM_SNAPSHOT, P - 1)
        with pytest.raises(ValueError):
            G.gem_gather(g.h, [0, 1], n + 1)
        with pytest.raises(ValueError):
            G.gem_pull_clocks(g.h, n - 1)
        after = (g.theta(), g.S(), g.M(), g.clock, g.pull_clocks())
    for x, y in zip(before, after):
        assert np.array_equal(x, y)


def test_hyperparameters_out_of_range_are_refused(env):
    """eps <= 0 would let an update of exactly zero divide zero by zero in
    pi's denominator (Alg. 1) and turn theta into NaN; kappa scales a positive
    proxy energy.  Both are refused at create and in a checkpoint header."""
    torch, G = env
    for field, value in (("eps", 0.0), ("eps", -1e-16), ("kappa", 0.0), ("kappa", -1.0)):
        hp = G.gem_hyperparams_default()
        setattr(hp, field, value)
        with pytest.raises(G.GemError) as e:
            G.Gem(64, 2, hp)
        assert e.value.code == G.GEM_EINVAL
    # the smallest positive eps still keeps an update of exactly zero from moving theta
    hp = G.gem_hyperparams_default()
    hp.eps = 1e-45
    d = torch.zeros(64, dtype=torch.float32, device="cuda")
    with G.Gem(64, 2, hp) as g:
        g.commit(d.data_ptr(), 1)
        g.commit(d.data_ptr(), 0)
        assert np.all(g.theta() == 0) and np.all(np.isfinite(g.M()))


def test_load_refuses_a_header_with_eps_zero(env, tmp_path):
    torch, G = env
    path = str(tmp_path / "ck.bin")
    with G.Gem(64, 2) as g:
        assert G.gem_save(g.h, path) == G.GEM_OK
        raw = bytearray(open(path, "rb").read())
        # header: magic[8], P int64, n int32, have_problem int32, t int64, then
        # the hyper-parameters (momentum, eps, kappa as binary32 first)
        eps_at = 8 + 8 + 4 + 4 + 8 + 4
        assert np.frombuffer(bytes(raw[eps_at:eps_at + 4]), np.float32)[0] == np.float32(1e-16)
        raw[eps_at:eps_at + 4] = np.float32(0.0).tobytes()
        open(path, "wb").write(bytes(raw))
        assert G.gem_load(g.h, path) == G.GEM_EIO


def test_empty_batch_and_run_are_no_ops(env):
    torch, G = env
    with G.Gem(10, 2) as g:
        g.set_quadratic(np.ones(10, np.float32), np.zeros(10, np.float32), 0.01, 0.1, 0)
        assert G.gem_commit_batch(g.h, [], G.GEM_F32, np.zeros(0, np.int32), None) == G.GEM_OK
        assert G.gem_sim_run(g.h, np.zeros(0, np.int32), None, 4) == G.GEM_OK
        assert g.clock == 0 and np.all(g.theta() == 0)


def test_copy_probe(env):
    torch, G = env
    # the last count needs more chunks than the grid's 2^20 blocks of 256
    # threads hold (grid-stride loop), with a ragged tail
    for count in (1, 4, 1003, 1 << 20, ((1 << 28) + 5) * 4 + 3):
        src = torch.arange(count, dtype=torch.float32, device="cuda")
        dst = torch.zeros(count, device="cuda")
        assert G.gem_copy_f32(src.data_ptr(), dst.data_ptr(), count) == G.GEM_OK
        torch.cuda.synchronize()
        assert torch.equal(src, dst)


@pytest.mark.parametrize("source", ["host", "device"])
def test_set_theta_restarts_from_theta0(env, source):
    """gem_set_theta: theta = theta0, every worker pulls it (S[w] = theta0, m = 0,
    clock and pull clocks 0), from host or device memory -- also mid-run; the
    run that follows equals the oracle started at theta0."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 3003, 4, 70
    h, ts = make_problem(P, 1e-3, 1.0, 12)
    rng = np.random.default_rng(12)
    theta0 = rng.standard_normal(P).astype(np.float32)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=12)
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 5)
        g.sim_run(worker[:20], tau[:20], 8)              # state to be discarded
        if source == "host":
            G.gem_set_theta(g.h, theta0)
        else:
            dev = torch.from_numpy(theta0).cuda()
            G.gem_set_theta(g.h, dev.data_ptr(), in_is_device=True)
            torch.cuda.synchronize()
        assert g.clock == 0 and np.all(g.pull_clocks() == 0)
        assert np.array_equal(g.theta(), theta0)
        assert np.all(g.S() == theta0[None, :]) and np.all(g.M() == 0)
        g.sim_run(worker, tau, 8)
        theta, S, M = g.theta(), g.S(), g.M()
    st = O.State.initial(n, P, theta0)
    O.run(O.Hyper(lr=0.01, sigma=0.1, seed=5), P, st, np.arange(P), h, ts, worker, tau)
    assert_parity("theta", theta, st.theta)
    assert_parity("S", S, st.S)
    assert_parity("M", M, st.M)


def test_reads_into_device_memory(env):
    """gem_read_theta and gem_read_state write device buffers as well as host
    ones, with the same values."""
    import ctypes as C
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 2050, 3
    h, ts = make_problem(P, 1e-3, 1.0, 13)
    worker, tau = G.gem_schedule_make(n, 30, G.GEM_LAW_EXP, seed=13)
    L = G.lib()
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 6)
        g.sim_run(worker, tau, 8)
        out = torch.zeros(P, dtype=torch.float32, device="cuda")
        assert L.gem_read_theta(g.h, C.c_void_p(out.data_ptr()), 1) == G.GEM_OK
        assert np.array_equal(out.cpu().numpy(), g.theta())
        for which, ref in ((G.GEM_SNAPSHOT, g.S()), (G.GEM_MOMENT, g.M())):
            for w in range(n):
                assert L.gem_read_state(g.h, w, which, C.c_void_p(out.data_ptr()), 1) == G.GEM_OK
                assert np.array_equal(out.cpu().numpy(), ref[w])
        assert L.gem_read_state(g.h, n, G.GEM_SNAPSHOT, C.c_void_p(out.data_ptr()), 1) == G.GEM_EWORKER
        assert L.gem_read_state(g.h, 0, 7, C.c_void_p(out.data_ptr()), 1) == G.GEM_EINVAL


def test_rows_read_across_tiles_into_misaligned_device_memory(env):
    """The snapshot and moment table is stored in tiles of 8192 parameters:
    rows read back whole across tile edges and a ragged last tile, into host
    memory, into device memory at a 4-byte offset, and through gem_gather."""
    import ctypes as C
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 3 * 8192 + 5, 3
    h, ts = make_problem(P, 1e-3, 1.0, 17)
    worker, tau = G.gem_schedule_make(n, 40, G.GEM_LAW_EXP, seed=17)
    hp = O.Hyper(lr=0.01, sigma=0.1, seed=8)
    st = O.State.initial(n, P)
    O.run(hp, P, st, np.arange(P), h, ts, worker, tau)
    L = G.lib()
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 8)
        g.sim_run(worker, tau, 32)
        assert_parity("theta", g.theta(), st.theta)
        buf = torch.full((P + 2,), -7.0, dtype=torch.float32, device="cuda")
        out = buf[1:P + 1]                        # 4 bytes past a 256-byte boundary
        for which, ref in ((G.GEM_SNAPSHOT, st.S), (G.GEM_MOMENT, st.M)):
            for w in range(n):
                assert L.gem_read_state(g.h, w, which, C.c_void_p(out.data_ptr()), 1) == G.GEM_OK
                got = buf.cpu().numpy()
                assert got[0] == -7.0 and got[-1] == -7.0       # nothing written outside
                assert_parity(f"row {w} ({which})", got[1:P + 1], ref[w])
        idx = np.array([0, 8191, 8192, 16383, 16384, 24575, 24576, P - 1], np.int64)
        th, S, M = g.gather(idx)
        assert np.array_equal(th, st.theta[idx])
        assert np.array_equal(S, st.S[:, idx]) and np.array_equal(M, st.M[:, idx])


def test_checkpoint_file_holds_contiguous_rows(env, tmp_path):
    """gem_save writes theta, then each worker's snapshot row, then each moment
    row as P contiguous floats, then the pull clocks, h and theta* -- the
    file layout does not depend on the device table's tiles."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 2 * 8192 + 77, 3
    h, ts = make_problem(P, 1e-3, 1.0, 19)
    worker, tau = G.gem_schedule_make(n, 50, G.GEM_LAW_EXP, seed=19)
    path = str(tmp_path / "ck.bin")
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 9)
        g.sim_run(worker, tau, 16)
        assert G.gem_save(g.h, path) == G.GEM_OK
        theta, S, M, pc = g.theta(), g.S(), g.M(), g.pull_clocks()
    raw = open(path, "rb").read()
    body = (1 + 2 * n + 2) * P * 4 + 8 * n
    hdr = len(raw) - body
    assert hdr > 0 and raw[:8] == b"GEMCKPT2"
    f = np.frombuffer(raw, dtype=np.float32, count=(1 + 2 * n) * P, offset=hdr).reshape(1 + 2 * n, P)
    assert np.array_equal(f[0], theta)
    assert np.array_equal(f[1:1 + n], S) and np.array_equal(f[1 + n:], M)
    off = hdr + (1 + 2 * n) * P * 4
    assert np.array_equal(np.frombuffer(raw, dtype=np.int64, count=n, offset=off), pc)
    tail = np.frombuffer(raw, dtype=np.float32, count=2 * P, offset=off + 8 * n).reshape(2, P)
    assert np.array_equal(tail[0], h) and np.array_equal(tail[1], ts)


def test_load_refuses_damaged_files_and_keeps_the_state(env, tmp_path):
    """gem_load checks the whole file before it writes anything: a truncated
    file, a clock outside [0, 2^32), or a pull clock after the clock is
    GEM_EIO, and the handle's state stays as it was."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n = 3000, 3
    h, ts = make_problem(P, 1e-3, 1.0, 23)
    worker, tau = G.gem_schedule_make(n, 40, G.GEM_LAW_EXP, seed=23)
    path = str(tmp_path / "ck.bin")
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 9)
        g.sim_run(worker, tau, 8)
        assert G.gem_save(g.h, path) == G.GEM_OK
    raw = bytearray(open(path, "rb").read())
    hdr = len(raw) - ((1 + 2 * n + 2) * P * 4 + 8 * n)
    pc_at = hdr + (1 + 2 * n) * P * 4
    t_at = 24   # magic, P, n, have_problem, then t
    assert int.from_bytes(raw[t_at:t_at + 8], "little", signed=True) == 40

    def damaged(edit):
        b = bytearray(raw)
        edit(b)
        q = str(tmp_path / "bad.bin")
        open(q, "wb").write(bytes(b))
        return q

    bad = [
        damaged(lambda b: b.__delitem__(slice(len(b) - 4, len(b)))),            # truncated
        damaged(lambda b: b.__setitem__(slice(t_at, t_at + 8), (-1).to_bytes(8, "little", signed=True))),
        damaged(lambda b: b.__setitem__(slice(t_at, t_at + 8), (2**32).to_bytes(8, "little"))),
        damaged(lambda b: b.__setitem__(slice(pc_at, pc_at + 8), (41).to_bytes(8, "little"))),
        damaged(lambda b: b.__setitem__(slice(pc_at + 8, pc_at + 16), (-3).to_bytes(8, "little", signed=True))),
    ]
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 9)
        g.sim_run(worker[:10], tau[:10], 8)
        before = (g.theta(), g.S(), g.M(), g.clock, g.pull_clocks())
        for q in bad:
            assert G.gem_load(g.h, q) == G.GEM_EIO, q
        after = (g.theta(), g.S(), g.M(), g.clock, g.pull_clocks())
        for x, y in zip(before, after):
            assert np.array_equal(x, y)
        assert G.gem_load(g.h, path) == G.GEM_OK and g.clock == 40


def test_diag_reset_restarts_the_sums(env):
    """gem_diag_reset zeroes the energy sums and counts; what follows sums only
    the later commits (against the oracle's per-commit diagnostics)."""
    torch, G = env
    from paper_1805_08469_amd.workloads import make_problem
    P, n, T = 4001, 4, 60
    h, ts = make_problem(P, 1e-3, 1.0, 14)
    worker, tau = G.gem_schedule_make(n, T, G.GEM_LAW_EXP, seed=14)
    with G.Gem(P, n) as g:
        g.set_quadratic(h, ts, 0.01, 0.1, 8)
        G.gem_diag_enable(g.h, True)
        g.sim_run(worker[:25], tau[:25], 8)
        G.gem_diag_reset(g.h)
        d0 = G.gem_diag(g.h)
        assert (d0.sum_ek, d0.sum_proxy, d0.n_clamped, d0.n_elem_commits, d0.n_commits) == \
               (0.0, 0.0, 0, 0, 0)
        g.sim_run(worker[25:], tau[25:], 8)
        d = G.gem_diag(g.h)
    st = O.State.initial(n, P)
    hp = O.Hyper(lr=0.01, sigma=0.1, seed=8)
    dg, _ = O.run(hp, P, st, np.arange(P), h, ts, worker, tau, diag=True)
    later = dg[25:]
    assert d.n_commits == T - 25
    assert d.n_elem_commits == P * (T - 25)
    assert d.n_clamped == int(later["n_clamped"].sum())
    assert d.sum_ek == pytest.approx(float(later["sum_ek"].sum()), rel=1e-9)
    assert d.sum_proxy == pytest.approx(float(later["sum_proxy"].sum()), rel=1e-9)
