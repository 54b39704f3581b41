"""GPU parity of the noise and the stale-gradient generator (gem_generate)
against the oracle, bit for bit."""
import numpy as np
import pytest

import oracle as O
from f32 import fma32
from gpu_util import assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_08469_amd import gem  # noqa: F401  (fails loudly without the HIP library)
    return torch


def _gen(torch, g, P, w, dtype):
    from paper_1805_08469_amd import gem as G
    if dtype == G.GEM_F32:
        out = torch.empty(P, dtype=torch.float32, device="cuda")
    else:
        out = torch.empty(P, dtype=torch.int16, device="cuda")
    rc = G.gem_generate(g.h, w, out.data_ptr(), dtype)
    assert rc == G.GEM_OK, G.gem_strerror(rc)
    torch.cuda.synchronize()
    a = out.cpu().numpy()
    if dtype == G.GEM_BF16:
        a = (a.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    return a


@pytest.mark.parametrize("seed", [0, 12345, 2**40 + 977])
def test_normals_bit_exact(torch_cuda, seed):
    """lr = -1, sigma = 1, h = 0 make the generator emit xi itself:
    dtheta = 1 * fma(0, s - theta*, 1 * xi) = xi."""
    from paper_1805_08469_amd import gem as G
    torch = torch_cuda
    P = (1 << 22) + 37
    with G.Gem(P, 2) as g:
        g.set_quadratic(np.zeros(P, np.float32), np.zeros(P, np.float32), -1.0, 1.0, seed)
        zeros = torch.zeros(P, dtype=torch.float32, device="cuda")
        for t in range(4):
            xi = _gen(torch, g, P, 0, G.GEM_F32)
            ref = O.normals(seed, t, 0, P)
            assert_parity(f"xi(t={t})", xi, ref)
            g.commit(zeros.data_ptr(), 1)   # advance the clock
        assert g.clock == 4


@pytest.mark.parametrize("P", [1, 5, 64, 1000, 65537])
@pytest.mark.parametrize("bf16", [False, True])
def test_generate_bit_exact(torch_cuda, P, bf16):
    from paper_1805_08469_amd import gem as G
    from paper_1805_08469_amd.workloads import make_problem
    torch = torch_cuda
    h, ts = make_problem(P, 1e-4, 1.0, 3)
    lr, sigma, seed = 0.01, 0.05, 99
    with G.Gem(P, 3) as g:
        g.set_quadratic(h, ts, lr, sigma, seed)
        d = _gen(torch, g, P, 2, G.GEM_BF16 if bf16 else G.GEM_F32)
    xi = O.normals(seed, 0, 0, P)
    s = np.zeros(P, np.float32)
    ref = (np.float32(-lr) * fma32(h, s - ts, np.float32(sigma) * xi)).astype(np.float32)
    if bf16:
        ref = O.round_bf16(ref)
    assert_parity("dtheta", d, ref)
