"""The device numerics against the IEEE operations, on the GPU, bit for bit.

The commit kernels take correctly rounded division and square root through
range-specialised forms (gem_device.hpp) where the general sequences' range
handling has nothing to do.  libgem_selftest.so compares them with hipcc's
general IEEE division and square root on the device: exhaustively over the
logarithm's quotient and the Box-Muller radius (the only inputs those forms
get), and for the guarded quotient of the scale factor on 2^30 random pairs
over the whole binary32 range plus every denominator significand of selected
binades against a spread of numerators."""
import ctypes as C
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_1805_08469_amd", "libgem_selftest.so")


@pytest.fixture(scope="module")
def lib():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} is not built")
    L = C.CDLL(LIB)
    u64p = C.POINTER(C.c_uint64)
    L.gem_selftest_ln_div.argtypes = [u64p]
    L.gem_selftest_radius.argtypes = [u64p]
    L.gem_selftest_div_random.argtypes = [C.c_uint64, C.c_int64, u64p]
    L.gem_selftest_div_grid.argtypes = [C.POINTER(C.c_float), C.c_int32, C.c_int32, u64p]
    return L


def _count(fn, *args):
    out = C.c_uint64(123456789)
    rc = fn(*args, C.byref(out))
    assert rc == 0, f"self-test returned {rc}"
    return out.value


def test_logarithm_quotient_exhaustive(lib):
    assert _count(lib.gem_selftest_ln_div) == 0


def test_box_muller_radius_exhaustive(lib):
    assert _count(lib.gem_selftest_radius) == 0


@pytest.mark.parametrize("seed", [1, 20180522])
def test_scale_factor_quotient_random(lib, seed):
    assert _count(lib.gem_selftest_div_random, seed, 1 << 30) == 0


@pytest.mark.parametrize("e_den", [-126, -61, -60, -59, -30, -1, 0, 1, 30, 59, 60, 61, 127])
def test_scale_factor_quotient_grid(lib, e_den):
    """Every significand of den in [2^e, 2^(e+1)) against numerators spread
    over +-[2^-70, 2^70] with the core range's edges, zeros, subnormals,
    infinities and NaN."""
    rng = np.random.default_rng(e_den + 1000)
    mags = np.ldexp(1.0 + rng.random(200), rng.integers(-70, 71, size=200))
    edges = [2.0 ** -60, 2.0 ** 60, np.nextafter(2.0 ** -60, 0), np.nextafter(2.0 ** 60, np.inf),
             0.0, 1e-40, 3.4e38, np.inf, np.nan, 1.0]
    nums = np.concatenate([mags * rng.choice([-1.0, 1.0], size=200), edges, [-e for e in edges]])
    nums = np.ascontiguousarray(nums.astype(np.float32))
    assert _count(lib.gem_selftest_div_grid, nums.ctypes.data_as(C.POINTER(C.c_float)), nums.size,
                  e_den) == 0
