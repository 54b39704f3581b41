"""Pins of the oracle's random-number layer against independent sources.

* Philox (Salmon et al., SC'11): the round and key-schedule structure is
  checked on the 64-bit-word member of the family against numpy's own
  Philox4x64-10; the 32-bit Weyl constants against their closed forms
  (golden ratio, sqrt(3) - 1); the 32-bit member against the known-answer
  values published with the reference implementation of that paper.
* Gaussian noise (Box & Muller 1958): the binary32 ln and sin/cos are checked
  exhaustively over every input the transform can see against numpy's
  binary64 libm, and the resulting normals against N(0, 1) statistically.
* bfloat16 rounding: against torch's CPU float -> bfloat16 conversion.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
from scipy import stats

import oracle as O


def test_philox4x64_matches_numpy():
    # numpy's Philox advances its 256-bit counter by one before each block.
    for key, ctr in [((0, 0), (0, 0, 0, 0)), ((0x1234, 0xABCD), (5, 0, 0, 0)),
                     ((2**64 - 1, 7), (2**64 - 1, 3, 0, 9))]:
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.array(ctr, dtype=np.uint64))
        ref = bg.random_raw(4)
        c = list(ctr)
        c[0] = (c[0] + 1) % 2**64
        if c[0] == 0:
            c[1] = (c[1] + 1) % 2**64
        got = O.philox4x64(c, key)
        assert [int(x) for x in got] == [int(x) for x in ref]


def test_philox_weyl_constants_closed_form():
    golden = (math.sqrt(5) - 1) / 2
    assert O.philox_weyl32(0) == math.floor(golden * 2**32)
    assert O.philox_weyl32(1) == math.floor((math.sqrt(3) - 1) * 2**32)
    # 64-bit: use exact integer square roots.
    s5 = math.isqrt(5 * 2**128)          # floor(sqrt(5) 2^64)
    assert O.philox_weyl64(0) == (s5 - 2**64) // 2
    s3 = math.isqrt(3 * 2**128)
    assert O.philox_weyl64(1) == s3 - 2**64


@pytest.mark.parametrize("ctr,key,expect", [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
])
def test_philox4x32_known_answers(ctr, key, expect):
    assert tuple(int(x) for x in O.philox4x32(ctr, key)) == expect


def test_ln2_split():
    # LN2_LO is ln2 - LN2_HI rounded to binary32; ln 2 from a rapidly
    # converging series ln 2 = sum 1/(k 2^k) in exact rationals.
    ln2 = sum(Fraction(1, k * 2**k) for k in range(1, 80))
    hi = Fraction(0x162E4, 2**17)
    lo = float(ln2 - hi)
    assert O.ln2_lo() == float(np.float32(lo))


def test_log_unit_exhaustive():
    # Every u1 = k 2^-24, k = 1..2^24 that the Box-Muller transform uses.
    k = np.arange(1, 2**24 + 1, dtype=np.float64)
    u = (k * 2.0**-24).astype(np.float32)
    got = O.log_unit(u).astype(np.float64)
    ref = np.log(u.astype(np.float64))
    assert got[-1] == 0.0                         # ln 1 = 0 exactly
    nz = ref != 0
    ulp = np.spacing(np.abs(ref[nz]).astype(np.float32)).astype(np.float64)
    assert np.max(np.abs(got[nz] - ref[nz]) / ulp) < 2.0
    assert np.all(got[:-1] < 0)


def test_sincos_turn24_exhaustive():
    k = np.arange(0, 2**24, dtype=np.uint32)
    s, c = O.sincos_turn24(k)
    ang = 2 * np.pi * k.astype(np.float64) / 2**24
    assert np.max(np.abs(s - np.sin(ang))) < 1.5 * 2**-23
    assert np.max(np.abs(c - np.cos(ang))) < 1.5 * 2**-23
    # exact quarter turns
    for kk, es, ec in [(0, 0.0, 1.0), (2**22, 1.0, 0.0), (2**23, 0.0, -1.0), (3 * 2**22, -1.0, 0.0)]:
        assert s[kk] == es and c[kk] == ec


def test_normals_are_standard_normal():
    z = np.concatenate([O.normals(seed, t, 0, 1_000_000) for seed, t in [(1, 0), (2**40 + 3, 77)]])
    assert abs(z.mean()) < 5 / math.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * math.sqrt(2 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # the four elements of one Philox call are independent-looking pairs
    r = np.corrcoef(z[0::4], z[1::4])[0, 1]
    assert abs(r) < 5 / math.sqrt(z.size / 4)


def test_normals_keyed_by_seed_t_i():
    a = O.normals(9, 4, 0, 64)
    assert np.array_equal(a[10:20], O.normals(9, 4, 10, 10))
    assert np.array_equal(a[[3, 17, 63]], O.normals_at(9, 4, [3, 17, 63]))
    assert not np.array_equal(a, O.normals(9, 5, 0, 64))
    assert not np.array_equal(a, O.normals(10, 4, 0, 64))


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(3)
    x = np.concatenate([
        rng.standard_normal(100_000).astype(np.float32) * np.float32(1e-3),
        rng.integers(0, 2**32, 100_000, dtype=np.uint64).astype(np.uint32).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.0e38, -3.0e38, 1e-40], dtype=np.float32),
    ])
    x = x[~np.isnan(x)]
    got = O.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
