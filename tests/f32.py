"""Exact binary32 helpers for tests (numpy has no single-precision fma).

fma32(a, b, c) returns RN_32(a*b + c) exactly: a*b is exact in binary64
(24 x 24 bits), the binary64 sum is made round-to-odd from its exact error
term, and binary64 round-to-odd followed by rounding to binary32 equals a
single rounding because 53 >= 24 + 2 (Boldo & Melquiond, 2008).
"""
import numpy as np


def fma32(a, b, c):
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    b = np.asarray(b, dtype=np.float32).astype(np.float64)
    c = np.asarray(c, dtype=np.float32).astype(np.float64)
    p = a * b
    s = p + c
    bb = s - p
    err = (p - (s - bb)) + (c - bb)
    bits = s.view(np.int64)
    inexact = err != 0
    even = (bits & 1) == 0
    fix = inexact & even & np.isfinite(s)
    toward = np.where(err > 0, np.inf, -np.inf)
    s = np.where(fix, np.nextafter(s, toward), s)
    return s.astype(np.float32)
