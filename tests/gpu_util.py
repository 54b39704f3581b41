"""Helpers shared by the GPU tests (no kernel code, no method arithmetic)."""
import numpy as np


def parity(gpu, ref):
    """(max relative error, number of entries that are not bit-identical).

    Relative error is |x - y| / max(|y|, 1e-3 rms(y)), so entries near zero are
    measured against the array's scale.  NaNs compare equal to NaNs (their
    payload bits may differ between the host and the device), and +0 equals -0:
    every use of a value in the method goes through |.| or an fma, so the sign
    of a zero never reaches a non-zero result."""
    x = np.asarray(gpu, dtype=np.float32)
    y = np.asarray(ref, dtype=np.float32)
    assert x.shape == y.shape
    both_nan = np.isnan(x) & np.isnan(y)
    both_zero = (x == 0) & (y == 0)        # +0 and -0 compare by value
    same_bits = (x.view(np.uint32) == y.view(np.uint32)) | both_nan | both_zero
    xd, yd = x.astype(np.float64), y.astype(np.float64)
    fin = np.isfinite(yd)
    rms = np.sqrt(np.mean(yd[fin] ** 2)) if fin.any() else 0.0
    scale = np.maximum(np.abs(yd), max(1e-3 * rms, 1e-30))
    with np.errstate(invalid="ignore"):
        rel = np.where(same_bits, 0.0, np.abs(xd - yd) / scale)
    rel = np.where(np.isnan(rel), np.inf, rel)
    return float(rel.max()) if rel.size else 0.0, int((~same_bits).sum())


def assert_parity(name, gpu, ref, tol=1e-5):
    """The parity bar: max relative error <= 1e-5; the design makes every
    entry bit-identical, which is checked too."""
    rel, bad = parity(gpu, ref)
    assert rel <= tol, f"{name}: max relative error {rel:.3e} ({bad} entries differ)"
    assert bad == 0, f"{name}: {bad} entries are not bit-identical (max rel {rel:.3e})"
