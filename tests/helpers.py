"""Shared helpers of the GPU parity tests: host copies of device inputs and
the tolerance check.

Tolerance (floating point): a GPU result y matches the binary64 oracle value
r when |y - r| <= TOL * max(|r|, M), with M the magnitude of the terms that
produce r (their absolute values summed the way the result sums them).
Element-wise relative error alone is ill-conditioned where terms cancel, so
it is guarded by M:
  reduce SUM:   M = sum_i |in_i|            (AVG: that / K)
  easgd worker: M = |x_i| + |eta| (|g_i| + |rho| |x_i - c|)
  easgd center: M = |c| + |eta rho| sum_i |x_i - c|
A binary32 implementation that sums K terms pairwise has error at most
about (log2 K + 3) * 2^-24 * M, under 4e-7 M for K <= 64, so TOL = 1e-5
holds with more than 20x margin for any correct summation order.
"""

from __future__ import annotations

import numpy as np
import torch

TOL = 1e-5


def host_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy().copy()


def host_stored(t: torch.Tensor) -> np.ndarray:
    """Host copy in the oracle's stored form: float32, or uint16 bf16 codes."""
    if t.dtype == torch.bfloat16:
        return t.detach().view(torch.int16).to("cpu").numpy().view(np.uint16).copy()
    return host_f32(t)


def widened(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def guarded_ratio(y: np.ndarray, ref: np.ndarray, mag: np.ndarray) -> float:
    """max |y - ref| / (TOL * max(|ref|, mag)); <= 1 passes."""
    y = y.astype(np.float64)
    if y.size == 0:
        return 0.0
    both_nan = np.isnan(y) & np.isnan(ref)
    den = TOL * np.maximum(np.abs(ref), mag)
    err = np.abs(y - ref)
    err[both_nan] = 0.0
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.where(den > 0, err / np.where(den > 0, den, 1.0), np.where(err == 0, 0.0, np.inf))
    return float(np.max(r))


def reduce_mag(ins, op_avg: bool) -> np.ndarray:
    m = sum(np.abs(widened(a)) for a in ins)
    return m / len(ins) if op_avg else m


def easgd_mags(xs, gs, xc, eta, rho):
    """Guard magnitudes of one step from the step's inputs (binary64)."""
    c = xc.astype(np.float64)
    ds = [x.astype(np.float64) - c for x in xs]
    mx = [np.abs(x.astype(np.float64)) + abs(eta) * (np.abs(widened(g)) + abs(rho) * np.abs(d))
          for x, g, d in zip(xs, gs, ds)]
    mc = np.abs(c) + abs(eta * rho) * sum(np.abs(d) for d in ds)
    return mx, mc


def assert_close(y, ref, mag, what=""):
    r = guarded_ratio(y, ref, mag)
    assert r <= 1.0, f"{what}: guarded error {r * TOL:.3e} exceeds {TOL} (ratio {r:.3f})"
    return r


def assert_bits_equal(a: np.ndarray, b: np.ndarray, what=""):
    assert a.shape == b.shape, what
    av = a.view(np.uint8) if a.dtype != np.uint8 else a
    bv = b.view(np.uint8) if b.dtype != np.uint8 else b
    if not np.array_equal(av, bv):
        bad = np.nonzero(a != b)[0]
        raise AssertionError(f"{what}: {bad.size} elements differ, first at {bad[:5]}")


def assert_exact(y: np.ndarray, ref64: np.ndarray, what=""):
    """Values equal exactly (the oracle's binary64 value is representable in
    binary32; +0 and -0 compare equal)."""
    assert np.array_equal(ref64.astype(np.float32).astype(np.float64), ref64), f"{what}: reference not binary32"
    bad = np.nonzero(y.astype(np.float64) != ref64)[0]
    assert bad.size == 0, f"{what}: {bad.size} elements differ, first at {bad[:5]}: {y[bad[:5]]} vs {ref64[bad[:5]]}"
