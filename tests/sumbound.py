"""Acceptance test for results whose summation order is not fixed (the
atomic-accumulation two-shot): the forward-error bound of floating-point
summation quoted at the end of the paper's Sec. IV."""
from __future__ import annotations

import numpy as np


def gamma(k: int, u: float = 2.0 ** -24) -> float:
    """gamma_k = k u / (1 - k u)."""
    return k * u / (1 - k * u)


def to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return bits.view(np.float32).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_within_summation_bound(got: np.ndarray, x: np.ndarray, dtype: str, what: str) -> None:
    """`got` [P, n] (raw bits) must hold the same bits on every rank, and each
    element must be within gamma_{P-1} * sum_i |x_i| of the exact sum of the
    P inputs (binary32 accumulation in any order), plus one rounding to
    bfloat16 (half an ulp, 2^-8 relative) for bfloat16 results."""
    p = x.shape[0]
    assert (got == got[0]).all(), f"{what}: ranks disagree"
    xf = to_f64(x, dtype)
    exact = xf.sum(axis=0)
    mag = np.abs(xf).sum(axis=0)
    y = to_f64(got[0], dtype)
    tol = gamma(p - 1) * mag + 2.0 ** -45 * mag
    if dtype == "bf16":
        tol = tol + 2.0 ** -8 * np.abs(y)
    err = np.abs(y - exact)
    bad = np.flatnonzero(~(err <= tol))
    assert bad.size == 0, (f"{what}: {bad.size} elements outside the bound; first {bad[0]}: "
                           f"got {y[bad[0]]!r} exact {exact[bad[0]]!r} tol {tol[bad[0]]!r}")
