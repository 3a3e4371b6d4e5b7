"""Seeded synthetic inputs for the collectives.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no part of the collectives' arithmetic: it only draws numbers and turns
them into the raw element bit patterns the library and the CPU oracle both
consume (``uint32`` arrays for binary32, ``uint16`` arrays for bfloat16,
shaped ``[P, n]``).

Recipes (rank r draws from its own generator, seed ``seed + r``, unless a
recipe says otherwise):

* ``uniform``  -- numpy PCG64 ``uniform(-1, 1)`` in float64, rounded to float32.
* ``normal``   -- ``normal(0, sigma)`` in float64, rounded to float32 and, for
  bfloat16, rounded again to bfloat16 by torch's CPU conversion.
* ``adversarial`` -- one generator (seed ``seed``) for all ranks: values across
  the +-65504 range, half of the elements
  with near-cancelling rank pairs (2k, 2k+1), all rounded to bfloat16;
  accumulating in bfloat16 instead of binary32 changes many results.
* ``ones`` / ``rank_index`` -- closed-form fills.
"""
from __future__ import annotations

import numpy as np

F32 = "f32"
BF16 = "bf16"
_ELEM_BYTES = {F32: 4, BF16: 2}


def elem_bytes(dtype: str) -> int:
    return _ELEM_BYTES[dtype]


def _to_bits(values_f32: np.ndarray, dtype: str) -> np.ndarray:
    values_f32 = np.ascontiguousarray(values_f32, dtype=np.float32)
    if dtype == F32:
        return values_f32.view(np.uint32).copy()
    if dtype == BF16:
        import torch

        t = torch.from_numpy(values_f32).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    raise ValueError(dtype)


def uniform(nranks: int, n: int, dtype: str = F32, seed: int = 0) -> np.ndarray:
    rows = [np.random.default_rng(seed + r).uniform(-1.0, 1.0, n).astype(np.float32)
            for r in range(nranks)]
    return _to_bits(np.stack(rows) if n else np.zeros((nranks, 0), np.float32), dtype)


def normal(nranks: int, n: int, dtype: str = BF16, sigma: float = 1.0, seed: int = 0) -> np.ndarray:
    rows = [np.random.default_rng(seed + r).normal(0.0, sigma, n).astype(np.float32)
            for r in range(nranks)]
    return _to_bits(np.stack(rows) if n else np.zeros((nranks, 0), np.float32), dtype)


def ones(nranks: int, n: int, dtype: str) -> np.ndarray:
    return _to_bits(np.ones((nranks, n), np.float32), dtype)


def rank_index(nranks: int, n: int, dtype: str) -> np.ndarray:
    return _to_bits(np.repeat(np.arange(nranks, dtype=np.float32)[:, None], n, axis=1), dtype)


def adversarial(nranks: int, n: int, seed: int = 0) -> np.ndarray:
    """bfloat16 inputs built so that the rounding scheme matters.

    Every rank holds values of magnitude U[0, 65504] with a random sign.  In
    half of the elements (chosen at random) each odd rank 2k+1 instead holds
    the near-opposite of rank 2k, -x_{2k} * (1 + e) with e ~ U[-2^-6, 2^-6],
    so the pair nearly cancels and the exact sum is small.  All values are
    rounded to bfloat16.  Accumulating in bfloat16 (rounding after every add)
    instead of binary32 with one final rounding changes many of the results.
    """
    rng = np.random.default_rng(seed)
    mags = rng.uniform(0.0, 65504.0, (nranks, n))
    signs = np.where(rng.random((nranks, n)) < 0.5, -1.0, 1.0)
    vals = signs * mags
    cancel = rng.random(n) < 0.5
    for r in range(1, nranks, 2):
        jitter = rng.uniform(-2.0 ** -6, 2.0 ** -6, n)
        vals[r] = np.where(cancel, -vals[r - 1] * (1.0 + jitter), vals[r])
    return _to_bits(vals.astype(np.float32), BF16)


def make(kind: str, nranks: int, n: int, dtype: str, seed: int = 0, sigma: float = 1.0) -> np.ndarray:
    if kind == "uniform":
        return uniform(nranks, n, dtype, seed)
    if kind == "normal":
        return normal(nranks, n, dtype, sigma, seed)
    if kind == "ones":
        return ones(nranks, n, dtype)
    if kind == "rank_index":
        return rank_index(nranks, n, dtype)
    if kind == "adversarial":
        if dtype != BF16:
            raise ValueError("the adversarial recipe is bfloat16")
        return adversarial(nranks, n, seed)
    raise ValueError(kind)
