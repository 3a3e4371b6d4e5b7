"""Second, independent oracle in numpy -- TEST INFRASTRUCTURE ONLY.

Same definition as ``llref.c`` (AllReduce of Sec. III; binary32 accumulation in
ascending rank order with one final rounding, per the summation error analysis
at the end of Sec. IV and recvReduce's accumulator conversion in Sec. V), but
written with numpy's element-wise float32 addition and a round-to-nearest-even
of its own.  It exists so that a mistake in one oracle shows up as a
disagreement with the other.
"""
from __future__ import annotations

import numpy as np


def widen(bits: np.ndarray) -> np.ndarray:
    """Raw element bits -> float32 values (bfloat16 widening is a 16-bit shift)."""
    if bits.dtype == np.uint32:
        return bits.view(np.float32)
    if bits.dtype == np.uint16:
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    raise TypeError(bits.dtype)


def narrow(values: np.ndarray, like: np.dtype) -> np.ndarray:
    """float32 values -> raw element bits of type ``like`` (uint32 or uint16)."""
    values = np.asarray(values, dtype=np.float32)
    if like == np.uint32:
        return values.view(np.uint32).copy()
    if like != np.uint16:
        raise TypeError(like)
    u = values.view(np.uint32).astype(np.uint64)
    is_nan = ((u & 0x7F800000) == 0x7F800000) & ((u & 0x007FFFFF) != 0)
    # Split into the kept upper 16 bits and the 16 discarded bits, then round
    # the discarded part: above half -> up, below -> down, exactly half -> to
    # the even kept value.
    kept = u >> 16
    rest = u & 0xFFFF
    up = (rest > 0x8000) | ((rest == 0x8000) & ((kept & 1) == 1))
    rounded = kept + up.astype(np.uint64)
    quiet_nan = (kept | 0x0040)
    out = np.where(is_nan, quiet_nan, rounded)
    return (out & 0xFFFF).astype(np.uint16)


def allreduce(x: np.ndarray) -> np.ndarray:
    p = x.shape[0]
    with np.errstate(over="ignore", invalid="ignore"):
        acc = widen(x[0]).copy()
        for q in range(1, p):
            acc = (acc + widen(x[q])).astype(np.float32)
    y = narrow(acc, x.dtype)
    return np.broadcast_to(y, x.shape).copy()


def reduce_scatter(x: np.ndarray) -> np.ndarray:
    p, total = x.shape
    m = total // p
    full = allreduce(x)[0]
    return np.stack([full[r * m:(r + 1) * m] for r in range(p)])


def allgather(x: np.ndarray) -> np.ndarray:
    p = x.shape[0]
    row = np.concatenate([x[q] for q in range(p)])
    return np.broadcast_to(row, (p, row.shape[0])).copy()
