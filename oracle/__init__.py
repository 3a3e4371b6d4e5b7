"""CPU oracle for the low-latency collectives -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (``include/llcoll.h``,
the HIP library under ``paper_2607_16100_amd/csrc`` and its Python binding)
never imports, links or calls anything here, and nothing here imports the
product.  The two sides share only the seeded input generators
(``paper_2607_16100_amd.workloads``), which hold none of the method's
arithmetic.

Two independent oracles live here:

* ``llref.c`` -- plain C loops (gcc, -O2 -fno-fast-math), loaded with ctypes.
  It is the primary oracle: the element-wise sum of the P rank buffers in
  ascending rank order, accumulated in binary32, rounded once to the element
  type (AllReduce, Sec. III; error analysis at the end of Sec. IV; recvReduce's
  accumulator conversion, Sec. V).  ReduceScatter keeps chunk r of that sum on
  rank r; AllGather concatenates the inputs (two-shot, Sec. III-A).
* ``npref.py`` -- the same definition written with numpy float32 arithmetic and
  its own round-to-nearest-even; the tests require both to agree bit for bit.

Arrays are passed as raw bit patterns: ``uint32`` for binary32 and ``uint16``
for bfloat16, shaped ``[P, n]``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import npref  # noqa: F401  (re-exported for the tests)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "llref.c")
_LIB = os.path.join(_HERE, "libllref.so")

F32 = 0
BF16 = 1

_lib = None


def build(force: bool = True) -> str:
    """Compile ``llref.c`` into ``libllref.so`` with gcc (IEEE scalar SSE math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        cmd = [
            "gcc", "-O2", "-std=c99", "-fno-fast-math", "-ffp-contract=off",
            "-fno-unsafe-math-optimizations", "-msse2", "-mfpmath=sse",
            "-Wall", "-Wextra", "-shared", "-fPIC", "-o", _LIB + ".tmp", _SRC,
        ]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        vp, sz, ci = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
        for name in ("ref_allreduce", "ref_reduce_scatter", "ref_allgather"):
            fn = getattr(lib, name)
            fn.argtypes = [vp, vp, sz, ci, ci]
            fn.restype = ci
        for name in ("ref_broadcast", "ref_reduce"):
            fn = getattr(lib, name)
            fn.argtypes = [vp, vp, sz, ci, ci, ci]
            fn.restype = ci
        lib.ref_bf16_from_f32_bits.argtypes = [ctypes.c_uint32]
        lib.ref_bf16_from_f32_bits.restype = ctypes.c_uint16
        lib.ref_f32_bits_from_bf16.argtypes = [ctypes.c_uint16]
        lib.ref_f32_bits_from_bf16.restype = ctypes.c_uint32
        _lib = lib
    return _lib


def _dtype_code(bits: np.ndarray) -> int:
    if bits.dtype == np.uint32:
        return F32
    if bits.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle takes uint32 (binary32 bits) or uint16 (bfloat16 bits), got {bits.dtype}")


def _prep(x: np.ndarray) -> np.ndarray:
    if x.ndim != 2:
        raise ValueError("inputs are shaped [P, n]")
    return np.ascontiguousarray(x)


def allreduce(x: np.ndarray) -> np.ndarray:
    """out[r, i] = round(x[0, i] + x[1, i] + ... + x[P-1, i]) for every rank r."""
    x = _prep(x)
    p, n = x.shape
    out = np.empty_like(x)
    rc = _load().ref_allreduce(x.ctypes.data, out.ctypes.data, n, _dtype_code(x), p)
    if rc != 0:
        raise ValueError("ref_allreduce rejected its arguments")
    return out


def reduce_scatter(x: np.ndarray) -> np.ndarray:
    """x is [P, P*m]; out[r] is chunk r (elements r*m .. r*m+m-1) of the sum."""
    x = _prep(x)
    p, total = x.shape
    if total % p:
        raise ValueError("reduce_scatter input length must be a multiple of P")
    m = total // p
    out = np.empty((p, m), dtype=x.dtype)
    rc = _load().ref_reduce_scatter(x.ctypes.data, out.ctypes.data, m, _dtype_code(x), p)
    if rc != 0:
        raise ValueError("ref_reduce_scatter rejected its arguments")
    return out


def allgather(x: np.ndarray) -> np.ndarray:
    """x is [P, s]; out[r] is x[0] ++ x[1] ++ ... ++ x[P-1] for every rank r."""
    x = _prep(x)
    p, s = x.shape
    out = np.empty((p, p * s), dtype=x.dtype)
    rc = _load().ref_allgather(x.ctypes.data, out.ctypes.data, s, _dtype_code(x), p)
    if rc != 0:
        raise ValueError("ref_allgather rejected its arguments")
    return out


def broadcast(x: np.ndarray, root: int) -> np.ndarray:
    """x is [P, n]; out[r] is x[root] for every rank r."""
    x = _prep(x)
    p, n = x.shape
    out = np.empty_like(x)
    rc = _load().ref_broadcast(x.ctypes.data, out.ctypes.data, n, _dtype_code(x), p, root)
    if rc != 0:
        raise ValueError("ref_broadcast rejected its arguments")
    return out


def reduce(x: np.ndarray, root: int) -> np.ndarray:
    """x is [P, n]; the root's result: the ordered sum of the P rows, rounded once."""
    x = _prep(x)
    p, n = x.shape
    out = np.empty(n, dtype=x.dtype)
    rc = _load().ref_reduce(x.ctypes.data, out.ctypes.data, n, _dtype_code(x), p, root)
    if rc != 0:
        raise ValueError("ref_reduce rejected its arguments")
    return out


def bf16_from_f32_bits(u: int) -> int:
    return int(_load().ref_bf16_from_f32_bits(int(u) & 0xFFFFFFFF))


def f32_bits_from_bf16(h: int) -> int:
    return int(_load().ref_f32_bits_from_bf16(int(h) & 0xFFFF))
