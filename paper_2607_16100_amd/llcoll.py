"""Python binding of the llcoll C ABI (``include/llcoll.h``, ``include/llprobe.h``,
``include/lltune.h``).

Argument marshalling only: every function has the C name, takes the same
arguments (device pointers and streams as integers; options as an
``Options`` object or None) and returns the C status code.  All computation
happens in the HIP library; if the library has not been built this module
fails to import -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# LLCOLL_LIBRARY may name another build of the same library (e.g. one built
# with different compile-time options); by default the in-tree build is used.
LIB_PATH = os.environ.get("LLCOLL_LIBRARY") or os.path.join(_HERE, "libllcoll.so")

LL_F32, LL_BF16 = 0, 1
LL_SUM = 0
LL_ALGO_AUTO, LL_ALGO_ONESHOT, LL_ALGO_TWOSHOT, LL_ALGO_TWOSHOT_LINE, LL_ALGO_ONESHOT_LINE = 0, 1, 2, 3, 4
LL_ALGO_ONESHOT_WAVES = 5
LL_ALGO_ONESHOT_SENTINEL, LL_ALGO_TWOSHOT_SENTINEL, LL_ALGO_TWOSHOT_SENTINEL_OUT = 6, 7, 8
LL_ALGO_TWOSHOT_ATOMIC = 9
LL_ALGO_TWOSHOT_WAVES, LL_ALGO_TWOSHOT_SENTINEL_WAVES, LL_ALGO_ONESHOT_SENTINEL_WAVES = 10, 11, 12
LL_ALGO_ONESHOT_LINE_WAVES, LL_ALGO_TWOSHOT_LINE_WAVES = 13, 14
LL_PROTO_AUTO, LL_PROTO_PACKET8, LL_PROTO_LINE128, LL_PROTO_SENTINEL = 0, 1, 2, 3
LL_FMT_PACKET8, LL_FMT_LINE128, LL_FMT_SENTINEL, LL_FMT_ATOMIC = 1, 2, 4, 8
LL_OPT_AUTO_SENTINEL, LL_OPT_NO_LINES = 0x1, 0x2
LL_STATIC_SCRATCH_BYTES = 64 << 20

LL_OK = 0
LL_ERR_INVALID = -1
LL_ERR_UNSUPPORTED = -2
LL_ERR_SCRATCH = -3
LL_ERR_HIP = -4
LL_ERR_TIMEOUT = -5

ALGOS = {
    "auto": LL_ALGO_AUTO, "oneshot": LL_ALGO_ONESHOT, "twoshot": LL_ALGO_TWOSHOT,
    "twoshot_line": LL_ALGO_TWOSHOT_LINE, "oneshot_line": LL_ALGO_ONESHOT_LINE,
    "oneshot_waves": LL_ALGO_ONESHOT_WAVES,
    "oneshot_sentinel": LL_ALGO_ONESHOT_SENTINEL, "twoshot_sentinel": LL_ALGO_TWOSHOT_SENTINEL,
    "twoshot_sentinel_out": LL_ALGO_TWOSHOT_SENTINEL_OUT, "twoshot_atomic": LL_ALGO_TWOSHOT_ATOMIC,
    "twoshot_waves": LL_ALGO_TWOSHOT_WAVES, "twoshot_sentinel_waves": LL_ALGO_TWOSHOT_SENTINEL_WAVES,
    "oneshot_sentinel_waves": LL_ALGO_ONESHOT_SENTINEL_WAVES,
    "oneshot_line_waves": LL_ALGO_ONESHOT_LINE_WAVES, "twoshot_line_waves": LL_ALGO_TWOSHOT_LINE_WAVES,
}
PROTOS = {"auto": LL_PROTO_AUTO, "packet8": LL_PROTO_PACKET8, "line128": LL_PROTO_LINE128,
          "sentinel": LL_PROTO_SENTINEL}
DTYPES = {"f32": LL_F32, "bf16": LL_BF16}

_vp, _sz, _i, _u32, _u64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64


class LLTuning(ctypes.Structure):
    """struct ll_tuning (include/lltune.h)."""
    _fields_ = [("size", _u32), ("workgroups_per_rank", _i), ("threads", _i), ("wave_units", _i),
                ("wave_kernels", _i), ("pipeline_lag", _i), ("first_wait", _i), ("poll_gap", _i),
                ("mute_rank", _i), ("clear_slots", _i), ("stamps", _vp), ("phases", _vp), ("grid_out", _vp),
                ("threads_out", _vp)]


class LLOptions(ctypes.Structure):
    """ll_options (include/llcoll.h)."""
    _fields_ = [("size", _u32), ("flags", _u32), ("poll_timeout", _u64), ("tuning", _vp)]


_OPT = ctypes.POINTER(LLOptions)

# name -> (restype, argtypes)
_SIGS = {
    "ll_options_init": (_i, [_OPT]),
    "ll_tuning_init": (_i, [ctypes.POINTER(LLTuning)]),
    "ll_slice_bytes": (_i, [_sz, _i, _i, _i, ctypes.POINTER(_sz)]),
    "ll_input_capacity": (_i, [_sz, _i, ctypes.POINTER(_sz)]),
    "ll_slice_layout": (_i, [_sz, _i, ctypes.POINTER(_sz)]),
    "ll_init": (_i, [_vp, _sz, _i, _vp]),
    "ll_fill_sentinel": (_i, [_vp, _sz, _i, _i, _vp]),
    "ll_allreduce": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp]),
    "ll_allreduce_algo": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp, _i]),
    "ll_allreduce_ex": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp, _i, _OPT]),
    "ll_auto_algo": (_i, [_sz, _i, _i, _sz, _OPT, ctypes.POINTER(_i)]),
    "ll_reduce_scatter": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp]),
    "ll_reduce_scatter_ex": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp, _i, _OPT]),
    "ll_allgather": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _vp]),
    "ll_allgather_ex": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _vp, _i, _OPT]),
    "ll_broadcast": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _u32, _vp, _i, _OPT]),
    "ll_reduce": (_i, [_vp, _sz, _vp, _sz, _i, _i, _i, _i, _u32, _vp, _i, _OPT]),
    "ll_scratch_bytes": (_i, [_sz, _i, ctypes.POINTER(_sz)]),
    "ll_scratch_iter_bytes": (_i, [_sz, _i, ctypes.POINTER(_sz)]),
    "ll_scratch_init": (_i, [_vp, _sz, _i, _vp]),
    "ll_allreduce_buffered": (_i, [_vp, _vp, _sz, _i, _i, _i, _vp, _sz, _u32, _vp, _i, _OPT, ctypes.POINTER(_u32)]),
    "ll_allreduce_static": (_i, [_vp, _vp, _sz, _i, _i, _i, _vp, _i, ctypes.POINTER(_u32)]),
    "ll_check": (_i, [_vp]),
    "ll_last_timeout": (_i, [ctypes.POINTER(_i), ctypes.POINTER(_u32), ctypes.POINTER(_u32)]),
    "ll_strerror": (ctypes.c_char_p, [_i]),
    "ll_buffered_plan": (_i, [_sz, _i, _i, _sz, ctypes.POINTER(_u32), ctypes.POINTER(_sz)]),
    "ll_iteration_span": (_i, [_sz, _sz, _u32, _i, _i, ctypes.POINTER(ctypes.c_int64)]),
    "ll_probe_empty": (_i, [_i, _i, _vp, _vp]),
    "ll_probe_floor": (_i, [_vp, _u64, _u64, _vp, _i, _i, _vp, _vp]),
    "ll_probe_chase": (_i, [_vp, _u64, _u64, _i, _vp, _vp]),
    "ll_probe_fence_l2": (_i, [_vp, _i, _vp, _vp]),
    "ll_probe_pingpong": (_i, [_vp, _i, _i, _i, _u64, _vp, _vp]),
    "ll_probe_spin": (_i, [_u64, _vp]),
    "ll_bench_allreduce": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _i, _i, _OPT, _vp, _i, _vp]),
    "ll_bench_reduce_scatter": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _i, _i, _OPT, _vp, _i, _vp]),
    "ll_bench_allgather": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _i, _i, _OPT, _vp, _i, _vp]),
    "ll_bench_rooted": (_i, [_i, _vp, _sz, _vp, _sz, _i, _i, _i, _u32, _i, _i, _OPT, _vp, _i, _vp]),
    "ll_bench_floor": (_i, [_vp, _u64, _u64, _u64, _vp, _i, _i, _i, _vp, _i, _vp]),
    "ll_bench_empty": (_i, [_i, _i, _i, _vp, _i, _vp]),
    "ll_bench_exchange": (_i, [_vp, _sz, _vp, _sz, _i, _i, _u32, _i, _vp, _i, ctypes.POINTER(_i), _vp]),
    "ll_probe_xcd": (_i, [_vp, _i, _i, _vp]),
    "ll_probe_litmus": (_i, [_vp, _sz, _i, _i, _i, _i, _i, _vp, _vp]),
    "ll_probe_stream": (_i, [_vp, _vp, _sz, _i, _i, _i, _vp]),
}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"llcoll HIP library not built ({LIB_PATH}); run __graft_entry__.build()")
# torch ships its own HIP runtime and loads it from its own directory.  Load
# torch first so that the library's dependency on libamdhip64.so.7 resolves to
# that same, already loaded runtime; loading the library first would put two
# HIP runtimes into one process.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


class LLError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__(f"{where}: {ll_strerror(status)} ({status})" if where else f"{ll_strerror(status)} ({status})")


def check(status: int, where: str = "") -> int:
    if status != LL_OK:
        raise LLError(status, where)
    return status


def exported_symbols():
    return list(_SIGS)


def library():
    return _lib


_TUNING_FIELDS = ("workgroups_per_rank", "threads", "wave_units", "wave_kernels", "pipeline_lag", "first_wait",
                  "poll_gap", "mute_rank", "clear_slots", "stamps", "phases")


class Options:
    """One call's ll_options, filled by ll_options_init, with an ll_tuning
    attached when any tuning field is given (or report=True, which also
    collects the launch shape in .grid / .threads after the call).  Pass the
    object itself to the wrappers below; None stands for NULL (defaults)."""

    def __init__(self, flags: int = 0, poll_timeout: int = 0, report: bool = False, **tuning):
        unknown = set(tuning) - set(_TUNING_FIELDS)
        if unknown:
            raise TypeError(f"unknown tuning fields {sorted(unknown)}")
        self.o = LLOptions()
        check(_lib.ll_options_init(ctypes.byref(self.o)), "ll_options_init")
        self.o.flags = flags
        self.o.poll_timeout = poll_timeout
        self._grid, self._threads = ctypes.c_int(0), ctypes.c_int(0)
        self.t = None
        if tuning or report:
            self.t = LLTuning()
            check(_lib.ll_tuning_init(ctypes.byref(self.t)), "ll_tuning_init")
            for k, v in tuning.items():
                setattr(self.t, k, v)
            self.t.grid_out = ctypes.addressof(self._grid)
            self.t.threads_out = ctypes.addressof(self._threads)
            self.o.tuning = ctypes.addressof(self.t)

    @property
    def ref(self):
        return ctypes.byref(self.o)

    @property
    def grid(self) -> int:
        return self._grid.value

    @property
    def threads(self) -> int:
        return self._threads.value


def _ref(opt):
    return opt.ref if opt is not None else None


# ---------------------------------------------------------------- C entry points
def ll_slice_bytes(count: int, dt: int, nranks: int, algo: int = LL_ALGO_AUTO):
    out = ctypes.c_size_t(0)
    st = _lib.ll_slice_bytes(count, dt, nranks, algo, ctypes.byref(out))
    return st, out.value


def ll_input_capacity(rank_stride: int, nranks: int):
    out = ctypes.c_size_t(0)
    st = _lib.ll_input_capacity(rank_stride, nranks, ctypes.byref(out))
    return st, out.value


def ll_slice_layout(rank_stride: int, nranks: int):
    """(status, [input, packet8 area, line area, atomic area, sentinel area, end]) byte offsets."""
    out = (ctypes.c_size_t * 6)()
    st = _lib.ll_slice_layout(rank_stride, nranks, out)
    return st, list(out)


def ll_init(sym_base, rank_stride, nranks, stream):
    return _lib.ll_init(sym_base, rank_stride, nranks, stream)


def ll_allreduce(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream):
    return _lib.ll_allreduce(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream)


def ll_allreduce_algo(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, algo):
    return _lib.ll_allreduce_algo(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, algo)


def ll_allreduce_ex(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, algo, opt=None):
    return _lib.ll_allreduce_ex(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, algo, _ref(opt))


def ll_auto_algo(count: int, dt: int, nranks: int, rank_stride: int = 0, opt=None):
    out = ctypes.c_int(-1)
    st = _lib.ll_auto_algo(count, dt, nranks, rank_stride, _ref(opt), ctypes.byref(out))
    return st, out.value


def ll_reduce_scatter(sym_base, rank_stride, out, recvcount, dt, op, nranks, epoch, stream):
    return _lib.ll_reduce_scatter(sym_base, rank_stride, out, recvcount, dt, op, nranks, epoch, stream)


def ll_reduce_scatter_ex(sym_base, rank_stride, out, recvcount, dt, op, nranks, epoch, stream, proto, opt=None):
    return _lib.ll_reduce_scatter_ex(sym_base, rank_stride, out, recvcount, dt, op, nranks, epoch, stream, proto,
                                     _ref(opt))


def ll_allgather(sym_base, rank_stride, out, sendcount, dt, nranks, epoch, stream):
    return _lib.ll_allgather(sym_base, rank_stride, out, sendcount, dt, nranks, epoch, stream)


def ll_allgather_ex(sym_base, rank_stride, out, sendcount, dt, nranks, epoch, stream, proto, opt=None):
    return _lib.ll_allgather_ex(sym_base, rank_stride, out, sendcount, dt, nranks, epoch, stream, proto, _ref(opt))


def ll_broadcast(sym_base, rank_stride, out, count, dt, root, nranks, epoch, stream, proto, opt=None):
    return _lib.ll_broadcast(sym_base, rank_stride, out, count, dt, root, nranks, epoch, stream, proto, _ref(opt))


def ll_reduce(sym_base, rank_stride, out, count, dt, op, root, nranks, epoch, stream, proto, opt=None):
    return _lib.ll_reduce(sym_base, rank_stride, out, count, dt, op, root, nranks, epoch, stream, proto, _ref(opt))


def ll_fill_sentinel(out, count, dt, nranks, stream):
    return _lib.ll_fill_sentinel(out, count, dt, nranks, stream)


def ll_scratch_bytes(iter_bytes: int, nranks: int):
    out = ctypes.c_size_t(0)
    st = _lib.ll_scratch_bytes(iter_bytes, nranks, ctypes.byref(out))
    return st, out.value


def ll_scratch_iter_bytes(scratch_stride: int, nranks: int):
    out = ctypes.c_size_t(0)
    st = _lib.ll_scratch_iter_bytes(scratch_stride, nranks, ctypes.byref(out))
    return st, out.value


def ll_scratch_init(scratch_base, scratch_stride, nranks, stream):
    return _lib.ll_scratch_init(scratch_base, scratch_stride, nranks, stream)


def ll_allreduce_buffered(inp, out, count, dt, op, nranks, scratch_base, scratch_stride, epoch, stream, algo,
                          opt=None):
    """(status, epochs used)."""
    used = ctypes.c_uint32(0)
    st = _lib.ll_allreduce_buffered(inp, out, count, dt, op, nranks, scratch_base, scratch_stride, epoch, stream,
                                    algo, _ref(opt), ctypes.byref(used))
    return st, used.value


def ll_allreduce_static(inp, out, count, dt, op, nranks, stream, algo):
    """(status, epochs used): AllReduce through the library's own scratch (no allocation)."""
    used = ctypes.c_uint32(0)
    st = _lib.ll_allreduce_static(inp, out, count, dt, op, nranks, stream, algo, ctypes.byref(used))
    return st, used.value


def ll_check(stream):
    return _lib.ll_check(stream)


def ll_last_timeout():
    r, m, e = ctypes.c_int(0), ctypes.c_uint32(0), ctypes.c_uint32(0)
    _lib.ll_last_timeout(ctypes.byref(r), ctypes.byref(m), ctypes.byref(e))
    return r.value, m.value, e.value


def ll_strerror(status: int) -> str:
    return _lib.ll_strerror(status).decode()


def ll_buffered_plan(count: int, dt: int, nranks: int, scratch_stride: int):
    """(status, iterations, elements per iteration)."""
    k, ic = ctypes.c_uint32(0), ctypes.c_size_t(0)
    st = _lib.ll_buffered_plan(count, dt, nranks, scratch_stride, ctypes.byref(k), ctypes.byref(ic))
    return st, k.value, ic.value


def ll_iteration_span(count: int, iter_count: int, it: int, nranks: int, dt: int):
    """(status, (first element, elements, two-shot chunk))."""
    out = (ctypes.c_int64 * 3)()
    st = _lib.ll_iteration_span(count, iter_count, it, nranks, dt, out)
    return st, tuple(out)


# ---------------------------------------------------------------- probes and benchmark loops
def ll_probe_empty(grid, threads, stamps, stream):
    return _lib.ll_probe_empty(grid, threads, stamps, stream)


def ll_probe_floor(chase, chase_len, start, sink, grid, threads, stamps, stream):
    return _lib.ll_probe_floor(chase, chase_len, start, sink, grid, threads, stamps, stream)


def ll_probe_chase(chase, chase_len, start, steps, out3, stream):
    return _lib.ll_probe_chase(chase, chase_len, start, steps, out3, stream)


def ll_probe_fence_l2(buf4k, iters, out7, stream):
    return _lib.ll_probe_fence_l2(buf4k, iters, out7, stream)


def ll_probe_pingpong(flags8k, rounds, grid, peer, limit_ticks, out3, stream):
    return _lib.ll_probe_pingpong(flags8k, rounds, grid, peer, limit_ticks, out3, stream)


def ll_probe_spin(ticks, stream):
    return _lib.ll_probe_spin(ticks, stream)


def ll_bench_allreduce(sym_base, rank_stride, out, count, dt, nranks, first_epoch, calls, algo, opt, stamps,
                       stamp_stride, stream):
    return _lib.ll_bench_allreduce(sym_base, rank_stride, out, count, dt, nranks, first_epoch, calls, algo, _ref(opt),
                                   stamps, stamp_stride, stream)


def ll_bench_reduce_scatter(sym_base, rank_stride, out, recvcount, dt, nranks, first_epoch, calls, proto, opt, stamps,
                            stamp_stride, stream):
    return _lib.ll_bench_reduce_scatter(sym_base, rank_stride, out, recvcount, dt, nranks, first_epoch, calls, proto,
                                        _ref(opt), stamps, stamp_stride, stream)


def ll_bench_allgather(sym_base, rank_stride, out, sendcount, dt, nranks, first_epoch, calls, proto, opt, stamps,
                       stamp_stride, stream):
    return _lib.ll_bench_allgather(sym_base, rank_stride, out, sendcount, dt, nranks, first_epoch, calls, proto,
                                   _ref(opt), stamps, stamp_stride, stream)


def ll_bench_rooted(kind, sym_base, rank_stride, out, count, dt, root, nranks, first_epoch, calls, proto, opt,
                    stamps, stamp_stride, stream):
    return _lib.ll_bench_rooted(kind, sym_base, rank_stride, out, count, dt, root, nranks, first_epoch, calls, proto,
                                _ref(opt), stamps, stamp_stride, stream)


def ll_bench_floor(chase, chase_len, first_line, line_step, sink, grid, threads, calls, stamps, stamp_stride,
                   stream):
    return _lib.ll_bench_floor(chase, chase_len, first_line, line_step, sink, grid, threads, calls, stamps,
                               stamp_stride, stream)


def ll_bench_empty(grid, threads, calls, stamps, stamp_stride, stream):
    return _lib.ll_bench_empty(grid, threads, calls, stamps, stamp_stride, stream)


def ll_bench_exchange(sym_base, rank_stride, out, count, dt, nranks, first_epoch, calls, stamps, stamp_stride,
                      stream):
    """(status, grid)."""
    g = ctypes.c_int(0)
    st = _lib.ll_bench_exchange(sym_base, rank_stride, out, count, dt, nranks, first_epoch, calls, stamps,
                                stamp_stride, ctypes.byref(g), stream)
    return st, g.value


def ll_probe_xcd(ids, grid, threads, stream):
    return _lib.ll_probe_xcd(ids, grid, threads, stream)


def ll_probe_stream(src, dst, nbytes, mode, grid, threads, stream):
    return _lib.ll_probe_stream(src, dst, nbytes, mode, grid, threads, stream)


def ll_probe_litmus(buf, buf_bytes, grid, lines, iters, reads, layout, counts4, stream):
    return _lib.ll_probe_litmus(buf, buf_bytes, grid, lines, iters, reads, layout, counts4, stream)
