"""Device memory plumbing for the collectives (torch allocations only).

``SymRegion`` holds one symmetric allocation of P rank slices plus an output
buffer, keeps the caller-owned epoch counter, and calls the C ABI through
``llcoll``.  torch provides memory, copies and the stream; no arithmetic of
the collectives happens here.
"""
from __future__ import annotations

import numpy as np
import torch

from . import llcoll as ll

_ALIGN = 256


def _aligned(nbytes: int, device) -> tuple[torch.Tensor, int]:
    """A uint8 tensor of at least nbytes whose returned address is 256-byte aligned."""
    t = torch.empty(nbytes + _ALIGN, dtype=torch.uint8, device=device)
    base = t.data_ptr()
    pad = (-base) % _ALIGN
    return t, pad


def _np_to_u8(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.uint8).reshape(-1))


class SymRegion:
    """P slices of ``rank_stride`` bytes in one allocation, plus ``out``.

    ``max_count`` elements of ``dtype`` ("f32" / "bf16") is the largest
    per-rank input the region must hold; ``sized_for`` names the algorithm
    the region is sized for ("auto": every algorithm and packet format);
    ``out_elems`` sizes the output buffer (defaults to what an AllGather of
    max_count needs).  ``opt`` (an llcoll.Options or None) is passed to every
    call that takes options unless the call names its own.
    """

    def __init__(self, nranks: int, max_count: int, dtype: str, device="cuda:0", out_elems: int | None = None,
                 rank_stride: int | None = None, sized_for: str = "auto", opt=None):
        self.nranks = nranks
        self.dtype = dtype
        self.dt = ll.DTYPES[dtype]
        self.esize = 4 if dtype == "f32" else 2
        self.opt = opt
        st, need = ll.ll_slice_bytes(max_count, self.dt, nranks, ll.ALGOS[sized_for])
        ll.check(st, "ll_slice_bytes")
        self.rank_stride = rank_stride if rank_stride is not None else need
        self.device = torch.device(device)
        self._sym, pad = _aligned(nranks * self.rank_stride, self.device)
        self.sym = self._sym[pad:pad + nranks * self.rank_stride]
        if out_elems is None:
            out_elems = nranks * nranks * max(max_count, 1)
        self._out, opad = _aligned(out_elems * self.esize, self.device)
        self.out = self._out[opad:opad + out_elems * self.esize]
        self.epoch = 0

    # -- addresses
    @property
    def base(self) -> int:
        return self.sym.data_ptr()

    @property
    def out_ptr(self) -> int:
        return self.out.data_ptr()

    @staticmethod
    def stream_handle(stream=None) -> int:
        s = stream if stream is not None else torch.cuda.current_stream()
        return s.cuda_stream

    # -- set-up
    def init(self, stream=None) -> None:
        ll.check(ll.ll_init(self.base, self.rank_stride, self.nranks, self.stream_handle(stream)), "ll_init")
        self.epoch = 0

    def next_epoch(self) -> int:
        if self.epoch >= 0xFFFFFFFF:
            raise RuntimeError("epoch space exhausted: call init() first")
        self.epoch += 1
        return self.epoch

    def write_inputs(self, bits: np.ndarray) -> None:
        """Copy rank r's raw element bits (row r of a [P, n] array) to offset 0 of slice r."""
        assert bits.shape[0] == self.nranks
        row_bytes = bits.shape[1] * bits.dtype.itemsize
        host = _np_to_u8(bits).reshape(self.nranks, row_bytes)
        view = self.sym.view(self.nranks, self.rank_stride)[:, :row_bytes]
        view.copy_(host.to(self.device, non_blocking=False))

    def write_inputs_device(self, rows: torch.Tensor) -> None:
        """Same as write_inputs for a [P, n_bytes] uint8 tensor already on the device."""
        view = self.sym.view(self.nranks, self.rank_stride)[:, :rows.shape[1]]
        view.copy_(rows)

    def read_area(self, area: int) -> np.ndarray:
        """Raw uint32 words of layout area `area` (1 = 8-byte packets, 2 =
        lines, 3 = atomic accumulators, 4 = sentinel) of every slice, shape
        [P, area_bytes / 4]."""
        st, offs = ll.ll_slice_layout(self.rank_stride, self.nranks)
        ll.check(st, "ll_slice_layout")
        lo, hi = offs[area], offs[area + 1]
        v = self.sym.view(self.nranks, self.rank_stride)[:, lo:hi]
        return v.cpu().numpy().copy().view(np.uint32)

    def read_out(self, nelems_total: int, np_dtype) -> np.ndarray:
        nbytes = nelems_total * np.dtype(np_dtype).itemsize
        return self.out[:nbytes].cpu().numpy().view(np_dtype).copy()

    # -- collectives (one launch each, on the given stream)
    def _opt(self, opt):
        return self.opt if opt is None else opt

    def broadcast(self, count: int, root: int, proto: str = "auto", stream=None, epoch: int | None = None,
                  opt=None) -> int:
        e = self.next_epoch() if epoch is None else epoch
        return ll.ll_broadcast(self.base, self.rank_stride, self.out_ptr, count, self.dt, root, self.nranks, e,
                               self.stream_handle(stream), ll.PROTOS[proto], self._opt(opt))

    def reduce(self, count: int, root: int, proto: str = "auto", stream=None, epoch: int | None = None,
               opt=None) -> int:
        e = self.next_epoch() if epoch is None else epoch
        return ll.ll_reduce(self.base, self.rank_stride, self.out_ptr, count, self.dt, ll.LL_SUM, root, self.nranks,
                            e, self.stream_handle(stream), ll.PROTOS[proto], self._opt(opt))

    def fill_out_sentinel(self, count: int, stream=None) -> int:
        """Fill the P outputs of `count` elements with the sentinel."""
        return ll.ll_fill_sentinel(self.out_ptr, count, self.dt, self.nranks, self.stream_handle(stream))

    def allreduce(self, count: int, algo: str = "auto", stream=None, epoch: int | None = None, opt=None) -> int:
        """One AllReduce.  For "twoshot_sentinel_out" and "twoshot_atomic" the
        outputs are first refilled with the sentinel (their precondition), on
        the same stream."""
        e = self.next_epoch() if epoch is None else epoch
        if algo in ("twoshot_sentinel_out", "twoshot_atomic") and count > 0:
            st = self.fill_out_sentinel(count, stream)
            if st != ll.LL_OK:
                return st
        return ll.ll_allreduce_ex(self.base, self.rank_stride, self.out_ptr, count, self.dt, ll.LL_SUM,
                                  self.nranks, e, self.stream_handle(stream), ll.ALGOS[algo], self._opt(opt))

    def reduce_scatter(self, recvcount: int, proto: str = "auto", stream=None, epoch: int | None = None,
                       opt=None) -> int:
        e = self.next_epoch() if epoch is None else epoch
        return ll.ll_reduce_scatter_ex(self.base, self.rank_stride, self.out_ptr, recvcount, self.dt, ll.LL_SUM,
                                       self.nranks, e, self.stream_handle(stream), ll.PROTOS[proto], self._opt(opt))

    def allgather(self, sendcount: int, proto: str = "auto", stream=None, epoch: int | None = None,
                  opt=None) -> int:
        e = self.next_epoch() if epoch is None else epoch
        return ll.ll_allgather_ex(self.base, self.rank_stride, self.out_ptr, sendcount, self.dt, self.nranks, e,
                                  self.stream_handle(stream), ll.PROTOS[proto], self._opt(opt))


class ScratchRegion:
    """Bounded scratch for multi-iteration AllReduce: P scratch slices of
    ``scratch_stride`` bytes (sized for iterations of ``iter_bytes`` bytes
    per rank), plus separate input and output buffers of P x ``max_count``
    elements.  ``in_place=True`` makes the output the input buffer."""

    def __init__(self, nranks: int, max_count: int, dtype: str, iter_bytes: int, device="cuda:0",
                 in_place: bool = False, opt=None):
        self.nranks = nranks
        self.opt = opt
        self.dtype = dtype
        self.dt = ll.DTYPES[dtype]
        self.esize = 4 if dtype == "f32" else 2
        st, self.scratch_stride = ll.ll_scratch_bytes(iter_bytes, nranks)
        ll.check(st, "ll_scratch_bytes")
        st, self.iter_bytes = ll.ll_scratch_iter_bytes(self.scratch_stride, nranks)
        ll.check(st, "ll_scratch_iter_bytes")
        self.device = torch.device(device)
        self._scr, pad = _aligned(nranks * self.scratch_stride, self.device)
        self.scratch = self._scr[pad:pad + nranks * self.scratch_stride]
        nbytes = nranks * max(max_count, 1) * self.esize
        self._in, ipad = _aligned(nbytes, self.device)
        self.inp = self._in[ipad:ipad + nbytes]
        if in_place:
            self.out = self.inp
        else:
            self._out, opad = _aligned(nbytes, self.device)
            self.out = self._out[opad:opad + nbytes]
        self.epoch = 0

    def init(self, stream=None) -> None:
        ll.check(ll.ll_scratch_init(self.scratch.data_ptr(), self.scratch_stride, self.nranks,
                                    SymRegion.stream_handle(stream)), "ll_scratch_init")
        self.epoch = 0

    def write_inputs(self, bits: np.ndarray) -> None:
        """Rank r's raw element bits (row r of a [P, n] array) at in + r*n*esize."""
        assert bits.shape[0] == self.nranks
        host = _np_to_u8(bits)
        self.inp[:host.numel()].copy_(host.to(self.device, non_blocking=False))

    def read_out(self, nelems_total: int, np_dtype) -> np.ndarray:
        nbytes = nelems_total * np.dtype(np_dtype).itemsize
        return self.out[:nbytes].cpu().numpy().view(np_dtype).copy()

    def allreduce(self, count: int, algo: str = "auto", stream=None, opt=None) -> int:
        """One call; advances the epoch by the iterations it used.  For
        "twoshot_sentinel_out" the outputs are refilled with the sentinel first."""
        s = SymRegion.stream_handle(stream)
        if algo == "twoshot_sentinel_out" and count > 0:
            st = ll.ll_fill_sentinel(self.out.data_ptr(), count, self.dt, self.nranks, s)
            if st != ll.LL_OK:
                return st
        st, used = ll.ll_allreduce_buffered(self.inp.data_ptr(), self.out.data_ptr(), count, self.dt, ll.LL_SUM,
                                            self.nranks, self.scratch.data_ptr(), self.scratch_stride,
                                            self.epoch + 1, s, ll.ALGOS[algo], self.opt if opt is None else opt)
        if st == ll.LL_OK:
            self.epoch += used
        self.last_iters = used
        return st
