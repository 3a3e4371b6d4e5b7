"""GPU tests of slot clearing: the reader of a flagged packet slot stores
zeros back into it after reading it (ll_tuning.clear_slots; by default on for
the one-shot wave kernels and for small two-shot and RS / AG wave calls).

- Results are bit-exact against the oracle with clearing forced on and off,
  for every wave kernel that clears, at several sizes and rank counts, over
  back-to-back calls on one region, and in bounded-scratch calls of many
  iterations (where a late zero store could erase a peer's refill of a
  sub-buffer if the iteration boundary did not wait for it).
- After a call with clearing, every dword of the slots read is zero; without
  it, their flags hold the call's epoch.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2607_16100_amd import workloads as wl  # noqa: E402

if torch.cuda.is_available():
    from paper_2607_16100_amd import llcoll as ll  # noqa: E402
    from paper_2607_16100_amd.region import ScratchRegion, SymRegion  # noqa: E402
else:  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

NP = {"f32": np.uint32, "bf16": np.uint16}
TEST_TIMEOUT_TICKS = 20_000_000  # 200 ms per flag wait
ALWAYS, NEVER = 1, 2
WAVE_ALGOS = ["oneshot_waves", "oneshot_line_waves", "twoshot_waves", "twoshot_line_waves"]


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def stream():
    return torch.cuda.current_stream().cuda_stream


def check_ok(st, what):
    assert st == ll.LL_OK, f"{what}: {ll.ll_strerror(st)}"
    st2 = ll.ll_check(stream())
    assert st2 == ll.LL_OK, f"{what}: ll_check says {ll.ll_strerror(st2)}"


def assert_bits_equal(got, want, what):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        r, i = bad[0]
        raise AssertionError(f"{what}: {len(bad)} elements differ; first at rank {r} index {i}: "
                             f"got {int(got[r, i]):#x} want {int(want[r, i]):#x}")


def opts(**kw):
    kw.setdefault("poll_timeout", TEST_TIMEOUT_TICKS)
    return ll.Options(**kw)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [3, 8])
def test_clearing_on_and_off_is_exact(dtype, p):
    """Every clearing wave kernel, clearing forced on and off, ragged sizes
    from one element to past the size-based cut-off, two calls per case."""
    sizes = [1, 1000, 50_001, 300_007]
    reg = SymRegion(p, max(sizes), dtype)
    reg.init()
    for n in sizes:
        for algo in WAVE_ALGOS:
            if algo.startswith("oneshot") and n * (4 if dtype == "f32" else 2) > (1 << 20):
                continue
            for clear in (ALWAYS, NEVER):
                for call in range(2):
                    x = wl.uniform(p, n, dtype, seed=100 * call + n % 97)
                    say(f"clear={clear} {algo} P={p} n={n} {dtype} call {call}")
                    reg.write_inputs(x)
                    check_ok(reg.allreduce(n, algo, opt=opts(clear_slots=clear)), f"{algo} n={n}")
                    got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
                    assert_bits_equal(got, oracle.allreduce(x), f"{algo} P={p} n={n} clear={clear}")


@pytest.mark.parametrize("p", [3, 7, 8])
def test_clearing_between_bounded_scratch_iterations(p):
    """Bounded-scratch two-shot with one wave per peer in 4 KiB iterations
    (dozens of them), clearing forced on, in place and out of place, three
    calls in a row: a zero store that landed after a peer's refill of the
    same sub-buffer would lose a packet and time out."""
    dtype, n = "bf16", 40_001
    for in_place in (False, True):
        reg = ScratchRegion(p, n, dtype, iter_bytes=4096, in_place=in_place)
        reg.init()
        for algo in ("twoshot_waves", "twoshot_line_waves"):
            for call in range(3):
                x = wl.normal(p, n, dtype, seed=7 * call + p)
                say(f"buffered clear {algo} P={p} in_place={in_place} call {call}")
                reg.write_inputs(x)
                check_ok(reg.allreduce(n, algo, opt=opts(clear_slots=ALWAYS)), f"buffered {algo}")
                assert reg.last_iters > 10
                got = reg.read_out(p * n, np.uint16).reshape(p, n)
                assert_bits_equal(got, oracle.allreduce(x), f"buffered {algo} P={p} in_place={in_place}")


@pytest.mark.parametrize("proto", ["packet8", "line128"])
def test_clearing_in_reduce_scatter_and_allgather(proto):
    """The stand-alone wave kernels with clearing forced on and off."""
    p, m = 8, 7168
    total = p * m
    reg = SymRegion(p, total, "bf16", out_elems=p * total)
    reg.init()
    x = wl.normal(p, total, "bf16", seed=11)
    for clear in (ALWAYS, NEVER):
        reg.opt = opts(wave_kernels=2, clear_slots=clear)
        say(f"RS/AG clear={clear} {proto}")
        reg.write_inputs(x)
        check_ok(reg.reduce_scatter(m, proto), "reduce_scatter")
        got_rs = reg.read_out(p * m, np.uint16).reshape(p, m)
        assert_bits_equal(got_rs, oracle.reduce_scatter(x), f"RS {proto} clear={clear}")
        reg.write_inputs(got_rs)
        check_ok(reg.allgather(m, proto), "allgather")
        got_ag = reg.read_out(p * p * m, np.uint16).reshape(p, p * m)
        assert_bits_equal(got_ag, oracle.allgather(got_rs), f"AG {proto} clear={clear}")


@pytest.mark.parametrize("algo,area", [("oneshot_waves", 1), ("oneshot_line_waves", 2), ("twoshot_waves", 1),
                                       ("twoshot_line_waves", 2)])
def test_slots_read_hold_zeros_after_a_clearing_call(algo, area):
    """After a call with clearing every dword of the packet area is zero
    (every slot the call used was read and cleared); after a call without
    it, the flag dwords of the slots used hold the call's epoch."""
    p, n = 8, 8192
    reg = SymRegion(p, n, "bf16", sized_for=algo)
    reg.init()
    x = wl.normal(p, n, "bf16", seed=5)
    reg.write_inputs(x)
    say(f"slots after {algo} clear=never")
    e = reg.next_epoch()
    check_ok(reg.allreduce(n, algo, epoch=e, opt=opts(clear_slots=NEVER)), algo)
    words = reg.read_area(area)
    flags = words[:, 1::2] if area == 1 else words.reshape(p, -1, 16)[:, :, 15]
    assert (flags == e).any(axis=1).all(), "every rank received packets flagged with the epoch"
    assert np.isin(flags, (0, e)).all()
    say(f"slots after {algo} clear=always")
    check_ok(reg.allreduce(n, algo, opt=opts(clear_slots=ALWAYS)), algo)
    assert not reg.read_area(area).any(), "a slot read by the call still holds packet bytes"
    got = reg.read_out(p * n, np.uint16).reshape(p, n)
    assert_bits_equal(got, oracle.allreduce(x), f"{algo} after clearing")
