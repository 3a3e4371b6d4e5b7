"""GPU parity at the edges of the final rounding and of IEEE arithmetic, the
minimal-exchange probe, and per-stream status words.

Edge values go through every AllReduce algorithm, ReduceScatter and Reduce in
every packet format, AllGather and Broadcast (bit copies), and the
bounded-scratch path:

* binary32 sums just above bfloat16's largest finite value, where the one
  rounding to bfloat16 (round to nearest even) must give +-Inf, and just
  below, where it must not;
* a sum that is back in range after an intermediate value that only the
  binary32 accumulator holds (rounding once, at the end);
* binary32 overflow to +-Inf;
* +-Inf inputs and Inf - Inf;
* quiet and signalling NaN inputs.

Where the oracle's result is a NaN only NaN-ness is compared (payloads and
signs of NaNs are not specified); everything else is compared bit for bit.
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

AR_ALGOS = ["oneshot", "twoshot", "twoshot_line", "oneshot_line", "oneshot_waves", "oneshot_sentinel",
            "twoshot_sentinel", "twoshot_waves", "twoshot_sentinel_waves", "oneshot_sentinel_waves",
            "oneshot_line_waves", "twoshot_line_waves", "twoshot_sentinel_out", "auto"]
PROTOS = ["packet8", "line128", "sentinel", "auto"]
NP = {"f32": np.uint32, "bf16": np.uint16}
TEST_TIMEOUT_TICKS = 20_000_000

# Columns of rank values (bit patterns), the first entries at ranks 0, 1, 2
# and the rest zero; "last" puts the value at rank P-1 instead.
F32_COLS = [
    [0x7F7F0000, 0x7B000000],              # bf16 max + half its ulp: finite binary32 0x7F7F8000
    [0x7F7FFFFF, 0x7F7FFFFF],              # binary32 overflow -> +Inf
    [0xFF7FFFFF, 0xFF7FFFFF],              # -> -Inf
    [0x7F800000, 0x3F800000],              # +Inf + 1
    [0x3F800000, "last", 0xFF800000],      # 1 + ... + -Inf at the last rank
    [0x7F800000, 0xFF800000],              # Inf - Inf -> NaN
    [0x7FC00001, 0x3F800000],              # quiet NaN
    [0x3F800000, 0x7F800001],              # signalling NaN
    [0x7F7FFFFF, 0x7F7FFFFF, 0xFF800000],  # overflow, then -Inf -> NaN
    [0x7F7FFFFF, 0x7F7FFFFF, 0xFF7FFFFF],  # overflow is not undone: Inf - max = Inf
    [0x7E967699] * 8,                      # 1e38 at every rank: overflows from the 4th rank on
    [0x3F800000, 0xBF800000],              # exact cancellation: +0
]
BF16_COLS = [
    [0x7F7F, 0x7B00],          # 0x7F7F8000 in binary32: a tie, rounds to even = +Inf
    [0x7F7F, 0x7A80],          # 0x7F7F4000: below the tie, stays at bf16 max
    [0xFF7F, 0xFB00],          # -Inf
    [0x7F7F, 0x7B00, 0xFB00],  # back to bf16 max: rounded once, at the end
    [0x7F7E, 0x7B00],          # 0x7F7E8000: a tie, rounds to even = 0x7F7E
    [0x7F7E, 0x7B01],          # just above that tie: 0x7F7F
    [0x7F7F, 0x7F7F],          # binary32 overflow -> +Inf
    [0x7F80, 0x3F80],          # +Inf + 1
    [0x3F80, "last", 0xFF80],  # -Inf at the last rank
    [0x7F80, 0xFF80],          # Inf - Inf -> NaN
    [0x7FC1, 0x3F80],          # quiet NaN
    [0x3F80, 0x7F81],          # signalling NaN
    [0x7F7F] * 8,              # bf16 max at every rank: binary32 overflow from the 3rd rank on
]


def edge_inputs(p: int, dtype: str, repeat: int = 40) -> np.ndarray:
    cols = F32_COLS if dtype == "f32" else BF16_COLS
    x = np.zeros((p, len(cols)), dtype=NP[dtype])
    for j, c in enumerate(cols):
        if len(c) >= 2 and c[1] == "last":
            x[0, j], x[p - 1, j] = c[0], c[2]
            continue
        for r, v in enumerate(c[:p]):
            x[r, j] = v
    # several tiles with a ragged tail: 40 repeats of the columns plus 7
    return np.ascontiguousarray(np.concatenate([np.tile(x, (1, repeat)), x[:, :7]], axis=1))


def isnan_bits(v: np.ndarray) -> np.ndarray:
    if v.dtype == np.uint32:
        return ((v & 0x7F800000) == 0x7F800000) & ((v & 0x007FFFFF) != 0)
    return ((v & 0x7F80) == 0x7F80) & ((v & 0x007F) != 0)


def assert_same(got, want, what):
    """Bit-exact, except that a NaN expected is only checked for being a NaN."""
    nan = isnan_bits(want)
    bad = (isnan_bits(got) != nan) | (~nan & (got != want))
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} elements differ; first at {tuple(idx)}: "
                             f"got {int(got[tuple(idx)]):#x} want {int(want[tuple(idx)]):#x}")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def stream():
    return torch.cuda.current_stream().cuda_stream


def check_ok(st, what, s=None):
    s = stream() if s is None else s
    assert st == ll.LL_OK, f"{what}: {ll.ll_strerror(st)}"
    st2 = ll.ll_check(s)
    assert st2 == ll.LL_OK, f"{what}: ll_check says {ll.ll_strerror(st2)}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [3, 6, 7, 8])
def test_edge_values_every_allreduce_algorithm(dtype, p):
    x = edge_inputs(p, dtype)
    n = x.shape[1]
    want = oracle.allreduce(x)
    assert isnan_bits(want).any() and (want == (0x7F800000 if dtype == "f32" else 0x7F80)).any()
    reg = SymRegion(p, n + 16, dtype)
    reg.init()
    for algo in AR_ALGOS:
        m = n if algo != "twoshot_sentinel_out" else n - n % (16 // x.itemsize)  # whole 16-byte rows
        xx = np.ascontiguousarray(x[:, :m])
        say(f"edge allreduce {algo} P={p} {dtype} n={m}")
        reg.write_inputs(xx)
        check_ok(reg.allreduce(m, algo), f"edge {algo}")
        got = reg.read_out(p * m, NP[dtype]).reshape(p, m)
        assert_same(got, want[:, :m], f"edge {algo} P={p} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [3, 7, 8])
def test_edge_values_rs_ag_broadcast_reduce(dtype, p):
    x = edge_inputs(p, dtype, repeat=10 * p)
    m = x.shape[1] // p
    x = np.ascontiguousarray(x[:, :p * m])
    reg = SymRegion(p, p * m, dtype, out_elems=p * p * m)
    reg.init()
    for proto in PROTOS:
        say(f"edge RS/AG/bcast/reduce {proto} P={p} {dtype}")
        reg.write_inputs(x)
        check_ok(reg.reduce_scatter(m, proto), "rs")
        assert_same(reg.read_out(p * m, NP[dtype]).reshape(p, m), oracle.reduce_scatter(x), f"RS {proto}")
        ag_in = np.ascontiguousarray(x[:, :m])
        reg.write_inputs(ag_in)
        check_ok(reg.allgather(m, proto), "ag")
        got = reg.read_out(p * p * m, NP[dtype]).reshape(p, p * m)
        assert np.array_equal(got, oracle.allgather(ag_in)), f"AG {proto}: not a bit copy"
        n = p * m
        reg.write_inputs(x)
        for root in (0, p - 1):
            check_ok(reg.broadcast(n, root, proto), "broadcast")
            got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
            assert np.array_equal(got, oracle.broadcast(x, root)), f"broadcast {proto} root {root}: not a bit copy"
            check_ok(reg.reduce(n, root, proto), "reduce")
            got = reg.read_out(n, NP[dtype]).reshape(1, n)
            assert_same(got, oracle.reduce(x, root).reshape(1, n), f"reduce {proto} root {root}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_values_bounded_scratch(dtype):
    p = 6
    x = edge_inputs(p, dtype, repeat=120)
    n = x.shape[1]
    reg = ScratchRegion(p, n, dtype, iter_bytes=1024)
    reg.init()
    want = oracle.allreduce(x)
    for algo in ("auto", "twoshot", "twoshot_line", "twoshot_sentinel", "twoshot_waves", "twoshot_line_waves",
                 "oneshot", "oneshot_sentinel"):
        say(f"edge buffered {algo} {dtype} n={n}")
        reg.write_inputs(x)
        check_ok(reg.allreduce(n, algo), f"edge buffered {algo}")
        assert reg.last_iters > 1
        assert_same(reg.read_out(p * n, NP[dtype]).reshape(p, n), want, f"edge buffered {algo} {dtype}")


# ---------------------------------------------------------------- exchange probe
@pytest.mark.parametrize("p,n", [(8, 8192), (4, 1024), (7, 4096 + 4)])
def test_exchange_probe_moves_the_inputs(p, n):
    """The minimal-exchange probe (no sum): after a few back-to-back calls no
    wait has timed out, and every element of every rank's output is that
    element of one of the P inputs."""
    x = wl.normal(p, n, "bf16", seed=11)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    reg.write_inputs(x)
    s = reg.stream_handle()
    say(f"exchange probe P={p} n={n}")
    st, grid = ll.ll_bench_exchange(reg.base, reg.rank_stride, reg.out_ptr, n, ll.LL_BF16, p, reg.epoch + 1, 20, 0,
                                    0, s)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    assert grid == p * -(-n * 2 // 512)  # one tile of 64 8-byte units per workgroup
    reg.epoch += 20
    assert ll.ll_check(s) == ll.LL_OK
    got = reg.read_out(p * n, np.uint16).reshape(p, n)
    for r in range(p):
        assert (got[r][None, :] == x).any(axis=0).all(), f"rank {r}: an output element is no rank's input"
    # the collective still works on the same region afterwards (epochs kept increasing)
    check_ok(reg.allreduce(n, "oneshot_waves"), "allreduce after the probe")
    assert np.array_equal(reg.read_out(p * n, np.uint16).reshape(p, n), oracle.allreduce(x))


# ---------------------------------------------------------------- per-stream status
def test_timeouts_are_reported_on_their_own_stream_only():
    """Two regions on two streams; the calls on region A have a muted rank and
    time out, those on region B do not.  ll_check of B's stream reports
    success and ll_check of A's stream the timeout, whatever order they are
    checked in; then both streams are clean again."""
    p, n = 8, 4096
    x = wl.normal(p, n, "bf16", seed=3)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    ra, rb = SymRegion(p, n, "bf16"), SymRegion(p, n, "bf16")
    for reg, s in ((ra, sa), (rb, sb)):
        reg.init(s)
        with torch.cuda.stream(s):
            reg.write_inputs(x)
    torch.cuda.synchronize()
    for order in ("b_first", "a_first"):
        say(f"muted call on stream A ({order})")
        muted = ll.Options(poll_timeout=200_000, mute_rank=5)  # 2 ms waits
        assert ra.allreduce(n, "oneshot_waves", stream=sa, opt=muted) == ll.LL_OK
        assert rb.allreduce(n, "oneshot_waves", stream=sb) == ll.LL_OK
        if order == "b_first":
            assert ll.ll_check(sb.cuda_stream) == ll.LL_OK
            assert ll.ll_check(sa.cuda_stream) == ll.LL_ERR_TIMEOUT
        else:
            assert ll.ll_check(sa.cuda_stream) == ll.LL_ERR_TIMEOUT
            assert ll.ll_check(sb.cuda_stream) == ll.LL_OK
        rank, missing, epoch = ll.ll_last_timeout()
        assert missing & (1 << 5) and epoch == ra.epoch and rank != 5
        assert ll.ll_check(sa.cuda_stream) == ll.LL_OK  # read and cleared
        assert np.array_equal(rb.read_out(p * n, np.uint16).reshape(p, n), oracle.allreduce(x))
        ra.init(sa)  # a timed-out region is re-initialised before reuse
    check_ok(ra.allreduce(n, "oneshot_waves", stream=sa), "region A after re-init", sa.cuda_stream)
    torch.cuda.synchronize()
    assert np.array_equal(ra.read_out(p * n, np.uint16).reshape(p, n), oracle.allreduce(x))
