"""GPU parity of the bounded-scratch AllReduce (multi-iteration, double
buffering): every algorithm, 1 .. 64 iterations, ragged last iterations,
in place, back-to-back calls, against the CPU oracle at 0 ulp."""
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
    from paper_2607_16100_amd.region import ScratchRegion  # noqa: E402
else:  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

ALGOS = ["oneshot", "oneshot_line", "oneshot_sentinel", "twoshot", "twoshot_line", "twoshot_sentinel",
         "twoshot_sentinel_out", "twoshot_waves", "twoshot_sentinel_waves", "twoshot_line_waves", "auto"]
NP = {"f32": np.uint32, "bf16": np.uint16}
TEST_TIMEOUT_TICKS = 20_000_000


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


def run(reg, x, algo, opt=None):
    p, n = x.shape
    reg.write_inputs(x)
    check_ok(reg.allreduce(n, algo, opt=opt), f"buffered {algo} P={p} n={n}")
    return reg.read_out(p * n, x.dtype).reshape(p, n)


def usable(algo, n, esize, iters):
    if algo == "twoshot_sentinel_out" and (n * esize) % 16:
        return False
    return True


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [2, 3, 6, 7, 8])
def test_iterations_parity(dtype, p):
    """Iteration size 4 KiB; messages of 1, 2, 3 and 7+ iterations with a
    ragged last iteration, every algorithm, two calls in a row."""
    es = 4 if dtype == "f32" else 2
    reg = ScratchRegion(p, 40_000, dtype, iter_bytes=4096)
    reg.init()
    d = reg.iter_bytes // es
    for n in [5, d, d + 8, 2 * d, 3 * d - 8, 7 * d + 8, 40_000]:
        x = wl.normal(p, n, dtype, seed=n + p)
        want = oracle.allreduce(x)
        for algo in ALGOS:
            if not usable(algo, n, es, 0):
                continue
            for k in range(2):
                say(f"buffered {algo} P={p} {dtype} n={n} call {k}")
                got = run(reg, x, algo)
                assert reg.last_iters == -(-n // d)
                assert_bits_equal(got, want, f"{algo} P={p} {dtype} n={n} call {k}")


def test_waves_one_iteration_only():
    reg = ScratchRegion(8, 10_000, "bf16", iter_bytes=4096)
    reg.init()
    x = wl.normal(8, 1000, "bf16", seed=4)
    assert_bits_equal(run(reg, x, "oneshot_waves"), oracle.allreduce(x), "waves, one iteration")
    reg.write_inputs(wl.normal(8, 10_000, "bf16", seed=5))
    assert reg.allreduce(10_000, "oneshot_waves") == ll.LL_ERR_UNSUPPORTED


@pytest.mark.parametrize("algo", [a for a in ALGOS if a != "twoshot_sentinel_out"] + ["oneshot_waves"])
def test_in_place(algo):
    """in == out: each rank's input is overwritten by its result."""
    p, n = 8, 30_000
    reg = ScratchRegion(p, n, "bf16", iter_bytes=16384 if algo != "oneshot_waves" else 1 << 20, in_place=True)
    reg.init()
    for k in range(2):
        x = wl.uniform(p, n, "bf16", seed=50 + k)
        say(f"in place {algo} call {k}")
        assert_bits_equal(run(reg, x, algo), oracle.allreduce(x), f"in place {algo} call {k}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [3, 5, 8])
def test_in_place_one_iteration(dtype, p):
    """in == out with the whole message in one iteration, where the one-tile
    kernels run: each wave reads a tile of its chunk's input and later
    writes the same tile of the output.  Two calls per algorithm, ragged
    chunk ends."""
    n = 30_001 if dtype == "f32" else 30_002
    reg = ScratchRegion(p, n, dtype, iter_bytes=1 << 20, in_place=True)
    reg.init()
    for algo in ("twoshot_waves", "twoshot_sentinel_waves", "twoshot_line_waves", "oneshot_waves",
                 "oneshot_sentinel_waves", "oneshot_line_waves", "auto"):
        for k in range(2):
            x = wl.normal(p, n, dtype, seed=70 + k + p)
            say(f"in place, one iteration: {algo} P={p} {dtype} call {k}")
            assert_bits_equal(run(reg, x, algo), oracle.allreduce(x), f"in place one iteration {algo} P={p}")
            assert reg.last_iters == 1


IN_PLACE_ALGOS = ["auto", "twoshot", "twoshot_line", "twoshot_sentinel", "twoshot_waves", "twoshot_sentinel_waves",
                  "twoshot_line_waves", "oneshot", "oneshot_line"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [3, 5, 6, 7])
def test_in_place_rank_counts_that_do_not_divide_the_iteration(dtype, p):
    """In place, several iterations, with rank counts whose P chunks of an
    iteration overrun it (P * chunk > iteration elements): a kernel that cut
    an iteration by the whole message's count would reduce elements of the
    next iteration and overwrite its inputs before every rank has read them."""
    es = 4 if dtype == "f32" else 2
    reg = ScratchRegion(p, 40_000, dtype, iter_bytes=4096, in_place=True)
    reg.init()
    d = reg.iter_bytes // es
    for n in [3 * d, 5 * d + 7, 40_000]:
        for algo in IN_PLACE_ALGOS:
            x = wl.normal(p, n, dtype, seed=n + 31 * p)
            say(f"in place {algo} P={p} {dtype} n={n} ({-(-n // d)} iterations)")
            assert_bits_equal(run(reg, x, algo), oracle.allreduce(x), f"in place {algo} P={p} {dtype} n={n}")
            assert reg.last_iters == -(-n // d)


def test_direct_output_rejects_in_place():
    reg = ScratchRegion(4, 1024, "f32", iter_bytes=4096, in_place=True)
    reg.init()
    assert reg.allreduce(1024, "twoshot_sentinel_out") == ll.LL_ERR_INVALID


@pytest.mark.parametrize("algo", ["oneshot", "twoshot_line", "oneshot_sentinel", "twoshot_sentinel", "twoshot_waves",
                                  "twoshot_sentinel_waves", "twoshot_line_waves"])
def test_many_iterations_small_grids(algo):
    """64 iterations with one small workgroup per rank (each lane serves many
    units per iteration) and with the automatic grid."""
    p, n = 8, 64 * 1024
    reg = ScratchRegion(p, n, "f32", iter_bytes=4096)
    reg.init()
    x = wl.normal(p, n, "f32", seed=77)
    want = oracle.allreduce(x)
    for wg, threads in [(1, 64), (2, 256), (0, 0)]:
        say(f"64 iterations {algo} wg={wg} t={threads}")
        assert_bits_equal(run(reg, x, algo, opts(workgroups_per_rank=wg, threads=threads)), want,
                          f"{algo} wg={wg} t={threads}")
        assert reg.last_iters == 64


def test_epochs_advance_by_iterations():
    p, n = 4, 10_000
    reg = ScratchRegion(p, n, "f32", iter_bytes=4096)
    reg.init()
    x = wl.uniform(p, n, "f32", seed=8)
    run(reg, x, "twoshot")
    assert reg.epoch == reg.last_iters == -(-n * 4 // reg.iter_bytes)
    # a call that would run past epoch 0xFFFFFFFF is refused before launching
    st, _ = ll.ll_allreduce_buffered(reg.inp.data_ptr(), reg.out.data_ptr(), n, ll.LL_F32, ll.LL_SUM, p,
                                     reg.scratch.data_ptr(), reg.scratch_stride, 0xFFFFFFFF, stream(),
                                     ll.LL_ALGO_TWOSHOT, None)
    assert st == ll.LL_ERR_INVALID


def test_e4_scale_32mib_message():
    """The paper's scratch study shape: 32 MiB per rank, 8 ranks, iterations
    of 4 MiB (8 iterations) and 1 MiB (32), one-shot and two-shot."""
    p, n = 8, (32 << 20) // 4
    x = wl.uniform(p, n, "f32", seed=32)
    want = oracle.allreduce(x)
    for it_bytes in (4 << 20, 1 << 20):
        reg = ScratchRegion(p, n, "f32", iter_bytes=it_bytes)
        reg.init()
        for algo in ("oneshot_line", "twoshot_line", "twoshot_sentinel", "twoshot_line_waves", "twoshot_sentinel_waves"):
            say(f"32 MiB {algo} iterations of {it_bytes >> 10} KiB")
            assert_bits_equal(run(reg, x, algo), want, f"32 MiB {algo} {it_bytes}")
        del reg


@pytest.mark.parametrize("algo", ["oneshot", "twoshot_sentinel", "twoshot_line_waves", "twoshot_sentinel_waves"])
def test_missing_peer_times_out_and_scratch_init_recovers(algo):
    p, n = 8, 8192
    reg = ScratchRegion(p, n, "f32", iter_bytes=4096)
    reg.init()
    x = wl.uniform(p, n, "f32", seed=2)
    reg.write_inputs(x)
    assert reg.allreduce(n, algo, opt=opts(poll_timeout=200_000, mute_rank=6)) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    reg.init()
    assert_bits_equal(run(reg, x, algo), oracle.allreduce(x), f"{algo} after timeout")
