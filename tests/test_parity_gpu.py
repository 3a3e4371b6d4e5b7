"""GPU parity: the HIP collectives against the CPU oracle, bit for bit.

Every test calls the library through its C ABI (``llcoll``) on cuda:0 and
compares raw element bits with ``oracle`` (0 ulp for binary32 and bfloat16:
binary32 accumulation in ascending rank order, one rounding).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2607_16100_amd import workloads as wl  # noqa: E402
from sumbound import assert_within_summation_bound  # noqa: E402

if torch.cuda.is_available():
    from paper_2607_16100_amd import llcoll as ll  # noqa: E402
    from paper_2607_16100_amd.region import SymRegion  # noqa: E402
else:  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

AR_ALGOS = ["oneshot", "twoshot", "twoshot_line", "oneshot_line", "oneshot_waves", "oneshot_sentinel",
            "twoshot_sentinel", "twoshot_waves", "twoshot_sentinel_waves", "oneshot_sentinel_waves",
            "oneshot_line_waves", "twoshot_line_waves", "auto"]
PROTOS = ["packet8", "line128", "sentinel"]
NP = {"f32": np.uint32, "bf16": np.uint16}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def stream():
    return torch.cuda.current_stream().cuda_stream


def check_ok(st, what):
    assert st == ll.LL_OK, f"{what}: {ll.ll_strerror(st)}"
    st2 = ll.ll_check(stream())
    assert st2 == ll.LL_OK, f"{what}: ll_check says {ll.ll_strerror(st2)}"


def run_allreduce(reg: SymRegion, x: np.ndarray, algo: str, opt=None) -> np.ndarray:
    p, n = x.shape
    reg.write_inputs(x)
    check_ok(reg.allreduce(n, algo, opt=opt), f"allreduce {algo} P={p} n={n}")
    return reg.read_out(p * n, x.dtype).reshape(p, n)


def assert_bits_equal(got, want, what):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        r, i = bad[0]
        raise AssertionError(f"{what}: {len(bad)} elements differ; first at rank {r} index {i}: "
                             f"got {int(got[r, i]):#x} want {int(want[r, i]):#x}")


TEST_TIMEOUT_TICKS = 20_000_000  # 200 ms per flag wait: thousands of times a correct call's duration


def opts(**kw):
    """Per-call options: the tests' short wait bound plus any tuning fields."""
    kw.setdefault("poll_timeout", TEST_TIMEOUT_TICKS)
    return ll.Options(**kw)


MUTED_TIMEOUT_TICKS = 200_000  # 2 ms: waits for a muted rank expire quickly


# ------------------------------------------------------------ configuration C1
def test_c1_oneshot_p4_f32_1024():
    """One-shot, 4 ranks, binary32, 1024 uniform(-1,1) elements per rank (seed r), epoch 1."""
    x = wl.uniform(4, 1024, "f32", seed=0)
    reg = SymRegion(4, 1024, "f32")
    reg.init()
    reg.write_inputs(x)
    check_ok(reg.allreduce(1024, "oneshot", epoch=1), "C1")
    got = reg.read_out(4 * 1024, np.uint32).reshape(4, 1024)
    assert_bits_equal(got, oracle.allreduce(x), "C1")


# ------------------------------------------------ every algorithm, ragged sizes
SMALL_N = [1, 2, 3, 5, 17, 63, 64, 65, 129, 1000, 4099, 30 * 8 * 3 + 7]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [2, 3, 4, 5, 6, 7, 8])
def test_allreduce_all_algorithms_ragged(dtype, p):
    """All four algorithms on one region, sizes across several units with ragged
    tails, alternating calls (the slice layout keeps every flag position fixed)."""
    reg = SymRegion(p, max(SMALL_N), dtype)
    reg.init()
    for n in SMALL_N:
        x = wl.uniform(p, n, dtype, seed=100 + n)
        want = oracle.allreduce(x)
        for algo in AR_ALGOS:
            say(f"allreduce {algo} P={p} {dtype} n={n}")
            assert_bits_equal(run_allreduce(reg, x, algo), want, f"{algo} P={p} {dtype} n={n}")


# Element counts around the unit boundaries of the one-tile kernels: a line
# unit carries 240 words (480 bfloat16 or 240 binary32 elements), a tile of
# one-lane units 1 KiB of payload (512 or 256 elements); 61440 bfloat16 are
# 128 line units, the most a launch of 4 workgroups per CU keeps resident at
# 8 ranks (one more unit takes the multi-tile kernel).
TILE_N = {"bf16": [2, 478, 480, 482, 958, 960, 1024, 480 * 37 + 2, 61440, 61442],
          "f32": [1, 239, 240, 241, 256, 257, 240 * 50 + 3, 30720, 30721]}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [2, 3, 5, 8])
def test_one_tile_kernels_at_unit_boundaries(dtype, p):
    """The one-tile kernels, one-shot and two-shot (8-byte packets, sentinel
    units, lines; the host takes them for 4-byte aligned streams whose tiles
    are all resident) at counts on both sides of a unit and of the resident
    limit, with slot clearing forced on and off, two calls per case.  The
    two-shot splits the counts into P chunks, so its tiles meet ragged chunk
    ends and, for the smallest counts, empty chunks."""
    sizes = TILE_N[dtype]
    reg = SymRegion(p, max(sizes), dtype)
    reg.init()
    for n in sizes:
        for algo in ("oneshot_waves", "oneshot_sentinel_waves", "oneshot_line_waves", "twoshot_waves",
                     "twoshot_sentinel_waves", "twoshot_line_waves"):
            for clear in (1, 2):
                for call in range(2):
                    x = wl.normal(p, n, dtype, seed=31 * n + call)
                    say(f"one-tile {algo} P={p} {dtype} n={n} clear={clear} call {call}")
                    got = run_allreduce(reg, x, algo, opt=opts(clear_slots=clear))
                    assert_bits_equal(got, oracle.allreduce(x), f"{algo} P={p} {dtype} n={n} clear={clear}")


@pytest.mark.parametrize("algo", AR_ALGOS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_allreduce_special_values(algo, dtype):
    """Order pins, signed zeros and subnormals go through the kernels unchanged."""
    p = 8
    cols = [
        [2.0 ** 24, 1.0, -(2.0 ** 24), 0, 0, 0, 0, 0],
        [-(2.0 ** 24), 0, 2.0 ** 24, 1.0, 0, 0, 0, 0],
        [256.0, 1.0, 1.0, 0, 0, 0, 0, 0],
        [256.0, 1.0, 0, 0, 0, 0, 0, 0],
        [-0.0] * 8,
        [2.0 ** -130, 2.0 ** -130, 0, 0, 0, 0, 0, 0],
    ]
    vals = np.array(cols * 50, dtype=np.float32).T.copy()  # [8, 300]
    bits = vals.view(np.uint32)
    if dtype == "bf16":
        bits = (bits >> 16).astype(np.uint16)
    reg = SymRegion(p, bits.shape[1], dtype)
    reg.init()
    assert_bits_equal(run_allreduce(reg, bits, algo), oracle.allreduce(bits), f"special {algo} {dtype}")


# ------------------------------------------------------------ configuration C2
@pytest.mark.parametrize("algo", ["oneshot", "oneshot_waves", "auto"])
def test_c2_oneshot_bf16_16k_10k_calls(algo):
    """8 ranks, bfloat16, 8192 normal(0,1) elements per rank, one-shot with
    8-byte packets (and AUTO, which takes the line one-shot with one wave per
    peer here), 10,000 back-to-back calls with the epoch incremented."""
    p, n = 8, 8192
    x = wl.normal(p, n, "bf16", sigma=1.0, seed=0)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    reg.write_inputs(x)
    s = stream()
    for i in range(10_000):
        st = reg.allreduce(n, algo)
        assert st == ll.LL_OK
        if i % 1000 == 999:
            assert ll.ll_check(s) == ll.LL_OK, f"C2: status after call {i}"
    assert ll.ll_check(s) == ll.LL_OK
    got = reg.read_out(p * n, np.uint16).reshape(p, n)
    assert_bits_equal(got, want, "C2 after 10k calls")
    assert reg.epoch == 10_000


@pytest.mark.parametrize("algo", ["oneshot_waves", "auto", "oneshot_line_waves", "twoshot_line"])
def test_benchmark_launch_loop_is_exact(algo):
    """The C-side launch loop the benchmark times (ll_bench_allreduce): 2000
    back-to-back calls on the 16 KiB, 8-rank workload with epochs 1..2000,
    the last ten with per-workgroup stamps, leave the oracle's result and no
    timed-out wait; every stamped workgroup ends after it starts."""
    p, n = 8, 8192
    x = wl.normal(p, n, "bf16", sigma=1.0, seed=0)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    reg.write_inputs(x)
    s = reg.stream_handle()
    code = ll.ALGOS[algo]
    say(f"bench loop {algo}: 1990 calls")
    shape = ll.Options(report=True)
    st = ll.ll_bench_allreduce(reg.base, reg.rank_stride, reg.out_ptr, n, ll.LL_BF16, p, reg.epoch + 1, 1990, code,
                               shape, 0, 0, s)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    reg.epoch += 1990
    assert ll.ll_check(s) == ll.LL_OK
    grid = shape.grid
    assert grid > 0
    stamps = torch.zeros(10 * 2 * grid, dtype=torch.int64, device="cuda")
    say(f"bench loop {algo}: 10 stamped calls, grid {grid}")
    st = ll.ll_bench_allreduce(reg.base, reg.rank_stride, reg.out_ptr, n, ll.LL_BF16, p, reg.epoch + 1, 10, code,
                               None, stamps.data_ptr(), 2 * grid, s)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    reg.epoch += 10
    assert ll.ll_check(s) == ll.LL_OK
    got = reg.read_out(p * n, np.uint16).reshape(p, n)
    assert_bits_equal(got, want, f"bench loop {algo}")
    t = stamps.view(10, 2, grid).cpu().numpy()
    assert (t[:, 0] > 0).all() and (t[:, 1] >= t[:, 0]).all()


@pytest.mark.parametrize("proto", PROTOS)
def test_benchmark_rs_ag_loops_are_exact(proto):
    """ll_bench_reduce_scatter / ll_bench_allgather, 500 calls each at C5's
    b=1 shape (8 ranks, 7168 bf16 per rank), leave the oracle's result."""
    p, total = 8, 7168
    m = total // p
    x = wl.normal(p, total, "bf16", sigma=1.0, seed=4)
    reg = SymRegion(p, total, "bf16", out_elems=p * total)
    reg.init()
    s = reg.stream_handle()
    reg.write_inputs(x)
    say(f"bench RS loop {proto}")
    st = ll.ll_bench_reduce_scatter(reg.base, reg.rank_stride, reg.out_ptr, m, ll.LL_BF16, p, reg.epoch + 1, 500,
                                    ll.PROTOS[proto], None, 0, 0, s)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    reg.epoch += 500
    assert ll.ll_check(s) == ll.LL_OK
    rs = reg.read_out(p * m, np.uint16).reshape(p, m)
    assert_bits_equal(rs, oracle.reduce_scatter(x), f"bench RS loop {proto}")
    reg.write_inputs(rs)
    say(f"bench AG loop {proto}")
    st = ll.ll_bench_allgather(reg.base, reg.rank_stride, reg.out_ptr, m, ll.LL_BF16, p, reg.epoch + 1, 500,
                               ll.PROTOS[proto], None, 0, 0, s)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    reg.epoch += 500
    assert ll.ll_check(s) == ll.LL_OK
    ag = reg.read_out(p * p * m, np.uint16).reshape(p, p * m)
    assert_bits_equal(ag, oracle.allreduce(x), f"bench AG loop {proto}")


@pytest.mark.parametrize("algo", AR_ALGOS)
def test_changing_inputs_never_return_stale_packets(algo):
    """New inputs every call (seed r + 1000 k): a packet left from an earlier
    epoch would show up as a wrong value."""
    p, n = 8, 8192
    reg = SymRegion(p, n, "bf16")
    reg.init()
    for k in range(60):
        x = wl.normal(p, n, "bf16", seed=1000 * k)
        assert_bits_equal(run_allreduce(reg, x, algo), oracle.allreduce(x), f"{algo} change {k}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_random_call_sequence_on_one_region(dtype):
    """One region, 150 calls in a seeded random order: every deterministic
    AllReduce algorithm and AUTO at random sizes (1 element .. 96 Ki),
    ReduceScatter / AllGather with every format, and Broadcast / Reduce with a
    random root, each with new inputs.  Whatever the previous call left in the
    packet areas (other sizes, formats, kernels, iteration layouts), no stale
    packet may ever be accepted."""
    p, nmax = 8, 96 * 1024
    rng = np.random.default_rng(20261202 if dtype == "bf16" else 7)
    reg = SymRegion(p, nmax, dtype, out_elems=p * nmax)
    reg.init()
    algos = AR_ALGOS
    for k in range(150):
        kind = rng.choice(["ar", "ar", "ar", "rs", "ag", "bcast", "reduce"])
        n = int(rng.integers(1, nmax + 1)) if rng.random() < 0.5 else int(rng.integers(1, 2048))
        seed = 10_000 + 1000 * k
        if kind == "ar":
            algo = str(rng.choice(algos))
            x = wl.normal(p, n, dtype, seed=seed)
            say(f"seq {k}: allreduce {algo} n={n}")
            assert_bits_equal(run_allreduce(reg, x, algo), oracle.allreduce(x), f"seq {k} {algo} n={n}")
        elif kind in ("rs", "ag"):
            proto = str(rng.choice(PROTOS))
            m = max(1, n // p)
            if kind == "rs":
                x = wl.normal(p, p * m, dtype, seed=seed)
                reg.write_inputs(x)
                say(f"seq {k}: reduce_scatter {proto} m={m}")
                check_ok(reg.reduce_scatter(m, proto), f"seq {k} rs")
                assert_bits_equal(reg.read_out(p * m, NP[dtype]).reshape(p, m), oracle.reduce_scatter(x),
                                  f"seq {k} rs {proto} m={m}")
            else:
                x = wl.normal(p, m, dtype, seed=seed)
                reg.write_inputs(x)
                say(f"seq {k}: allgather {proto} m={m}")
                check_ok(reg.allgather(m, proto), f"seq {k} ag")
                assert_bits_equal(reg.read_out(p * p * m, NP[dtype]).reshape(p, p * m), oracle.allgather(x),
                                  f"seq {k} ag {proto} m={m}")
        else:
            proto = str(rng.choice(PROTOS))
            root = int(rng.integers(0, p))
            x = wl.normal(p, n, dtype, seed=seed)
            reg.write_inputs(x)
            if kind == "bcast":
                say(f"seq {k}: broadcast {proto} root={root} n={n}")
                check_ok(reg.broadcast(n, root, proto), f"seq {k} bcast")
                assert_bits_equal(reg.read_out(p * n, NP[dtype]).reshape(p, n), oracle.broadcast(x, root),
                                  f"seq {k} bcast {proto} n={n}")
            else:
                say(f"seq {k}: reduce {proto} root={root} n={n}")
                check_ok(reg.reduce(n, root, proto), f"seq {k} reduce")
                got = reg.read_out(n, NP[dtype]).reshape(1, n)
                assert_bits_equal(got, oracle.reduce(x, root).reshape(1, n), f"seq {k} reduce {proto} n={n}")


# ------------------------------------------------------------ configuration C3
def test_c3_twoshot_bf16_1mib_vs_oneshot():
    """8 ranks, bfloat16, 64 x 8192 normal(0, 0.5) per rank: two-shot (both
    packet formats) equals the oracle and equals one-shot."""
    p, n = 8, 64 * 8192
    x = wl.normal(p, n, "bf16", sigma=0.5, seed=0)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    outs = {}
    for algo in AR_ALGOS:
        say(f"C3 {algo}")
        outs[algo] = run_allreduce(reg, x, algo)
        assert_bits_equal(outs[algo], want, f"C3 {algo}")
    assert np.array_equal(outs["twoshot"], outs["oneshot"])


# ------------------------------------------------------------ configuration C4
C4_SIZES = [2 ** k for k in range(1, 27)]


def test_c4_size_sweep_parity():
    """8 ranks, binary32 uniform(-1,1): every power-of-two size from 2 to 2^26
    elements per rank, one-shot and two-shot with both packet formats."""
    p = 8
    big = C4_SIZES[-1]
    reg = SymRegion(p, big, "f32", out_elems=p * big)
    reg.init()
    for n in C4_SIZES:
        x = wl.uniform(p, n, "f32", seed=0)
        want = oracle.allreduce(x)
        for algo in AR_ALGOS:
            say(f"C4 {algo} n={n}")
            assert_bits_equal(run_allreduce(reg, x, algo), want, f"C4 {algo} n={n}")


# ------------------------------------------------------------ configuration C5
@pytest.mark.parametrize("p", [8, 4])
@pytest.mark.parametrize("b", [1, 16, 256])
@pytest.mark.parametrize("kind", ["normal", "adversarial"])
def test_c5_reduce_scatter_and_allgather(p, b, kind):
    """hidden 7168 x batch b, bfloat16: ReduceScatter of b*7168 per rank and
    AllGather of b*7168/P per rank, both packet formats; AG(RS(x)) == AR(x)."""
    total = 7168 * b
    m = total // p
    x = wl.make(kind, p, total, "bf16", seed=0)
    want_rs = oracle.reduce_scatter(x)
    reg = SymRegion(p, total, "bf16", out_elems=p * total)
    reg.init()
    for proto, wk in [(pr, w) for pr in PROTOS for w in (1, 2)] + [("auto", 0)]:
        reg.opt = opts(wave_kernels=wk)
        say(f"C5 RS {kind} P={p} b={b} {proto} kernels={wk}")
        reg.write_inputs(x)
        check_ok(reg.reduce_scatter(m, proto), "reduce_scatter")
        got_rs = reg.read_out(p * m, np.uint16).reshape(p, m)
        assert_bits_equal(got_rs, want_rs, f"RS {proto} kernels={wk}")
        say(f"C5 AG {kind} P={p} b={b} {proto} kernels={wk}")
        reg.write_inputs(got_rs)
        check_ok(reg.allgather(m, proto), "allgather")
        got_ag = reg.read_out(p * p * m, np.uint16).reshape(p, p * m)
        assert_bits_equal(got_ag, oracle.allgather(got_rs), f"AG {proto} kernels={wk}")
        assert_bits_equal(got_ag, oracle.allreduce(x), f"AG(RS) == AR {proto} kernels={wk}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("proto", PROTOS)
@pytest.mark.parametrize("p,m", [(2, 1), (3, 7), (4, 33), (8, 5), (8, 61), (5, 250), (6, 13), (6, 100), (7, 9),
                                 (7, 333)])
def test_rs_ag_ragged(dtype, proto, p, m):
    """Chunks whose byte offsets are not 4-byte aligned (odd bfloat16 counts),
    with both kernel families."""
    x = wl.uniform(p, p * m, dtype, seed=7)
    reg = SymRegion(p, p * m, dtype, out_elems=p * p * m)
    reg.init()
    for wk in (1, 2):
        reg.opt = opts(wave_kernels=wk)
        reg.write_inputs(x)
        check_ok(reg.reduce_scatter(m, proto), "rs")
        rs = reg.read_out(p * m, NP[dtype]).reshape(p, m)
        assert_bits_equal(rs, oracle.reduce_scatter(x), f"RS ragged {proto} kernels={wk}")
        reg.write_inputs(x[:, :m].copy())
        check_ok(reg.allgather(m, proto), "ag")
        ag = reg.read_out(p * p * m, NP[dtype]).reshape(p, p * m)
        assert_bits_equal(ag, oracle.allgather(x[:, :m].copy()), f"AG ragged {proto} kernels={wk}")


# ------------------------------------------------------------ invariants
@pytest.mark.parametrize("algo", AR_ALGOS)
def test_result_independent_of_launch_shape(algo):
    p, n = 8, 50_000
    x = wl.uniform(p, n, "bf16", seed=3)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    for wg, threads in [(1, 64), (1, 1024), (3, 256), (16, 128), (0, 0)]:
        if algo == "twoshot_sentinel":  # the direct-output variant shares the launch shapes
            say(f"launch twoshot_sentinel_out wg={wg} threads={threads}")
            assert_bits_equal(run_allreduce(reg, x, "twoshot_sentinel_out",
                                            opts(workgroups_per_rank=wg, threads=threads)),
                              want, f"direct wg={wg} t={threads}")
        for units in ([1, 2, 4, 0] if algo.endswith("_waves") else [0]):
            say(f"launch {algo} wg={wg} threads={threads} units={units}")
            o = opts(workgroups_per_rank=wg, threads=threads, wave_units=units)
            assert_bits_equal(run_allreduce(reg, x, algo, o), want, f"{algo} wg={wg} t={threads} u={units}")


WAVE_ALGOS = ["oneshot_waves", "oneshot_sentinel_waves", "oneshot_line_waves", "twoshot_waves",
              "twoshot_sentinel_waves", "twoshot_line_waves"]


@pytest.mark.parametrize("algo", WAVE_ALGOS)
@pytest.mark.parametrize("n", [5, 300])
def test_workgroups_past_the_last_tile(algo, n):
    """A forced launch with more workgroups per rank than there are tiles: the
    wave kernels issue their first loads and stores before they look at the
    tile count, so a workgroup past the last tile must load and store nothing.
    The result is exact and the output past P*n elements is untouched."""
    p = 8
    x = wl.normal(p, n, "bf16", seed=n)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    guard = np.uint8(0xA5)
    reg.out.fill_(int(guard))
    got = run_allreduce(reg, x, algo, opts(workgroups_per_rank=16))
    assert_bits_equal(got, oracle.allreduce(x), f"{algo} n={n} W=16")
    tail = reg.out[p * n * 2:].cpu().numpy()
    assert (tail == guard).all(), f"{algo}: {int((tail != guard).sum())} bytes written past the output"


@pytest.mark.parametrize("proto", PROTOS)
def test_rs_ag_workgroups_past_the_last_tile(proto):
    """The same for the wave-per-peer ReduceScatter and AllGather."""
    p, m = 8, 37
    x = wl.normal(p, p * m, "bf16", seed=5)
    reg = SymRegion(p, p * m, "bf16", out_elems=p * p * m + 4096)
    reg.init()
    guard = np.uint8(0x5A)
    reg.opt = opts(wave_kernels=2, workgroups_per_rank=16)
    reg.out.fill_(int(guard))
    reg.write_inputs(x)
    check_ok(reg.reduce_scatter(m, proto), "rs")
    rs = reg.read_out(p * m, np.uint16).reshape(p, m)
    assert (reg.out[p * m * 2:].cpu().numpy() == guard).all(), "RS wrote past its output"
    reg.out.fill_(int(guard))
    reg.write_inputs(rs)
    check_ok(reg.allgather(m, proto), "ag")
    ag = reg.read_out(p * p * m, np.uint16).reshape(p, p * m)
    assert (reg.out[p * p * m * 2:].cpu().numpy() == guard).all(), "AG wrote past its output"
    assert_bits_equal(rs, oracle.reduce_scatter(x), f"RS {proto} W=16")
    assert_bits_equal(ag, oracle.allgather(rs), f"AG {proto} W=16")


@pytest.mark.parametrize("lag", [0, 1, 2, 5])
def test_result_independent_of_pipeline_lag(lag):
    """Two-shot, ReduceScatter and AllGather give the same bits for every
    pipeline distance (and launch shape), on sizes with many steps."""
    p, n = 8, 300_000
    x = wl.normal(p, n, "bf16", seed=13)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "bf16", out_elems=p * n)
    reg.init()
    for wg, threads in [(1, 64), (4, 256), (0, 0)]:
        reg.opt = opts(pipeline_lag=lag, workgroups_per_rank=wg, threads=threads)
        for algo in ("twoshot", "twoshot_line", "twoshot_sentinel", "twoshot_sentinel_out"):
            say(f"lag={lag} {algo} wg={wg} t={threads}")
            assert_bits_equal(run_allreduce(reg, x, algo), want, f"{algo} lag={lag} wg={wg}")
        m = n // p
        for proto in PROTOS:
            reg.write_inputs(x)
            check_ok(reg.reduce_scatter(m, proto), "rs")
            rs = reg.read_out(p * m, np.uint16).reshape(p, m)
            assert_bits_equal(rs, oracle.reduce_scatter(x), f"RS {proto} lag={lag}")
            reg.write_inputs(rs)
            check_ok(reg.allgather(m, proto), "ag")
            ag = reg.read_out(p * p * m, np.uint16).reshape(p, p * m)
            assert_bits_equal(ag, oracle.allgather(rs), f"AG {proto} lag={lag}")


def test_large_epochs_and_reinit():
    """Epochs near the top of the 32-bit range, one per call, then ll_init and a
    restart at epoch 1."""
    p, n = 4, 3000
    x = wl.uniform(p, n, "f32", seed=9)
    want = oracle.allreduce(x)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(x)
    epochs = (0x7FFFFFFF, 0x80000000, 0xFFFFFFEE, 0xFFFFFFF0, 0xFFFFFFF2, 0xFFFFFFF4, 0xFFFFFFF6, 0xFFFFFFF8,
              0xFFFFFFF9, 0xFFFFFFFA, 0xFFFFFFFC, 0xFFFFFFFE, 0xFFFFFFFF)
    assert len(epochs) == len(AR_ALGOS)
    for algo, e in zip(AR_ALGOS, epochs):
        check_ok(reg.allreduce(n, algo, epoch=e), f"epoch {e:#x}")
        assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), want, f"{algo} epoch {e:#x}")
    reg.init()
    check_ok(reg.allreduce(n, "twoshot", epoch=1), "after init")
    assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), want, "after re-init")


def test_count_zero_is_a_no_op():
    reg = SymRegion(4, 16, "f32")
    reg.init()
    assert reg.allreduce(0, "oneshot") == ll.LL_OK
    assert reg.reduce_scatter(0, "packet8") == ll.LL_OK
    assert reg.allgather(0, "line128") == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_OK


# ------------------------------------------------------------ failure handling
@pytest.mark.parametrize("algo", ["oneshot", "twoshot_line", "oneshot_sentinel", "twoshot_sentinel", "twoshot_waves",
                                  "twoshot_sentinel_waves", "oneshot_waves", "oneshot_sentinel_waves",
                                  "oneshot_line_waves", "twoshot_line_waves"])
def test_missing_peer_times_out_and_is_reported(algo):
    """Rank 3 publishes nothing; its peers' bounded waits expire (after 2 ms),
    every kernel still finishes, and ll_check reports the timeout.  (In two-shot
    the peers then publish late, so rank 3 may be the first to give up.)"""
    p, n = 8, 4096
    x = wl.uniform(p, n, "f32", seed=1)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(x)
    st = reg.allreduce(n, algo, opt=opts(poll_timeout=MUTED_TIMEOUT_TICKS, mute_rank=3))
    assert st == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    rank, missing, epoch = ll.ll_last_timeout()
    assert epoch == reg.epoch and missing != 0
    if algo.startswith("oneshot"):
        # only rank 3's packets are missing; the first rank to give up names it
        assert rank != 3 and missing == (1 << 3)
    reg.init()
    check_ok(reg.allreduce(n, algo), "after timeout")
    assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), oracle.allreduce(x), "after timeout")


def test_next_epoch_sees_new_inputs():
    """Back-to-back calls with consecutive epochs and different inputs: each
    call returns the sum of its own inputs."""
    p, n = 4, 512
    a = wl.uniform(p, n, "f32", seed=1)
    b = wl.uniform(p, n, "f32", seed=2)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(a)
    check_ok(reg.allreduce(n, "oneshot", epoch=5), "a")
    assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), oracle.allreduce(a), "epoch 5")
    reg.write_inputs(b)
    check_ok(reg.allreduce(n, "oneshot", epoch=6), "b")
    assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), oracle.allreduce(b), "epoch 6")


# ------------------------------------------------------------ sentinel mode
SENT = 0xFFFFFFFF


@pytest.mark.parametrize("algo", ["oneshot_sentinel", "twoshot_sentinel", "twoshot_sentinel_waves",
                                  "oneshot_sentinel_waves"])
def test_sentinel_slots_are_restored_after_every_call(algo):
    """Sentinel mode resets every slot it has read (Sec. IV, Sentinel): after
    a call the sentinel area holds only the sentinel again, and the flagged
    packet areas are untouched by sentinel calls."""
    p, n = 8, 40_000
    x = wl.normal(p, n, "bf16", seed=21)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    assert (reg.read_area(4) == SENT).all() and (reg.read_area(1) == 0).all() and (reg.read_area(2) == 0).all()
    for k in range(3):
        say(f"sentinel restore {algo} call {k}")
        assert_bits_equal(run_allreduce(reg, x, algo), oracle.allreduce(x), f"{algo} call {k}")
        area = reg.read_area(4)
        assert (area == SENT).all(), f"{algo}: {(area != SENT).sum()} words not reset after call {k}"
    assert (reg.read_area(1) == 0).all() and (reg.read_area(2) == 0).all()
    m = n // p
    for proto_call in ("rs", "ag"):
        reg.write_inputs(x)
        st = reg.reduce_scatter(m, "sentinel") if proto_call == "rs" else reg.allgather(m, "sentinel")
        check_ok(st, proto_call)
        assert (reg.read_area(4) == SENT).all(), f"{proto_call}: slots not reset"


@pytest.mark.parametrize("algo", ["oneshot_sentinel", "twoshot_sentinel"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_data_equal_to_sentinel_times_out_and_reinit_recovers(algo, dtype):
    """A payload word equal to the sentinel is never seen as arrived (the
    hazard of Sec. IV, Sentinel): the waits on it expire, ll_check reports
    the timeout, and after ll_init a call on clean data is exact again.  The
    flagged protocols carry the same data without trouble."""
    p, n = 4, 2048
    x = wl.uniform(p, n, dtype, seed=5)
    bad = x.copy()
    if dtype == "f32":
        bad[2, 17] = SENT
    else:
        bad[2, 16] = bad[2, 17] = 0xFFFF  # one dword of two -NaN halves
    reg = SymRegion(p, n, dtype)
    reg.init()
    reg.write_inputs(bad)
    say(f"sentinel-valued data {algo} {dtype}")
    assert reg.allreduce(n, algo, opt=opts(poll_timeout=MUTED_TIMEOUT_TICKS)) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    rank, missing, _ = ll.ll_last_timeout()
    assert missing != 0
    if algo == "oneshot_sentinel":
        assert rank != 2 and missing == (1 << 2)
    # the flagged one-shot handles the same words (NaN propagates through the sum)
    reg.init()
    check_ok(reg.allreduce(n, "oneshot"), "flagged on sentinel-valued data")
    got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
    want = oracle.allreduce(bad)
    ok = np.ones(n, bool)
    ok[16:18] = False
    assert np.array_equal(got[:, ok], want[:, ok])
    reg.init()
    reg.write_inputs(x)
    check_ok(reg.allreduce(n, algo), "after re-init")
    assert_bits_equal(reg.read_out(p * n, NP[dtype]).reshape(p, n), oracle.allreduce(x), f"{algo} after re-init")


def test_sentinel_and_flagged_calls_interleave():
    """Sentinel and flagged calls share one region call after call (each
    protocol keeps to its own area), 50 calls, inputs changing every call."""
    p, n = 8, 7168
    reg = SymRegion(p, n, "bf16")
    reg.init()
    algos = ["oneshot_sentinel", "oneshot", "twoshot_sentinel", "twoshot_line", "oneshot_waves"]
    for k in range(50):
        x = wl.uniform(p, n, "bf16", seed=1000 + k)
        algo = algos[k % len(algos)]
        assert_bits_equal(run_allreduce(reg, x, algo), oracle.allreduce(x), f"interleave {algo} call {k}")


# ------------------------------------------------ sentinel-initialised output
DIRECT_CASES = [(2, 4, "f32"), (3, 300, "f32"), (4, 12, "f32"), (5, 1004, "f32"), (8, 4, "f32"), (8, 1000, "f32"),
                (8, 8192, "f32"), (8, 65544, "f32"), (8, 8, "bf16"), (8, 7168, "bf16"), (8, 8192, "bf16"),
                (7, 4000, "bf16"), (8, 1 << 19, "bf16"), (4, 96, "bf16")]


def test_direct_output_twoshot_parity():
    """Two-shot sentinel with the AllGather stored straight into the peers'
    sentinel-filled outputs: bit-exact on sizes that leave the last chunk
    short or some chunks empty, several calls in a row on one region."""
    for p, n, dtype in DIRECT_CASES:
        x = wl.normal(p, n, dtype, seed=n + p)
        want = oracle.allreduce(x)
        reg = SymRegion(p, n, dtype)
        reg.init()
        for k in range(2):
            say(f"direct P={p} n={n} {dtype} call {k}")
            assert_bits_equal(run_allreduce(reg, x, "twoshot_sentinel_out"), want, f"direct P={p} n={n} {dtype}")
        assert (reg.read_area(4) == SENT).all()


def test_direct_output_needs_16_byte_rows():
    x = wl.uniform(4, 1001, "f32", seed=3)  # (fresh device memory may hold the sentinel)
    reg = SymRegion(4, 1001, "f32")
    reg.init()
    reg.write_inputs(x)
    assert reg.allreduce(1001, "twoshot_sentinel_out") == ll.LL_ERR_UNSUPPORTED
    check_ok(reg.allreduce(1000, "twoshot_sentinel_out"), "1000 elements")
    assert_bits_equal(reg.read_out(4 * 1000, np.uint32).reshape(4, 1000), oracle.allreduce(x[:, :1000].copy()),
                      "1000 elements")


def test_fill_sentinel_sets_exactly_the_outputs():
    p, n = 4, 1001
    reg = SymRegion(p, n, "bf16", out_elems=p * n + 64)
    reg.out.zero_()
    check_ok(ll.ll_fill_sentinel(reg.out_ptr, n, ll.LL_BF16, p, stream()), "fill")
    b = reg.out.cpu().numpy()
    assert (b[:p * n * 2] == 0xFF).all() and (b[p * n * 2:] == 0).all()


def test_direct_output_missing_peer_times_out():
    p, n = 8, 4096
    x = wl.uniform(p, n, "f32", seed=1)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(x)
    assert reg.allreduce(n, "twoshot_sentinel_out", opt=opts(poll_timeout=MUTED_TIMEOUT_TICKS, mute_rank=5)) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    reg.init()
    check_ok(reg.allreduce(n, "twoshot_sentinel_out"), "after timeout")
    assert_bits_equal(reg.read_out(p * n, np.uint32).reshape(p, n), oracle.allreduce(x), "after timeout")


@pytest.mark.parametrize("p", [2, 4, 6, 7, 8])
def test_auto_with_sentinel_allowed(p):
    """With sentinel mode allowed, AUTO gives the same bits at every size."""
    for n in [7, 4096, 20_000, 300_000, 3_000_001]:
        x = wl.normal(p, n, "bf16", seed=n)
        reg = SymRegion(p, n, "bf16", opt=opts(flags=ll.LL_OPT_AUTO_SENTINEL))
        reg.init()
        say(f"auto+sentinel P={p} n={n}")
        assert_bits_equal(run_allreduce(reg, x, "auto"), oracle.allreduce(x), f"auto+sentinel P={p} n={n}")
        m = n // p
        if m:
            reg.write_inputs(x)
            check_ok(reg.reduce_scatter(m, "auto"), "rs auto")
            rs = reg.read_out(p * m, np.uint16).reshape(p, m)
            assert_bits_equal(rs, oracle.reduce_scatter(x[:, :p * m].copy()), f"RS auto+sentinel P={p} m={m}")
        del reg


# ------------------------------------------------ atomic-accumulation two-shot
ATOMIC_CASES = [(2, 4, "f32"), (3, 300, "f32"), (4, 1024, "f32"), (5, 1004, "f32"), (8, 8, "f32"),
                (8, 8192, "f32"), (8, 100_000, "f32"), (8, 8, "bf16"), (8, 8192, "bf16"), (7, 4000, "bf16"),
                (8, 64 * 8192, "bf16"), (4, 7168 * 16, "bf16"), (8, 1 << 20, "f32")]


def test_atomic_twoshot_within_bound_and_identical_on_all_ranks():
    for p, n, dtype in ATOMIC_CASES:
        x = wl.normal(p, n, dtype, seed=7 * n + p)
        reg = SymRegion(p, n, dtype)
        reg.init()
        for k in range(3):  # accumulators and counters must be back at zero after each call
            say(f"atomic P={p} n={n} {dtype} call {k}")
            got = run_allreduce(reg, x, "twoshot_atomic")
            assert_within_summation_bound(got, x, dtype, f"atomic P={p} n={n} {dtype} call {k}")
        assert (reg.read_area(3) == 0).all(), "accumulators or counters not reset"
        assert (reg.read_area(4) == SENT).all()


def test_atomic_twoshot_adversarial_sums():
    """The C5 adversarial recipe (near-cancelling rank pairs) still meets the
    bound; with binary32 accumulation cancellation is what stresses it."""
    for p in (4, 8):
        n = 7168 * 16
        x = wl.adversarial(p, n, seed=11)
        reg = SymRegion(p, n, "bf16")
        reg.init()
        assert_within_summation_bound(run_allreduce(reg, x, "twoshot_atomic"), x, "bf16", f"adversarial P={p}")


def test_atomic_twoshot_launch_shapes():
    p, n = 8, 50_000
    x = wl.uniform(p, n, "f32", seed=31)
    reg = SymRegion(p, n, "f32")
    reg.init()
    for wg, threads in [(1, 64), (3, 256), (16, 128), (0, 0)]:
        say(f"atomic launch wg={wg} threads={threads}")
        assert_within_summation_bound(run_allreduce(reg, x, "twoshot_atomic", opts(workgroups_per_rank=wg,
                                                                                   threads=threads)),
                                      x, "f32", f"atomic wg={wg}")


def test_atomic_twoshot_missing_peer_times_out():
    p, n = 8, 4096
    x = wl.uniform(p, n, "f32", seed=1)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(x)
    assert reg.allreduce(n, "twoshot_atomic", opt=opts(poll_timeout=MUTED_TIMEOUT_TICKS, mute_rank=2)) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    reg.init()
    assert_within_summation_bound(run_allreduce(reg, x, "twoshot_atomic"), x, "f32", "after timeout")


# ------------------------------------------------ Broadcast and Reduce
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("p", [2, 3, 5, 6, 7, 8])
def test_broadcast_and_reduce_parity(dtype, p):
    reg = SymRegion(p, 70_001, dtype)
    reg.init()
    for n in [1, 3, 255, 4096, 70_001]:
        x = wl.normal(p, n, dtype, seed=3 * n + p)
        reg.write_inputs(x)
        for root in sorted({0, p - 1, p // 2}):
            for proto in PROTOS + ["auto"]:
                say(f"broadcast/reduce P={p} {dtype} n={n} root={root} {proto}")
                check_ok(reg.broadcast(n, root, proto), "broadcast")
                got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
                assert_bits_equal(got, oracle.broadcast(x, root), f"broadcast {proto} root={root} n={n}")
                check_ok(reg.reduce(n, root, proto), "reduce")
                got = reg.read_out(n, NP[dtype]).reshape(1, n)
                assert_bits_equal(got, oracle.reduce(x, root).reshape(1, n), f"reduce {proto} root={root} n={n}")
    assert (reg.read_area(4) == SENT).all()


def test_broadcast_reduce_compose_to_allreduce():
    """Reduce to a root, then Broadcast of the root's result, equals AllReduce."""
    p, n = 8, 30_000
    x = wl.adversarial(p, n, seed=4)
    reg = SymRegion(p, n, "bf16")
    reg.init()
    reg.write_inputs(x)
    check_ok(reg.reduce(n, 5, "line128"), "reduce")
    red = reg.read_out(n, np.uint16)
    reg.write_inputs(np.tile(red, (p, 1)))
    check_ok(reg.broadcast(n, 5, "packet8"), "broadcast")
    assert_bits_equal(reg.read_out(p * n, np.uint16).reshape(p, n), oracle.allreduce(x), "reduce+broadcast")


@pytest.mark.parametrize("p", [2, 5, 8])
def test_rooted_auto_with_sentinel_allowed(p):
    """Broadcast and Reduce under AUTO with sentinel units allowed (the
    one-tile sentinel kernel up to 64 KiB, lines above), every root, two
    calls per size; the sentinel slots are back to the sentinel afterwards."""
    sizes = [1000, 8192, 32768, 100_000]
    reg = SymRegion(p, max(sizes), "bf16")
    reg.init()
    sent = opts(flags=ll.LL_OPT_AUTO_SENTINEL)
    for n in sizes:
        for root in range(p):
            for call in range(2):
                x = wl.normal(p, n, "bf16", seed=n + 10 * root + call)
                reg.write_inputs(x)
                say(f"rooted auto+sentinel P={p} n={n} root={root} call {call}")
                check_ok(reg.broadcast(n, root, "auto", opt=sent), "broadcast")
                assert_bits_equal(reg.read_out(p * n, np.uint16).reshape(p, n), oracle.broadcast(x, root),
                                  f"broadcast P={p} n={n} root={root}")
                check_ok(reg.reduce(n, root, "auto", opt=sent), "reduce")
                assert_bits_equal(reg.read_out(n, np.uint16).reshape(1, n), oracle.reduce(x, root).reshape(1, n),
                                  f"reduce P={p} n={n} root={root}")
    assert (reg.read_area(4) == SENT).all()


@pytest.mark.parametrize("kind", ["broadcast", "reduce"])
def test_rooted_missing_rank_times_out(kind):
    p, n = 8, 4096
    x = wl.uniform(p, n, "f32", seed=6)
    reg = SymRegion(p, n, "f32")
    reg.init()
    reg.write_inputs(x)
    mute = opts(poll_timeout=MUTED_TIMEOUT_TICKS, mute_rank=2 if kind == "broadcast" else 6)  # root, or contributor
    st = reg.broadcast(n, 2, "packet8", opt=mute) if kind == "broadcast" else reg.reduce(n, 2, "packet8", opt=mute)
    assert st == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    rank, missing, _ = ll.ll_last_timeout()
    assert missing == (1 << (2 if kind == "broadcast" else 6))
    reg.init()
    check_ok(reg.reduce(n, 2, "packet8"), "after timeout")
    assert_bits_equal(reg.read_out(n, np.uint32).reshape(1, n), oracle.reduce(x, 2).reshape(1, n), "after timeout")


@pytest.mark.parametrize("proto", ["packet8", "sentinel", "line128"])
def test_rs_ag_wave_kernels_launch_shapes_and_timeouts(proto):
    """The wave-per-peer ReduceScatter / AllGather at several workgroup counts
    and units per lane, then a muted rank that makes the waits expire."""
    p, m = 8, 40_000
    x = wl.normal(p, p * m, "bf16", seed=17)
    reg = SymRegion(p, p * m, "bf16", out_elems=p * p * m)
    reg.init()
    for wg in (1, 3, 0):
        for units in (1, 2, 4, 0):
            reg.opt = opts(wave_kernels=2, workgroups_per_rank=wg, wave_units=units)
            say(f"RS/AG waves {proto} wg={wg} units={units}")
            reg.write_inputs(x)
            check_ok(reg.reduce_scatter(m, proto), "rs")
            rs = reg.read_out(p * m, np.uint16).reshape(p, m)
            assert_bits_equal(rs, oracle.reduce_scatter(x), f"RS waves wg={wg} u={units}")
            reg.write_inputs(rs)
            check_ok(reg.allgather(m, proto), "ag")
            assert_bits_equal(reg.read_out(p * p * m, np.uint16).reshape(p, p * m), oracle.allgather(rs),
                              f"AG waves wg={wg} u={units}")
    reg.opt = opts(wave_kernels=2, poll_timeout=MUTED_TIMEOUT_TICKS, mute_rank=4)
    reg.write_inputs(x)
    assert reg.reduce_scatter(m, proto) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    assert reg.allgather(m, proto) == ll.LL_OK
    assert ll.ll_check(stream()) == ll.LL_ERR_TIMEOUT
    reg.opt = opts(wave_kernels=2)
    reg.init()
    reg.write_inputs(x)
    check_ok(reg.reduce_scatter(m, proto), "rs after timeout")
    assert_bits_equal(reg.read_out(p * m, np.uint16).reshape(p, m), oracle.reduce_scatter(x), "RS after timeout")
    if proto == "sentinel":
        assert (reg.read_area(4) == SENT).all()


# ------------------------------------------------ fallback off line packets
@pytest.mark.parametrize("p,n,dtype,sized_for", [(8, 4 * 8192, "bf16", "auto"), (8, 64 * 8192, "bf16", "auto"),
                                                 (4, 7168 * 16, "bf16", "auto"),
                                                 (8, 16 << 20, "f32", "twoshot")])
def test_no_lines_fallback_parity(p, n, dtype, sized_for):
    """LL_OPT_NO_LINES at the sizes where AUTO otherwise runs 128-byte lines
    (the 64 KiB line one-shot at 8 ranks, the 224 KiB line one-shot at 4,
    the 1 MiB line two-shot with one wave per peer, the 64 MiB line
    two-shot): AUTO takes the 8-byte-packet algorithm
    of the same shape, whose correctness rests on the 8-byte atomicity the
    memory model guarantees, and the result is the oracle's, bit for bit.  The
    64 MiB case runs on a region sized for 8-byte packets only."""
    es = 4 if dtype == "f32" else 2
    st, plain = ll.ll_auto_algo(n, ll.DTYPES[dtype], p)
    assert st == ll.LL_OK and "line" in [k for k, v in ll.ALGOS.items() if v == plain][0]
    opt = opts(flags=ll.LL_OPT_NO_LINES)
    reg = SymRegion(p, n, dtype, sized_for=sized_for, out_elems=p * n, opt=opt)
    st, chosen = ll.ll_auto_algo(n, ll.DTYPES[dtype], p, reg.rank_stride, opt)
    name = [k for k, v in ll.ALGOS.items() if v == chosen][0]
    assert st == ll.LL_OK and "line" not in name and "sentinel" not in name
    reg.init()
    x = wl.uniform(p, n, dtype, seed=21) if dtype == "f32" else wl.normal(p, n, dtype, seed=21)
    for k in range(2):
        say(f"no-lines fallback P={p} n={n} {dtype} ({name}) call {k}")
        assert_bits_equal(run_allreduce(reg, x, "auto"), oracle.allreduce(x), f"no lines P={p} n={n} call {k}")
    if sized_for != "auto":
        assert reg.allreduce(n, "twoshot_line") == ll.LL_ERR_SCRATCH  # the region holds no line area
    del reg
    torch.cuda.empty_cache()
