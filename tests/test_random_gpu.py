"""GPU parity over a seeded random sample of calls: every collective, packet
format, algorithm and per-call option, at random rank counts, element types
and sizes (ragged, unaligned and multi-tile), several calls per region so that
the epochs advance across algorithms.  Each result is compared bit for bit
with the CPU oracle (0 ulp; binary32 accumulation in ascending rank order, one
rounding).
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
    from paper_2607_16100_amd.region import SymRegion  # noqa: E402
else:  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

NP = {"f32": np.uint32, "bf16": np.uint16}
AR_ALGOS = ["auto", "oneshot", "twoshot", "twoshot_line", "oneshot_line", "oneshot_waves", "oneshot_sentinel",
            "twoshot_sentinel", "twoshot_waves", "twoshot_sentinel_waves", "oneshot_sentinel_waves",
            "oneshot_line_waves", "twoshot_line_waves", "twoshot_sentinel_out"]
ONE_LANE = {"oneshot", "twoshot", "twoshot_line", "oneshot_line", "oneshot_sentinel", "twoshot_sentinel",
            "twoshot_sentinel_out"}
PROTOS = ["auto", "packet8", "line128", "sentinel"]
KINDS = ["allreduce"] * 5 + ["reduce_scatter", "allgather", "broadcast", "reduce"]
MAX_N = 1 << 18  # elements per rank (the regions' input capacity)
TIMEOUT_TICKS = 20_000_000  # 200 ms per flag wait
CASES = 600


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def log_uniform(rng, lo, hi):
    return int(np.exp(rng.uniform(np.log(lo), np.log(hi + 1)))) if hi > lo else lo


def random_options(rng, kind, algo):
    """Per-call options: flags for AUTO and random launch-shape fields."""
    kw = {"poll_timeout": TIMEOUT_TICKS}
    flags = 0
    if rng.random() < 0.3:
        flags |= ll.LL_OPT_AUTO_SENTINEL
    if rng.random() < 0.15:
        flags |= ll.LL_OPT_NO_LINES
    kw["flags"] = flags
    tuning = {}
    if rng.random() < 0.3:
        tuning["wave_units"] = int(rng.choice([1, 2, 4]))
    if rng.random() < 0.3:
        tuning["clear_slots"] = int(rng.integers(0, 3))
    if kind == "allreduce" and rng.random() < 0.2:
        tuning["pipeline_lag"] = int(rng.integers(0, 5))
    if kind in ("reduce_scatter", "allgather") and rng.random() < 0.3:
        tuning["wave_kernels"] = int(rng.integers(0, 3))
    if rng.random() < 0.15:
        tuning["workgroups_per_rank"] = int(rng.choice([1, 3, 16, 64]))
    if algo in ONE_LANE and rng.random() < 0.15:
        tuning["threads"] = int(rng.choice([64, 256, 1024]))
    if rng.random() < 0.1:
        tuning["first_wait"] = int(rng.integers(0, 4))
        tuning["poll_gap"] = int(rng.integers(0, 4))
    return ll.Options(**kw, **tuning)


def make_cases(seed=20261202):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(CASES):
        p = int(rng.integers(2, 9))
        dtype = str(rng.choice(["f32", "bf16"]))
        kind = str(rng.choice(KINDS))
        algo = str(rng.choice(AR_ALGOS)) if kind == "allreduce" else str(rng.choice(PROTOS))
        if kind == "allreduce":
            n = log_uniform(rng, 1, (1 << 16) if algo in ONE_LANE else MAX_N)
            if algo == "twoshot_sentinel_out":  # its outputs are filled in 16-byte units
                k = 4 if dtype == "f32" else 8
                n = (n + k - 1) // k * k
        elif kind == "reduce_scatter":
            n = log_uniform(rng, 1, MAX_N // p)
        elif kind == "allgather":
            n = log_uniform(rng, 1, (1 << 15) // p)
        else:
            n = log_uniform(rng, 1, 1 << 17)
        root = int(rng.integers(0, p))
        cases.append((p, dtype, kind, algo, n, root, i))
    cases.sort(key=lambda c: (c[0], c[1], c[6]))
    return cases, rng


def run_case(reg, rng, p, dtype, kind, algo, n, root, i):
    x_n = p * n if kind == "reduce_scatter" else n
    x = wl.normal(p, x_n, dtype, sigma=float(rng.choice([0.01, 1.0, 300.0])), seed=1000 + i)
    reg.write_inputs(x)
    opt = random_options(rng, kind, algo if kind == "allreduce" else "")
    what = f"case {i}: {kind} {algo} P={p} {dtype} n={n} root={root}"
    say(what)
    if kind == "allreduce":
        st = reg.allreduce(n, algo, opt=opt)
    elif kind == "reduce_scatter":
        st = reg.reduce_scatter(n, algo, opt=opt)
    elif kind == "allgather":
        st = reg.allgather(n, algo, opt=opt)
    elif kind == "broadcast":
        st = reg.broadcast(n, root, algo, opt=opt)
    else:
        st = reg.reduce(n, root, algo, opt=opt)
    assert st == ll.LL_OK, f"{what}: {ll.ll_strerror(st)}"
    st2 = ll.ll_check(torch.cuda.current_stream().cuda_stream)
    assert st2 == ll.LL_OK, f"{what}: ll_check says {ll.ll_strerror(st2)}"
    if kind == "allreduce":
        got, want = reg.read_out(p * n, NP[dtype]).reshape(p, n), oracle.allreduce(x)
    elif kind == "reduce_scatter":
        got, want = reg.read_out(p * n, NP[dtype]).reshape(p, n), oracle.reduce_scatter(x)
    elif kind == "allgather":
        got, want = reg.read_out(p * p * n, NP[dtype]).reshape(p, p * n), oracle.allgather(x)
    elif kind == "broadcast":
        got, want = reg.read_out(p * n, NP[dtype]).reshape(p, n), oracle.broadcast(x, root)
    else:
        got, want = reg.read_out(n, NP[dtype]).reshape(1, n), oracle.reduce(x, root).reshape(1, n)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        r, j = bad[0]
        raise AssertionError(f"{what}: {len(bad)} elements differ; first at row {r} index {j}: "
                             f"got {int(got[r, j]):#x} want {int(want[r, j]):#x}")


def test_random_calls_match_the_oracle():
    """600 seeded random calls on one region per (rank count, element type)."""
    cases, rng = make_cases()
    groups = {}
    for c in cases:
        groups.setdefault((c[0], c[1]), []).append(c)
    for (p, dtype), group in sorted(groups.items()):
        reg = SymRegion(p, MAX_N, dtype, out_elems=p * max(MAX_N, p * (1 << 15)))
        reg.init()
        for c in group:
            run_case(reg, rng, *c)
        del reg
        torch.cuda.empty_cache()


BUF_ALGOS = ["auto", "oneshot", "oneshot_line", "oneshot_sentinel", "twoshot", "twoshot_line", "twoshot_sentinel",
             "twoshot_sentinel_out", "twoshot_waves", "twoshot_sentinel_waves", "twoshot_line_waves"]


def test_random_bounded_scratch_calls_match_the_oracle():
    """The bounded-scratch AllReduce (ll_allreduce_buffered) over 40 random
    regions (rank count, element type, iteration size, in place or not), five
    random calls each: one to several iterations with ragged last ones, every
    algorithm and random per-call options."""
    from paper_2607_16100_amd.region import ScratchRegion

    rng = np.random.default_rng(7_2026)
    for g in range(40):
        p = int(rng.integers(2, 9))
        dtype = str(rng.choice(["f32", "bf16"]))
        es = 4 if dtype == "f32" else 2
        iter_bytes = int(rng.choice([4096, 16384, 65536, 262144]))
        in_place = bool(rng.random() < 0.4)
        max_count = 6 * iter_bytes // es
        reg = ScratchRegion(p, max_count, dtype, iter_bytes=iter_bytes, in_place=in_place)
        reg.init()
        d = reg.iter_bytes // es
        for c in range(5):
            if rng.random() < 0.4:
                n = log_uniform(rng, 1, d)
            else:  # one to five iterations, the last one ragged
                n = min(max_count, int(d * rng.uniform(1.0, 5.9)))
            algo = str(rng.choice(BUF_ALGOS))
            if algo == "twoshot_sentinel_out":
                if in_place:  # its output is filled with the sentinel before the call
                    algo = "twoshot_sentinel"
                else:
                    k = 16 // es
                    n = min(max_count, (n + k - 1) // k * k)
            x = wl.normal(p, n, dtype, sigma=float(rng.choice([0.01, 1.0, 300.0])), seed=50_000 + 10 * g + c)
            want = oracle.allreduce(x)
            reg.write_inputs(x)
            opt = random_options(rng, "allreduce", algo)
            what = f"group {g} call {c}: buffered {algo} P={p} {dtype} n={n} iteration {reg.iter_bytes} B in_place={in_place}"
            say(what)
            st = reg.allreduce(n, algo, opt=opt)
            assert st == ll.LL_OK, f"{what}: {ll.ll_strerror(st)}"
            st2 = ll.ll_check(torch.cuda.current_stream().cuda_stream)
            assert st2 == ll.LL_OK, f"{what}: ll_check says {ll.ll_strerror(st2)}"
            got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
            if not np.array_equal(got, want):
                bad = np.argwhere(got != want)
                r, j = bad[0]
                raise AssertionError(f"{what}: {len(bad)} elements differ; first at row {r} index {j}: "
                                     f"got {int(got[r, j]):#x} want {int(want[r, j]):#x}")
        del reg
        torch.cuda.empty_cache()
