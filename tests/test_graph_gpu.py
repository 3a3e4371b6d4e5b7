"""Library calls captured into a HIP graph: every replay, with new inputs and
the region reset between replays (a captured call keeps its epoch), matches
the CPU oracle bit for bit, for one-shot and two-shot algorithms in every
packet format, the one-lane kernels and the bounded-scratch path."""
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
CALLS = 12


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("algo,n,dtype", [
    ("oneshot_waves", 8192, "bf16"),
    ("oneshot_line_waves", 16384, "bf16"),
    ("oneshot_sentinel_waves", 4096, "f32"),
    ("twoshot_line_waves", 131072, "bf16"),
    ("twoshot_waves", 65536, "f32"),
    ("oneshot", 1000, "f32"),
    ("twoshot_line", 20000, "bf16"),
    ("auto", 524288, "bf16"),
])
def test_replays_of_a_captured_region_call(algo, n, dtype):
    p = 8
    reg = SymRegion(p, n, dtype)
    reg.init()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):  # lazy set-up and the stream's status word, before capture
        reg.write_inputs(wl.normal(p, n, dtype, seed=1))
        assert reg.allreduce(n, algo) == ll.LL_OK
    torch.cuda.synchronize()
    assert ll.ll_check(side.cuda_stream) == ll.LL_OK
    reg.init(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for i in range(CALLS):
            assert reg.allreduce(n, algo, epoch=1 + i) == ll.LL_OK
    torch.cuda.synchronize()
    for rep in range(3):
        x = wl.normal(p, n, dtype, sigma=float(10.0 ** (rep - 1)), seed=100 + rep)
        say(f"{algo} n={n} {dtype}: replay {rep}")
        reg.write_inputs(x)
        reg.init()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert ll.ll_check(side.cuda_stream) == ll.LL_OK
        assert ll.ll_check(torch.cuda.current_stream().cuda_stream) == ll.LL_OK
        got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
        assert np.array_equal(got, oracle.allreduce(x)), f"{algo} replay {rep}"


@pytest.mark.parametrize("algo", ["auto", "twoshot_line_waves", "oneshot_line"])
def test_replays_of_a_captured_bounded_scratch_call(algo):
    p, dtype = 6, "bf16"
    reg = ScratchRegion(p, 100_000, dtype, iter_bytes=16384)
    reg.init()
    n = 3 * (reg.iter_bytes // 2) + 77  # four iterations, the last one ragged
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        reg.write_inputs(wl.normal(p, n, dtype, seed=2))
        assert reg.allreduce(n, algo) == ll.LL_OK
    torch.cuda.synchronize()
    assert ll.ll_check(side.cuda_stream) == ll.LL_OK
    reg.init(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for _ in range(4):
            assert reg.allreduce(n, algo) == ll.LL_OK
    torch.cuda.synchronize()
    for rep in range(3):
        x = wl.normal(p, n, dtype, seed=200 + rep)
        say(f"buffered {algo}: replay {rep}")
        reg.write_inputs(x)
        reg.init()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert ll.ll_check(side.cuda_stream) == ll.LL_OK
        got = reg.read_out(p * n, NP[dtype]).reshape(p, n)
        assert np.array_equal(got, oracle.allreduce(x)), f"buffered {algo} replay {rep}"
