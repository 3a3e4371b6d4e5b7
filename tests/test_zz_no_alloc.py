"""The entry point that allocates nothing (ll_allreduce_static): its output
equals that of ll_allreduce_buffered, the entry point it is a variant of, bit
for bit, on two calls in a row, the second with a smaller input.

This file is collected last (its name sorts after every other test file), so
that a failure here cannot hide the results of the others."""
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

NP = {"f32": np.uint32, "bf16": np.uint16}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def static_call(x, algo, in_place=False):
    """One ll_allreduce_static call on x ([P, n] element bits); returns the P outputs."""
    p, n = x.shape
    dt = ll.LL_F32 if x.dtype == np.uint32 else ll.LL_BF16
    inp = torch.from_numpy(np.ascontiguousarray(x).view(np.uint8).reshape(-1).copy()).cuda()
    out = inp if in_place else torch.empty_like(inp)
    s = torch.cuda.current_stream().cuda_stream
    st, used = ll.ll_allreduce_static(inp.data_ptr(), out.data_ptr(), n, dt, ll.LL_SUM, p, s, ll.ALGOS[algo])
    assert st == ll.LL_OK, ll.ll_strerror(st)
    assert ll.ll_check(s) == ll.LL_OK
    assert used >= 1
    return out.cpu().numpy().view(x.dtype).reshape(p, n), used


def buffered_call(x, algo):
    """The same AllReduce through ll_allreduce_buffered with a caller-allocated scratch."""
    p, n = x.shape
    dtype = "f32" if x.dtype == np.uint32 else "bf16"
    reg = ScratchRegion(p, n, dtype, iter_bytes=64 << 10)
    reg.init()
    reg.write_inputs(x)
    st = reg.allreduce(n, algo)
    assert st == ll.LL_OK, ll.ll_strerror(st)
    assert ll.ll_check(torch.cuda.current_stream().cuda_stream) == ll.LL_OK
    return reg.read_out(p * n, x.dtype).reshape(p, n)


CASES = [
    # (P, dtype, first n, second n, algorithm)
    (8, "bf16", 1_000_003, 8192, "auto"),
    (8, "bf16", 300_000, 4096, "twoshot_line"),
    (5, "f32", 250_001, 777, "auto"),
    (8, "f32", 40_000, 1000, "oneshot_waves"),
    (3, "bf16", 99_999, 5, "twoshot_waves"),
    (7, "f32", 123_457, 64, "oneshot_line"),
]


@pytest.mark.parametrize("p,dtype,n1,n2,algo", CASES)
def test_static_scratch_matches_buffered_entry_point(p, dtype, n1, n2, algo):
    for k, n in enumerate((n1, n2)):
        x = wl.normal(p, n, dtype, seed=1000 * k + n + p)
        if algo == "oneshot_waves" and n * x.itemsize > 64 << 10:
            algo_k = "auto"  # one-shot wave kernels run one iteration only
        else:
            algo_k = algo
        say(f"static P={p} {dtype} n={n} {algo_k} (call {k + 1})")
        got, used = static_call(x, algo_k)
        want = buffered_call(x, algo_k)
        assert np.array_equal(got, want), f"call {k + 1}: static and buffered outputs differ"
        assert np.array_equal(got, oracle.allreduce(x)), f"call {k + 1}: differs from the oracle"


def test_static_scratch_in_place_and_refusals():
    p, n = 8, 200_000
    x = wl.uniform(p, n, "bf16", seed=9)
    got, used = static_call(x, "auto", in_place=True)
    assert used > 1 and np.array_equal(got, oracle.allreduce(x))
    dummy = torch.zeros(64, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for algo in ("oneshot_sentinel", "twoshot_sentinel_waves", "twoshot_atomic"):
        st, _ = ll.ll_allreduce_static(dummy.data_ptr(), dummy.data_ptr(), 4, ll.LL_F32, ll.LL_SUM, p, s,
                                       ll.ALGOS[algo])
        assert st == ll.LL_ERR_UNSUPPORTED, algo
    st, _ = ll.ll_allreduce_static(dummy.data_ptr(), dummy.data_ptr(), (16 << 30) // 4 + 1, ll.LL_F32, ll.LL_SUM, p,
                                   s, ll.LL_ALGO_AUTO)
    assert st == ll.LL_ERR_UNSUPPORTED  # beyond the largest message
