"""GPU checks of the chip facts the packet formats rely on, and of the
measurement probes (all bounded; nothing here can wait forever)."""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_16100_amd import llcoll as ll  # noqa: E402


def stream():
    return torch.cuda.current_stream().cuda_stream


def test_workgroups_are_dealt_round_robin_over_xcds():
    """Consecutive workgroups run on consecutive XCDs: workgroup b runs on XCD
    (b + s) mod 8, where s, the XCD of workgroup 0, may differ from launch to
    launch.  So rank r = b mod P of an 8-rank launch owns one XCD and every
    rank-to-rank packet crosses the fabric."""
    grid = 256
    ids = torch.full((grid,), 99, dtype=torch.int32, device="cuda")
    assert ll.ll_probe_xcd(ids.data_ptr(), grid, 64, stream()) == ll.LL_OK
    torch.cuda.synchronize()
    x = ids.cpu().numpy()
    nx = int(x.max()) + 1
    print("XCDs seen:", nx, "first 16:", x[:16].tolist(), flush=True)
    assert nx == 8
    assert np.array_equal(x, (np.arange(grid) + x[0]) % 8)


@pytest.mark.parametrize("size", ["short", "long"])
@pytest.mark.parametrize("layout,name", [(0, "8-byte packets"), (1, "128-byte lines, flag per 64-byte half")])
def test_no_torn_packets_across_xcds(layout, name, size):
    """Writers on one XCD rewrite packets while readers on another XCD read
    them: every unit whose flag is set must carry that round's payload.  The
    long run (256 writer and 256 reader workgroups, writers rewriting their
    lines a million times while the readers read 50,000 times) takes about
    1.2 s per layout."""
    grid, lines, iters, reads = (16, 256, 3000, 3000) if size == "short" else (512, 256, 1_000_000, 50_000)
    buf = torch.zeros(grid // 2 * lines * 32, dtype=torch.int32, device="cuda")
    counts = torch.zeros(4, dtype=torch.int64, device="cuda")
    st = ll.ll_probe_litmus(buf.data_ptr(), buf.numel() * 4, grid, lines, iters, reads, layout,
                            counts.data_ptr(), stream())
    assert st == ll.LL_OK
    torch.cuda.synchronize()
    seen, torn, split16, splitline = counts.cpu().numpy().tolist()
    print(f"litmus {name} ({size}): seen={seen} torn={torn} split16={split16} splitline={splitline}", flush=True)
    assert seen > (100_000 if size == "short" else 1_000_000_000)
    assert torn == 0


def test_floor_and_empty_kernels_run():
    words = 1 << 20
    chase = torch.zeros(words, dtype=torch.int64, device="cuda")
    sink = torch.zeros(4, dtype=torch.int64, device="cuda")
    stamps = torch.zeros(2 * 64, dtype=torch.int64, device="cuda")
    assert ll.ll_probe_empty(64, 256, stamps.data_ptr(), stream()) == ll.LL_OK
    assert ll.ll_probe_floor(chase.data_ptr(), words, 4096, sink.data_ptr(), 64, 256, stamps.data_ptr(),
                             stream()) == ll.LL_OK
    torch.cuda.synchronize()
    s = stamps.cpu().numpy()
    assert np.all(s[64:] >= s[:64]) and np.all(s > 0)


def test_pingpong_completes():
    flags = torch.zeros(2048, dtype=torch.int32, device="cuda")
    out = torch.zeros(3, dtype=torch.int64, device="cuda")
    assert ll.ll_probe_pingpong(flags.data_ptr(), 500, 8, 1, 10_000_000, out.data_ptr(), stream()) == ll.LL_OK
    torch.cuda.synchronize()
    ticks, done, cycles = out.cpu().numpy().tolist()
    print(f"pingpong: {done} rounds, {ticks * 10 / max(done, 1):.0f} ns per round", flush=True)
    assert done == 500


@pytest.mark.parametrize("grid", [1, 7, 512])
def test_streaming_probe_moves_exactly_its_bytes(grid):
    """The streaming probe copies src to dst word for word (mode 0), leaves dst
    alone when it only reads (mode 1), writes its fill pattern (mode 2), and
    stops at `bytes`, with grids smaller and larger than the word count."""
    nbytes = 16 * 1000 + 16 * 37
    n16 = nbytes // 16
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    src = torch.randint(-2**31, 2**31 - 1, (n16 * 4,), dtype=torch.int32, device="cuda", generator=g)
    dst = torch.full((n16 * 4 + 64,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    guard = dst[n16 * 4:].clone()
    before = dst.clone()
    assert ll.ll_probe_stream(src.data_ptr(), dst.data_ptr(), nbytes, 1, grid, 256, stream()) == ll.LL_OK
    torch.cuda.synchronize()
    assert torch.equal(dst, before)
    assert ll.ll_probe_stream(src.data_ptr(), dst.data_ptr(), nbytes, 0, grid, 256, stream()) == ll.LL_OK
    torch.cuda.synchronize()
    assert torch.equal(dst[:n16 * 4], src)
    assert torch.equal(dst[n16 * 4:], guard)
    assert ll.ll_probe_stream(0, dst.data_ptr(), nbytes, 2, grid, 256, stream()) == ll.LL_OK
    torch.cuda.synchronize()
    words = dst[:n16 * 4].view(n16, 4).cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    assert np.array_equal(words[:, 0], np.arange(n16))
    assert (words[:, 1] == 1).all() and (words[:, 2] == 2).all() and (words[:, 3] == 3).all()
    assert torch.equal(dst[n16 * 4:], guard)
