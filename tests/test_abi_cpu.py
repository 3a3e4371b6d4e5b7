"""The C-ABI library on the CPU: it loads, exports what the headers declare, and
rejects bad arguments before touching the HIP runtime (no GPU needed)."""
from __future__ import annotations

import os
import re

import pytest

from paper_2607_16100_amd import llcoll as ll

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("llcoll.h", "llprobe.h", "lltune.h")]

F32, BF16 = ll.LL_F32, ll.LL_BF16
GOOD_BASE = 1 << 40          # fake, 256-aligned device addresses: never dereferenced
GOOD_OUT = 1 << 41


def declared_functions():
    names = []
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(ll_[a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_headers_declare_the_boundary():
    names = declared_functions()
    for must in ("ll_slice_bytes", "ll_init", "ll_allreduce", "ll_allreduce_algo", "ll_reduce_scatter",
                 "ll_allgather", "ll_check", "ll_strerror", "ll_probe_empty", "ll_probe_floor"):
        assert must in names


def test_library_exports_every_declared_symbol():
    lib = ll.library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(ll.exported_symbols())


def stride_for(count, dt, p):
    st, s = ll.ll_slice_bytes(count, dt, p)
    assert st == ll.LL_OK
    return s


def ar(count=1024, dt=F32, p=4, base=GOOD_BASE, stride=None, out=GOOD_OUT, epoch=1, op=ll.LL_SUM,
       algo=ll.LL_ALGO_ONESHOT):
    if stride is None:
        stride = stride_for(max(count, 1), dt if dt in (F32, BF16) else F32, p if 2 <= p <= 8 else 2)
    return ll.ll_allreduce_algo(base, stride, out, count, dt, op, p, epoch, 0, algo)


@pytest.mark.parametrize("kwargs,want", [
    (dict(base=0), ll.LL_ERR_INVALID),
    (dict(out=0), ll.LL_ERR_INVALID),
    (dict(p=1), ll.LL_ERR_INVALID),
    (dict(p=9), ll.LL_ERR_INVALID),
    (dict(base=GOOD_BASE + 128), ll.LL_ERR_INVALID),
    (dict(out=GOOD_OUT + 8), ll.LL_ERR_INVALID),
    (dict(stride=1000), ll.LL_ERR_INVALID),
    (dict(epoch=0), ll.LL_ERR_INVALID),
    (dict(dt=7), ll.LL_ERR_UNSUPPORTED),
    (dict(op=1), ll.LL_ERR_UNSUPPORTED),
    (dict(algo=15), ll.LL_ERR_INVALID),
    (dict(algo=9, count=1001), ll.LL_ERR_UNSUPPORTED),  # atomic two-shot: count*esize % 16 == 0
    (dict(algo=8, count=1001), ll.LL_ERR_UNSUPPORTED),  # direct output needs count*esize % 16 == 0
    (dict(algo=-1), ll.LL_ERR_INVALID),
    (dict(stride=256), ll.LL_ERR_SCRATCH),
    (dict(count=1 << 29, stride=1 << 20), ll.LL_ERR_UNSUPPORTED),
    (dict(out=GOOD_BASE + 512), ll.LL_ERR_INVALID),   # out overlaps the region
    (dict(count=0), ll.LL_OK),                        # nothing to do, no launch
])
def test_allreduce_argument_checks(kwargs, want):
    assert ar(**kwargs) == want


def test_scratch_error_when_input_exceeds_capacity():
    stride = stride_for(1000, F32, 8)
    cap = ll.ll_input_capacity(stride, 8)[1]
    assert ar(count=cap // 4 + 1, p=8, stride=stride) == ll.LL_ERR_SCRATCH
    assert ar(count=100000, p=8, stride=stride) == ll.LL_ERR_SCRATCH


def test_rs_ag_argument_checks():
    stride = stride_for(8 * 64, BF16, 8)
    rs = ll.ll_reduce_scatter_ex
    ag = ll.ll_allgather_ex
    assert rs(GOOD_BASE, stride, GOOD_OUT, 64, BF16, ll.LL_SUM, 8, 0, 0, 0) == ll.LL_ERR_INVALID
    assert rs(GOOD_BASE, stride, GOOD_OUT, 64, BF16, 3, 8, 1, 0, 0) == ll.LL_ERR_UNSUPPORTED
    assert rs(GOOD_BASE, stride, GOOD_OUT, 64, BF16, ll.LL_SUM, 8, 1, 0, 5) == ll.LL_ERR_INVALID
    assert rs(GOOD_BASE, stride, GOOD_OUT, 65, BF16, ll.LL_SUM, 8, 1, 0, 0) == ll.LL_ERR_SCRATCH
    assert rs(GOOD_BASE, stride, GOOD_OUT, 0, BF16, ll.LL_SUM, 8, 1, 0, 0) == ll.LL_OK
    assert ag(GOOD_BASE, stride, GOOD_OUT, 8 * 64 + 1, BF16, 8, 1, 0, 0) == ll.LL_ERR_SCRATCH
    assert ag(GOOD_BASE, stride, 0, 64, BF16, 8, 1, 0, 0) == ll.LL_ERR_INVALID
    assert ag(GOOD_BASE, stride, GOOD_OUT, 0, BF16, 8, 1, 0, 0) == ll.LL_OK


def test_fill_sentinel_and_auto_sentinel_argument_checks():
    assert ll.ll_fill_sentinel(0, 16, F32, 4, 0) == ll.LL_ERR_INVALID
    assert ll.ll_fill_sentinel(GOOD_OUT + 8, 16, F32, 4, 0) == ll.LL_ERR_INVALID
    assert ll.ll_fill_sentinel(GOOD_OUT, 16, F32, 9, 0) == ll.LL_ERR_INVALID
    assert ll.ll_fill_sentinel(GOOD_OUT, 16, 4, 4, 0) == ll.LL_ERR_UNSUPPORTED
    assert ll.ll_fill_sentinel(GOOD_OUT, 0, BF16, 4, 0) == ll.LL_OK


@pytest.mark.parametrize("p", [2, 4, 8])
def test_scratch_sizing_round_trips(p):
    for d in [1, 256, 4096, 5000, 1 << 20, 64 << 20]:
        st, stride = ll.ll_scratch_bytes(d, p)
        assert st == ll.LL_OK and stride % 256 == 0
        st, it = ll.ll_scratch_iter_bytes(stride, p)
        assert st == ll.LL_OK and it >= d and it % 256 == 0
        assert ll.ll_scratch_iter_bytes(stride - 256, p)[1] < it  # minimal
    assert ll.ll_scratch_bytes(0, p)[0] == ll.LL_ERR_INVALID
    assert ll.ll_scratch_bytes((256 << 20) + 1, p)[0] == ll.LL_ERR_INVALID
    assert ll.ll_scratch_iter_bytes(256, p)[0] == ll.LL_ERR_SCRATCH
    assert ll.ll_scratch_iter_bytes(1000, p)[0] == ll.LL_ERR_INVALID


def test_buffered_argument_checks():
    stride = ll.ll_scratch_bytes(4096, 4)[1]
    scr = 1 << 42
    IN, OUT = GOOD_BASE, GOOD_OUT

    def b(inp=IN, out=OUT, count=4096, dt=F32, op=0, p=4, base=scr, s=stride, epoch=1, algo=0):
        return ll.ll_allreduce_buffered(inp, out, count, dt, op, p, base, s, epoch, 0, algo, None)

    assert b(inp=0)[0] == ll.LL_ERR_INVALID
    assert b(out=OUT + 8)[0] == ll.LL_ERR_INVALID
    assert b(base=scr + 64)[0] == ll.LL_ERR_INVALID
    assert b(epoch=0)[0] == ll.LL_ERR_INVALID
    assert b(p=1)[0] == ll.LL_ERR_INVALID
    assert b(op=1)[0] == ll.LL_ERR_UNSUPPORTED
    assert b(algo=15)[0] == ll.LL_ERR_INVALID
    assert b(algo=ll.LL_ALGO_ONESHOT_LINE_WAVES, count=1 << 20)[0] == ll.LL_ERR_UNSUPPORTED  # one iteration only
    assert b(algo=ll.LL_ALGO_TWOSHOT_ATOMIC)[0] == ll.LL_ERR_UNSUPPORTED
    assert b(s=256)[0] == ll.LL_ERR_SCRATCH
    assert b(out=IN + 16)[0] == ll.LL_ERR_INVALID            # partial overlap of in and out
    assert b(out=scr + 4096)[0] == ll.LL_ERR_INVALID         # output inside the scratch region
    assert b(algo=ll.LL_ALGO_ONESHOT_WAVES, count=1 << 20)[0] == ll.LL_ERR_UNSUPPORTED  # waves: one iteration
    assert b(algo=ll.LL_ALGO_TWOSHOT_SENTINEL_OUT, out=IN)[0] == ll.LL_ERR_INVALID
    assert b(algo=ll.LL_ALGO_TWOSHOT_SENTINEL_OUT, count=1001)[0] == ll.LL_ERR_UNSUPPORTED
    assert b(epoch=0xFFFFFFFF, count=4096)[0] == ll.LL_ERR_INVALID  # 4 iterations would pass 2^32 - 1
    assert b(count=0) == (ll.LL_OK, 0)


def test_broadcast_reduce_argument_checks():
    stride = stride_for(1000, F32, 4)
    bc, rd = ll.ll_broadcast, ll.ll_reduce
    assert bc(GOOD_BASE, stride, GOOD_OUT, 1000, F32, 4, 4, 1, 0, 0) == ll.LL_ERR_INVALID   # root >= P
    assert bc(GOOD_BASE, stride, GOOD_OUT, 1000, F32, -1, 4, 1, 0, 0) == ll.LL_ERR_INVALID
    assert bc(GOOD_BASE, stride, GOOD_OUT, 1000, F32, 0, 4, 0, 0, 0) == ll.LL_ERR_INVALID   # epoch 0
    assert bc(GOOD_BASE, stride, GOOD_OUT, 1000, F32, 0, 4, 1, 0, 4) == ll.LL_ERR_INVALID   # proto
    assert bc(GOOD_BASE, stride, GOOD_OUT, 100_000, F32, 0, 4, 1, 0, 0) == ll.LL_ERR_SCRATCH
    assert bc(GOOD_BASE, stride, GOOD_BASE + 256, 10, F32, 0, 4, 1, 0, 0) == ll.LL_ERR_INVALID  # out in region
    assert bc(GOOD_BASE, stride, GOOD_OUT, 0, F32, 0, 4, 1, 0, 0) == ll.LL_OK
    assert rd(GOOD_BASE, stride, GOOD_OUT, 1000, F32, 1, 0, 4, 1, 0, 0) == ll.LL_ERR_UNSUPPORTED  # op
    assert rd(GOOD_BASE, stride, GOOD_OUT, 1000, 3, 0, 0, 4, 1, 0, 0) == ll.LL_ERR_UNSUPPORTED   # dtype
    assert rd(GOOD_BASE, stride, GOOD_OUT, 1000, F32, 0, 9, 4, 1, 0, 0) == ll.LL_ERR_INVALID
    assert rd(GOOD_BASE, stride, GOOD_OUT, 0, F32, 0, 0, 4, 1, 0, 0) == ll.LL_OK


def test_init_argument_checks():
    assert ll.ll_init(0, 4096, 4, 0) == ll.LL_ERR_INVALID
    assert ll.ll_init(GOOD_BASE, 4096, 1, 0) == ll.LL_ERR_INVALID
    assert ll.ll_init(GOOD_BASE + 8, 4096, 4, 0) == ll.LL_ERR_INVALID
    assert ll.ll_init(GOOD_BASE, 256, 8, 0) == ll.LL_ERR_SCRATCH  # packet areas do not fit


@pytest.mark.parametrize("dt,es", [(F32, 4), (BF16, 2)])
@pytest.mark.parametrize("p", [2, 3, 4, 8])
def test_slice_bytes_gives_enough_capacity(dt, es, p):
    prev = 0
    for count in [1, 2, 3, 7, 64, 1000, 4096, 8192, 7168 * 16, 1 << 20, (64 << 20) // es]:
        st, stride = ll.ll_slice_bytes(count, dt, p)
        assert st == ll.LL_OK and stride % 4096 == 0  # every format: no format bits
        assert stride >= prev  # monotone in the input size
        prev = stride
        st, cap = ll.ll_input_capacity(stride, p)
        assert st == ll.LL_OK
        assert cap >= count * es and cap % 256 == 0
        # the region is not much larger than the input plus the slots it needs:
        # P-1 one-shot slots per area at 2x (8-byte packets), 128/120x (lines)
        # and 1x (sentinel) the input, plus per-slot rounding
        assert stride <= (1 + (p - 1) * (2 + 128 / 120 + 1) * 1.02 + 2.1) * max(cap, 256) + 8 * 1024 * p


def test_slice_bytes_argument_checks():
    assert ll.ll_slice_bytes(10, F32, 1)[0] == ll.LL_ERR_INVALID
    assert ll.ll_slice_bytes(10, 5, 4)[0] == ll.LL_ERR_UNSUPPORTED
    assert ll.ll_slice_bytes((256 << 20) // 4 + 1, F32, 4)[0] == ll.LL_ERR_UNSUPPORTED
    assert ll.ll_input_capacity(1000, 4)[0] == ll.LL_ERR_INVALID


@pytest.mark.parametrize("p", [2, 5, 8])
def test_slice_layout_areas_are_ordered_and_fit(p):
    for count in [1, 1000, 7168, 1 << 20]:
        stride = ll.ll_slice_bytes(count, F32, p)[1] + 4096
        st, offs = ll.ll_slice_layout(stride, p)
        assert st == ll.LL_OK
        assert offs[0] == 0 and offs[1] == ll.ll_input_capacity(stride, p)[1]
        assert all(a < b for a, b in zip(offs, offs[1:])) and offs[5] <= stride
        assert all(o % 256 == 0 for o in offs)
        # every 16-byte sentinel slot of one rank pair holds count*4 bytes
        assert offs[5] - offs[4] >= 2 * (p - 1) * ((count * 4 + p - 1) // p)
        assert offs[5] - offs[4] >= (p - 1) * count * 4
        # the accumulator holds a bfloat16 chunk in binary32, plus counters
        assert offs[4] - offs[3] >= 2 * ((count * 4 + p - 1) // p)
    assert ll.ll_slice_layout(1000, p)[0] == ll.LL_ERR_INVALID
    assert ll.ll_slice_layout(256, p)[0] == ll.LL_ERR_SCRATCH


def test_capacity_is_a_function_of_stride_and_ranks_only():
    # the layout (and with it every flag position) depends on nothing else
    for p in (2, 8):
        s = ll.ll_slice_bytes(5000, F32, p)[1]
        assert ll.ll_input_capacity(s, p) == ll.ll_input_capacity(s, p)
        assert ll.ll_input_capacity(s + 4096, p)[1] >= ll.ll_input_capacity(s, p)[1]


def test_options_are_checked_before_any_hip_call():
    stride = stride_for(1024, F32, 4)

    def call(opt):
        return ll.ll_allreduce_ex(GOOD_BASE, stride, GOOD_OUT, 1024, F32, ll.LL_SUM, 4, 1, 0, ll.LL_ALGO_ONESHOT, opt)

    bad = ll.Options()
    bad.o.size = 8  # not sizeof(ll_options)
    assert call(bad) == ll.LL_ERR_INVALID
    assert call(ll.Options(flags=0x80)) == ll.LL_ERR_INVALID  # unknown flag
    for field, value in [("workgroups_per_rank", -1), ("workgroups_per_rank", 5000), ("threads", 100),
                         ("threads", 2048), ("wave_units", 3), ("wave_kernels", 3), ("pipeline_lag", -2),
                         ("pipeline_lag", 65), ("first_wait", 1001), ("poll_gap", -1), ("mute_rank", 8),
                         ("mute_rank", -2), ("clear_slots", -1), ("clear_slots", 3)]:
        assert call(ll.Options(**{field: value})) == ll.LL_ERR_INVALID, (field, value)
    t = ll.Options(mute_rank=1)
    t.t.size = 4
    assert call(t) == ll.LL_ERR_INVALID
    # the same checks in the other entry points that take options
    assert ll.ll_reduce_scatter_ex(GOOD_BASE, stride, GOOD_OUT, 256, F32, ll.LL_SUM, 4, 1, 0, 0, bad) == \
        ll.LL_ERR_INVALID
    assert ll.ll_allgather_ex(GOOD_BASE, stride, GOOD_OUT, 256, F32, 4, 1, 0, 0, bad) == ll.LL_ERR_INVALID
    assert ll.ll_broadcast(GOOD_BASE, stride, GOOD_OUT, 256, F32, 0, 4, 1, 0, 0, bad) == ll.LL_ERR_INVALID
    assert ll.ll_auto_algo(1024, F32, 4, 0, bad)[0] == ll.LL_ERR_INVALID
    # well-formed options with nothing to do: no launch, success
    assert ll.ll_allreduce_ex(GOOD_BASE, stride, GOOD_OUT, 0, F32, ll.LL_SUM, 4, 1, 0, 0,
                              ll.Options(flags=ll.LL_OPT_NO_LINES, mute_rank=2, threads=128)) == ll.LL_OK


def test_no_setting_outlives_a_call():
    """The product header declares no function that changes what later calls
    do (the tuning and test hooks are per-call options in lltune.h), and a
    call's options do not change the choices of calls made without them."""
    text = open(os.path.join(ROOT, "include", "llcoll.h")).read()
    assert "ll_set_" not in text and "ll_debug_" not in text
    lib = ll.library()
    for name in ("ll_set_launch", "ll_set_auto_sentinel", "ll_set_poll_timeout", "ll_debug_mute_rank",
                 "ll_debug_stamp_next", "ll_last_grid"):
        assert not hasattr(lib, name), name
    A = ll.ALGOS
    defaults = [ll.ll_auto_algo(n, BF16, p) for p in (2, 4, 8) for n in (4096, 8192, 1 << 19, 1 << 24)]
    stride = stride_for(1 << 19, BF16, 8)
    for opt in (ll.Options(flags=ll.LL_OPT_AUTO_SENTINEL), ll.Options(flags=ll.LL_OPT_NO_LINES),
                ll.Options(flags=3, poll_timeout=5, mute_rank=3, threads=64, workgroups_per_rank=2, wave_units=4,
                           wave_kernels=1, pipeline_lag=0, clear_slots=2)):
        ll.ll_auto_algo(8192, BF16, 8, 0, opt)
        ll.ll_allreduce_ex(GOOD_BASE, stride, GOOD_OUT, 0, BF16, ll.LL_SUM, 8, 1, 0, 0, opt)  # count 0: no launch
    assert [ll.ll_auto_algo(n, BF16, p) for p in (2, 4, 8) for n in (4096, 8192, 1 << 19, 1 << 24)] == defaults
    assert ll.ll_auto_algo(8192, BF16, 8) == (ll.LL_OK, A["oneshot_waves"])


def test_strerror_covers_every_code():
    for code in (0, -1, -2, -3, -4, -5):
        assert ll.ll_strerror(code) and ll.ll_strerror(code) != "unknown status"
    assert ll.ll_strerror(42) == "unknown status"


def test_probe_argument_checks():
    assert ll.ll_probe_empty(0, 64, 0, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_empty(8, 100, 0, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_floor(0, 10, 0, GOOD_OUT, 8, 64, 0, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_floor(GOOD_BASE, 10, 10, GOOD_OUT, 8, 64, 0, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_litmus(GOOD_BASE, 1024, 16, 64, 1, 1, 0, GOOD_OUT, 0) == ll.LL_ERR_INVALID  # buffer too small
    assert ll.ll_probe_pingpong(GOOD_BASE, 10, 8, 8, 100, GOOD_OUT, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_stream(GOOD_BASE, GOOD_OUT, 1024, 3, 8, 64, 0) == ll.LL_ERR_INVALID  # no such mode
    assert ll.ll_probe_stream(GOOD_BASE, GOOD_OUT, 1000, 0, 8, 64, 0) == ll.LL_ERR_INVALID  # not 16-byte words
    assert ll.ll_probe_stream(GOOD_BASE, GOOD_OUT, 0, 0, 8, 64, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_stream(0, GOOD_OUT, 1024, 0, 8, 64, 0) == ll.LL_ERR_INVALID  # copy needs a source
    assert ll.ll_probe_stream(GOOD_BASE, 0, 1024, 2, 8, 64, 0) == ll.LL_ERR_INVALID
    assert ll.ll_probe_stream(GOOD_BASE + 8, GOOD_OUT, 1024, 0, 8, 64, 0) == ll.LL_ERR_INVALID  # misaligned
    assert ll.ll_probe_stream(GOOD_BASE, GOOD_OUT, 1024, 0, 8, 96, 0) == ll.LL_ERR_INVALID


def test_product_fails_loudly_without_the_library(tmp_path, monkeypatch):
    """No silent fallback: importing the binding with the library missing raises."""
    import importlib.util
    import shutil

    src = os.path.join(ROOT, "paper_2607_16100_amd", "llcoll.py")
    pkg = tmp_path / "fakepkg"
    pkg.mkdir()
    shutil.copy(src, pkg / "llcoll.py")
    spec = importlib.util.spec_from_file_location("fakepkg.llcoll", pkg / "llcoll.py")
    mod = importlib.util.module_from_spec(spec)
    with pytest.raises(ImportError):
        spec.loader.exec_module(mod)


def test_auto_algo_choices():
    """AUTO's choice (host logic only): the measured crossovers at the
    configurations' sizes, and one-way crossovers from one-shot to two-shot as
    messages grow."""
    A = ll.ALGOS
    f32, bf16 = ll.LL_F32, ll.LL_BF16
    assert ll.ll_auto_algo(4096, bf16, 8) == (ll.LL_OK, A["oneshot_waves"])            # 8 KiB
    assert ll.ll_auto_algo(8192, bf16, 8) == (ll.LL_OK, A["oneshot_waves"])            # C2, 16 KiB
    assert ll.ll_auto_algo(64 * 8192, bf16, 8) == (ll.LL_OK, A["twoshot_line_waves"])  # C3, 1 MiB
    assert ll.ll_auto_algo(16 << 20, f32, 8) == (ll.LL_OK, A["twoshot_line_waves"])    # C4, 64 MiB
    assert ll.ll_auto_algo(1024, f32, 4) == (ll.LL_OK, A["oneshot_waves"])             # C1
    sent = ll.Options(flags=ll.LL_OPT_AUTO_SENTINEL)
    assert ll.ll_auto_algo(8192, bf16, 8, 0, sent) == (ll.LL_OK, A["oneshot_sentinel_waves"])
    assert ll.ll_auto_algo(64 * 8192, bf16, 8, 0, sent) == (ll.LL_OK, A["twoshot_sentinel_waves"])
    assert ll.ll_auto_algo(16 << 20, f32, 8, 0, sent) == (ll.LL_OK, A["twoshot_line_waves"])
    assert ll.ll_auto_algo(16 << 20, f32, 6) == (ll.LL_OK, A["twoshot_line"])          # 64 MiB, 6 ranks
    assert ll.ll_auto_algo(2048, bf16, 8, 0, sent) == (ll.LL_OK, A["oneshot_waves"])     # 4 KiB: flags win
    assert ll.ll_auto_algo(2048, bf16, 2, 0, sent) == (ll.LL_OK, A["oneshot_sentinel_waves"])
    assert ll.ll_auto_algo(4 << 20, f32, 5) == (ll.LL_OK, A["twoshot_line_waves"])     # 16 MiB, 5 ranks
    assert ll.ll_auto_algo(8 << 20, f32, 5) == (ll.LL_OK, A["twoshot_line"])           # 32 MiB, 5 ranks
    # measured crossovers away from the configurations' sizes
    assert ll.ll_auto_algo(4 << 20, bf16, 8) == (ll.LL_OK, A["twoshot_line_waves"])           # 8 MiB
    assert ll.ll_auto_algo(2 * 8192, bf16, 8) == (ll.LL_OK, A["oneshot_line_waves"])         # 32 KiB
    assert ll.ll_auto_algo(4 * 8192, bf16, 8) == (ll.LL_OK, A["twoshot_line_waves"])         # 64 KiB
    assert ll.ll_auto_algo(1 << 19, bf16, 2) == (ll.LL_OK, A["oneshot_line_waves"])          # 1 MiB, 2 ranks
    assert ll.ll_auto_algo(1 << 20, bf16, 2) == (ll.LL_OK, A["oneshot_line_waves"])          # 2 MiB, 2 ranks
    assert ll.ll_auto_algo(1 << 19, bf16, 3) == (ll.LL_OK, A["twoshot_line_waves"])          # 1 MiB, 3 ranks
    assert ll.ll_auto_algo(1 << 16, bf16, 7, 0, sent) == (ll.LL_OK, A["twoshot_sentinel_waves"])  # 128 KiB
    assert ll.ll_auto_algo(64 * 8192, bf16, 8) == (ll.LL_OK, A["twoshot_line_waves"])        # 1 MiB
    assert ll.ll_auto_algo(1 << 20, bf16, 8, 0, sent) == (ll.LL_OK, A["twoshot_line_waves"])  # 2 MiB
    assert ll.ll_auto_algo(1 << 17, bf16, 3) == (ll.LL_OK, A["oneshot_line_waves"])          # 256 KiB
    assert ll.ll_auto_algo(4 << 20, bf16, 6) == (ll.LL_OK, A["twoshot_line_waves"])          # 8 MiB
    assert ll.ll_auto_algo(8 << 20, bf16, 6) == (ll.LL_OK, A["twoshot_line_waves"])          # 16 MiB
    assert ll.ll_auto_algo(16 << 20, bf16, 6) == (ll.LL_OK, A["twoshot_line"])               # 32 MiB
    assert ll.ll_auto_algo(8 << 20, bf16, 8) == (ll.LL_OK, A["twoshot_line_waves"])          # 16 MiB
    assert ll.ll_auto_algo(64 << 20, bf16, 7) == (ll.LL_OK, A["twoshot_line_waves"])         # 128 MiB
    assert ll.ll_auto_algo(1 << 19, bf16, 2, 0, sent) == (ll.LL_OK, A["oneshot_sentinel_waves"])
    assert ll.ll_auto_algo(1 << 20, bf16, 2, 0, sent) == (ll.LL_OK, A["oneshot_sentinel_waves"])  # 2 MiB
    assert ll.ll_auto_algo(3 << 19, bf16, 2, 0, sent) == (ll.LL_OK, A["twoshot_line_waves"])      # 3 MiB
    assert ll.ll_auto_algo(4 << 20, bf16, 2, 0, sent) == (ll.LL_OK, A["twoshot_sentinel_waves"])  # 8 MiB
    assert ll.ll_auto_algo(1, f32, 1)[0] == ll.LL_ERR_INVALID
    assert ll.ll_auto_algo(1, f32, 9)[0] == ll.LL_ERR_INVALID
    assert ll.ll_auto_algo(1, 7, 8)[0] == ll.LL_ERR_UNSUPPORTED
    names = {v: k for k, v in A.items()}
    for sentinel in (0, 1):
        opt = ll.Options(flags=ll.LL_OPT_AUTO_SENTINEL if sentinel else 0)
        for p in range(2, 9):
            for dt, es in ((f32, 4), (bf16, 2)):
                seen_twoshot = False
                for k in range(0, 29):
                    st, algo = ll.ll_auto_algo((1 << k) // es or 1, dt, p, 0, opt)
                    assert st == ll.LL_OK
                    name = names[algo]
                    assert name not in ("auto", "twoshot_sentinel_out", "twoshot_atomic")
                    if sentinel == 0:
                        assert "sentinel" not in name
                    if name.startswith("twoshot"):
                        seen_twoshot = True
                    else:
                        assert not seen_twoshot, f"P={p} {2**k} bytes: one-shot after two-shot"


def test_one_algorithm_regions():
    """ll_slice_bytes with a named algorithm sizes a region for that
    algorithm's packet format only: a stride with that format's bit, several
    times smaller than an every-format region at large sizes; calls in other
    formats are refused before any HIP call, and AUTO chooses inside the
    region's format."""
    A = ll.ALGOS
    fmt_of = {"oneshot": 1, "twoshot": 1, "oneshot_waves": 1, "twoshot_waves": 1, "twoshot_line": 2,
              "oneshot_line": 2, "oneshot_line_waves": 2, "twoshot_line_waves": 2, "oneshot_sentinel": 4,
              "twoshot_sentinel": 4, "twoshot_sentinel_out": 4, "twoshot_sentinel_waves": 4,
              "oneshot_sentinel_waves": 4, "twoshot_atomic": 8}
    for p in (2, 5, 8):
        for count, dt, es in ((8192, BF16, 2), (1 << 24, F32, 4), (1000, F32, 4)):
            full = ll.ll_slice_bytes(count, dt, p)[1]
            for name, f in fmt_of.items():
                st, stride = ll.ll_slice_bytes(count, dt, p, A[name])
                assert st == ll.LL_OK
                assert (stride // 256) % 16 == f, name          # the format bits
                assert ll.ll_input_capacity(stride, p)[1] >= count * es
                assert stride < full
                if count == 1 << 24 and p == 8:
                    # 8-byte packets need 15x the input, lines and sentinel units
                    # 8.5x and 8x, the atomic accumulators ~1.3x; all formats 29.5x
                    assert stride * (1.9 if f == 1 else 3.3) < full, name
                st, offs = ll.ll_slice_layout(stride, p)
                sizes = [offs[i + 1] - offs[i] for i in (1, 2, 3, 4)]  # 8-byte, line, atomic, sentinel areas
                present = [bool(f & 1), bool(f & 2), bool(f & 8), bool(f & 4)]
                assert [sz > 0 for sz in sizes] == present, name
                # a call in the region's format passes the checks (count 0: no launch); others are refused
                for other, g in fmt_of.items():
                    want = ll.LL_OK if g == f else ll.LL_ERR_SCRATCH
                    if other in ("twoshot_sentinel_out", "twoshot_atomic"):
                        continue  # their extra preconditions are tested elsewhere
                    got = ll.ll_allreduce_algo(GOOD_BASE, stride, GOOD_OUT, count, dt, ll.LL_SUM, p, 1, 0, A[other]) \
                        if g != f else ll.ll_allreduce_algo(GOOD_BASE, stride, GOOD_OUT, 0, dt, ll.LL_SUM, p, 1, 0,
                                                            A[other])
                    assert got == want, (name, other)
                if f in (1, 2):
                    st, auto = ll.ll_auto_algo(count, dt, p, stride)
                    assert st == ll.LL_OK and fmt_of[[k for k, v in A.items() if v == auto][0]] == f
    # proto-named calls follow the same rule
    stride = ll.ll_slice_bytes(7168, BF16, 8, A["twoshot_line"])[1]
    assert ll.ll_reduce_scatter_ex(GOOD_BASE, stride, GOOD_OUT, 896, BF16, ll.LL_SUM, 8, 1, 0,
                                   ll.LL_PROTO_PACKET8) == ll.LL_ERR_SCRATCH
    assert ll.ll_allgather_ex(GOOD_BASE, stride, GOOD_OUT, 896, BF16, 8, 1, 0, ll.LL_PROTO_SENTINEL) == \
        ll.LL_ERR_SCRATCH
    assert ll.ll_broadcast(GOOD_BASE, stride, GOOD_OUT, 7168, BF16, 0, 8, 1, 0, ll.LL_PROTO_PACKET8) == \
        ll.LL_ERR_SCRATCH
    assert ll.ll_slice_bytes(10, F32, 4, 15)[0] == ll.LL_ERR_INVALID


def test_no_lines_option_keeps_auto_off_line_packets():
    """LL_OPT_NO_LINES: at every size and rank count AUTO takes the
    8-byte-packet algorithm of the shape it would otherwise run with lines."""
    A = ll.ALGOS
    names = {v: k for k, v in A.items()}
    opt = ll.Options(flags=ll.LL_OPT_NO_LINES)
    for p in range(2, 9):
        for k in range(0, 29):
            n = (1 << k) // 4 or 1
            _, plain = ll.ll_auto_algo(n, ll.LL_F32, p)
            st, safe = ll.ll_auto_algo(n, ll.LL_F32, p, 0, opt)
            assert st == ll.LL_OK and "line" not in names[safe]
            assert names[safe] == names[plain].replace("_line", ""), (p, 1 << k, names[plain], names[safe])
    # a lines-only region has nothing AUTO may use with the option
    stride = ll.ll_slice_bytes(4096, ll.LL_F32, 8, A["twoshot_line"])[1]
    assert ll.ll_auto_algo(4096, ll.LL_F32, 8, stride, opt)[0] == ll.LL_ERR_SCRATCH


@pytest.mark.parametrize("p", [2, 3, 5, 6, 7, 8])
@pytest.mark.parametrize("dt,es", [(F32, 4), (BF16, 2)])
def test_iterations_tile_the_message_and_chunks_stay_inside(p, dt, es):
    """The iteration arithmetic every kernel uses: the iterations of a
    bounded-scratch call cover [0, count) exactly once, in order, and the P
    chunks of an iteration never reach past it (rank counts that do not
    divide the iteration included)."""
    for iter_bytes in (4096, 65536, 1 << 20):
        st, stride = ll.ll_scratch_bytes(iter_bytes, p)
        assert st == ll.LL_OK
        for count in (1, 5, 1000, iter_bytes // es, iter_bytes // es + 3, 7 * (iter_bytes // es) - 1, 123_457):
            st, iters, ic = ll.ll_buffered_plan(count, dt, p, stride)
            assert st == ll.LL_OK
            assert iters == -(-count // ic) and ic * es <= iter_bytes
            covered = 0
            for it in range(iters):
                st, (e0, n, chunk) = ll.ll_iteration_span(count, ic, it, p, dt)
                assert st == ll.LL_OK
                assert e0 == covered and n > 0
                covered += n
                assert (chunk * es) % 16 == 0 and chunk * p >= n
                ends = [min(max(n - c * chunk, 0), chunk) for c in range(p)]
                assert sum(ends) == n                      # the chunks partition the iteration
                assert all(ends[c] == 0 or c * chunk + ends[c] <= n for c in range(p))
            assert covered == count
            st, (e0, n, _) = ll.ll_iteration_span(count, ic, iters, p, dt)
            assert st == ll.LL_OK and n == 0               # nothing past the last iteration


def test_static_entry_point_argument_checks():
    """ll_allreduce_static rejects bad arguments before any HIP call."""
    good = dict(inp=GOOD_BASE, out=GOOD_OUT, count=1024, dt=F32, op=ll.LL_SUM, nranks=8, stream=0,
                algo=ll.LL_ALGO_AUTO)

    def call(**kw):
        a = dict(good, **kw)
        return ll.ll_allreduce_static(a["inp"], a["out"], a["count"], a["dt"], a["op"], a["nranks"], a["stream"],
                                      a["algo"])[0]

    assert call(inp=0) == ll.LL_ERR_INVALID
    assert call(out=GOOD_OUT + 8) == ll.LL_ERR_INVALID
    assert call(nranks=1) == ll.LL_ERR_INVALID and call(nranks=9) == ll.LL_ERR_INVALID
    assert call(dt=5) == ll.LL_ERR_UNSUPPORTED and call(op=2) == ll.LL_ERR_UNSUPPORTED
    assert call(algo=99) == ll.LL_ERR_INVALID
    for name in ("oneshot_sentinel", "twoshot_sentinel", "twoshot_sentinel_out", "twoshot_atomic",
                 "twoshot_sentinel_waves", "oneshot_sentinel_waves"):
        assert call(algo=ll.ALGOS[name]) == ll.LL_ERR_UNSUPPORTED, name
    assert call(count=(16 << 30) // 4 + 1) == ll.LL_ERR_UNSUPPORTED
    assert call(count=0) == ll.LL_OK
    assert ll.LL_STATIC_SCRATCH_BYTES == 64 << 20
