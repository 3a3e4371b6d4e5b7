"""Pins for the CPU oracle (no GPU).

The oracle is checked against things that do not depend on it: closed forms,
special inputs whose ascending-order sum differs from every other order, an
exact rational model of IEEE rounding (``exactfp``), torch's bfloat16
conversion, the paper's forward-error bound (end of Sec. IV) and the
definitions of ReduceScatter / AllGather (Sec. III-A).  Each pin is also shown
to reject a plausible wrong oracle (descending order, pairwise tree, own value
first, per-step bfloat16 rounding, flush-to-zero) planted here on the CPU.
"""
from __future__ import annotations

import math
import os
import random

import numpy as np
import pytest

import exactfp
import oracle
from oracle import npref
from paper_2607_16100_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def f32_bits(vals):
    return np.asarray(vals, dtype=np.float32).view(np.uint32)


def bf16_bits_exact(vals):
    """bfloat16 bits of values that are exactly representable (asserted)."""
    u = np.asarray(vals, dtype=np.float32).view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value is not bfloat16-exact"
    return (u >> 16).astype(np.uint16)


def as_f32(bits_row):
    return npref.widen(np.asarray(bits_row))


def _reduce_on_every_rank(x):
    """The C oracle's Reduce (root = last rank), laid out like an AllReduce
    so that every AllReduce pin below applies to it unchanged."""
    return np.tile(oracle.reduce(x, x.shape[0] - 1), (x.shape[0], 1))


ORACLES = [("c", oracle.allreduce), ("numpy", npref.allreduce), ("c_reduce", _reduce_on_every_rank)]


# ---------------------------------------------------------------- wrong oracles
@np.errstate(over="ignore")  # the overflow pins feed these on purpose
def wrong_descending(x):
    acc = npref.widen(x[-1]).copy()
    for q in range(x.shape[0] - 2, -1, -1):
        acc = (acc + npref.widen(x[q])).astype(np.float32)
    return npref.narrow(acc, x.dtype)


@np.errstate(over="ignore")  # the overflow pins feed these on purpose
def wrong_pairwise(x):
    vals = [npref.widen(x[q]).copy() for q in range(x.shape[0])]
    while len(vals) > 1:
        nxt = [(vals[i] + vals[i + 1]).astype(np.float32) for i in range(0, len(vals) - 1, 2)]
        if len(vals) % 2:
            nxt.append(vals[-1])
        vals = nxt
    return npref.narrow(vals[0], x.dtype)


@np.errstate(over="ignore")  # the overflow pins feed these on purpose
def wrong_own_first(x, r):
    acc = npref.widen(x[r]).copy()
    for q in range(x.shape[0]):
        if q != r:
            acc = (acc + npref.widen(x[q])).astype(np.float32)
    return npref.narrow(acc, x.dtype)


@np.errstate(over="ignore")  # the overflow pins feed these on purpose
def wrong_zero_start(x):
    acc = np.zeros(x.shape[1], np.float32)
    for q in range(x.shape[0]):
        acc = (acc + npref.widen(x[q])).astype(np.float32)
    return npref.narrow(acc, x.dtype)


@np.errstate(over="ignore")  # the overflow pins feed these on purpose
def wrong_bf16_per_step(x):
    acc = npref.widen(x[0]).copy()
    for q in range(1, x.shape[0]):
        acc = npref.widen(npref.narrow((acc + npref.widen(x[q])).astype(np.float32), np.uint16))
    return npref.narrow(acc, np.uint16)


def wrong_truncate_bf16(acc_f32):
    return (np.asarray(acc_f32, np.float32).view(np.uint32) >> 16).astype(np.uint16)


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 3, 4, 5, 6, 7, 8])
def test_all_ones_sum_to_p(name, fn, dtype, p):
    x = wl.ones(p, 37, dtype)
    out = fn(x)
    assert np.all(npref.widen(out) == np.float32(p))


@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 3, 4, 5, 6, 7, 8])
def test_rank_index_fill_sums_to_triangular(name, fn, dtype, p):
    x = wl.rank_index(p, 41, dtype)
    out = fn(x)
    assert np.all(npref.widen(out) == np.float32(p * (p - 1) // 2))


# ---------------------------------------------------------------- order pins
# Vector A (ranks 0..7): ascending sequential gives 0; descending or own-first
# for rank 2 gives 1.  Vector B: ascending sequential gives 1; a pairwise tree
# or descending order gives 0.  All entries are exact in bfloat16 as well.
VEC_A = [2.0 ** 24, 1.0, -(2.0 ** 24), 0.0, 0.0, 0.0, 0.0, 0.0]
VEC_B = [-(2.0 ** 24), 0.0, 2.0 ** 24, 1.0, 0.0, 0.0, 0.0, 0.0]


def column_input(vec, dtype, n=3):
    bits = f32_bits(vec) if dtype == wl.F32 else bf16_bits_exact(vec)
    return np.repeat(bits[:, None], n, axis=1)


@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_order_pin_a(name, fn, dtype):
    x = column_input(VEC_A, dtype)
    assert np.all(npref.widen(fn(x)) == 0.0)
    # the pin separates the plausible wrong orders
    assert np.all(npref.widen(wrong_descending(x)) == 1.0)
    assert np.all(npref.widen(wrong_own_first(x, 2)) == 1.0)


@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_order_pin_b(name, fn, dtype):
    x = column_input(VEC_B, dtype)
    assert np.all(npref.widen(fn(x)) == 1.0)
    assert np.all(npref.widen(wrong_pairwise(x)) == 0.0)
    assert np.all(npref.widen(wrong_descending(x)) == 0.0)


# ---------------------------------------------------------------- rounding pins
@pytest.mark.parametrize("name,fn", ORACLES)
def test_accumulate_in_f32_then_round_once(name, fn):
    x = column_input([256.0, 1.0, 1.0, 0.0, 0.0, 0.0, 0.0, 0.0], wl.BF16)
    assert np.all(npref.widen(fn(x)) == 258.0)
    assert np.all(npref.widen(wrong_bf16_per_step(x)) == 256.0)


@pytest.mark.parametrize("name,fn", ORACLES)
def test_final_rounding_ties_to_even(name, fn):
    # f32 sums 257 and 259 lie exactly halfway between bfloat16 neighbours
    x257 = column_input([256.0, 1.0, 0.0, 0.0], wl.BF16)
    x259 = column_input([256.0, 2.0, 1.0, 0.0], wl.BF16)
    assert np.all(npref.widen(fn(x257)) == 256.0)
    assert np.all(npref.widen(fn(x259)) == 260.0)
    # truncation instead of rounding gives 258 for 259
    assert npref.widen(wrong_truncate_bf16(np.float32(259.0)))[()] == 258.0


@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_signed_zero(name, fn, dtype):
    negz = column_input([-0.0] * 4, dtype)
    out = fn(negz)
    assert np.all(np.signbit(npref.widen(out)))  # -0 + -0 + ... stays -0
    assert np.all(np.signbit(npref.widen(wrong_zero_start(negz))) == False)  # noqa: E712
    mixed = column_input([-0.0, 0.0, -0.0], dtype)
    assert not np.any(np.signbit(npref.widen(fn(mixed))))  # -0 + +0 = +0


@pytest.mark.parametrize("name,fn", ORACLES)
def test_subnormals_are_not_flushed(name, fn):
    tiny = np.float32(2.0 ** -140)  # binary32 subnormal
    x = column_input([tiny, tiny, 0.0, 0.0], wl.F32)
    out = npref.widen(fn(x))
    assert np.all(out == np.float32(2.0 ** -139))
    ftz = np.float32(0.0)  # what a flush-to-zero oracle would give
    assert not np.any(out == ftz)


# ------------------------------------------------ overflow, infinities, NaN
# IEEE 754 binary32 addition with round to nearest even, and one rounding to
# bfloat16: the expected bits below follow from those rules alone.
BF16_MAX, BF16_INF, BF16_NINF = 0x7F7F, 0x7F80, 0xFF80
F32_MAX, F32_INF = 0x7F7FFFFF, 0x7F800000


def _cols(cols, dtype, p=4):
    x = np.zeros((p, len(cols)), dtype=np.uint16 if dtype == wl.BF16 else np.uint32)
    for j, c in enumerate(cols):
        x[:len(c), j] = c
    return x


def _isnan(v):
    v = np.asarray(v)
    if v.dtype == np.uint32:
        return ((v & 0x7F800000) == 0x7F800000) & ((v & 0x007FFFFF) != 0)
    return ((v & 0x7F80) == 0x7F80) & ((v & 0x007F) != 0)


@pytest.mark.parametrize("name,fn", ORACLES)
def test_bf16_overflow_rounds_once_to_inf(name, fn):
    # 0x7B00 = 2^119, half a bfloat16 ulp at bf16 max (2^127 * (2 - 2^-7)).
    x = _cols([[BF16_MAX, 0x7B00],           # binary32 sum 0x7F7F8000: a tie; bf16 max is odd -> Inf
               [BF16_MAX, 0x7A80],           # 0x7F7F4000: under the tie -> bf16 max
               [0xFF7F, 0xFB00],             # the negative tie -> -Inf
               [BF16_MAX, 0x7B00, 0xFB00],   # back to bf16 max before the only rounding
               [0x7F7E, 0x7B00],             # 0x7F7E8000: a tie, 0x7F7E is even -> stays
               [0x7F7E, 0x7B01],             # just over that tie -> 0x7F7F
               [BF16_MAX, BF16_MAX]],        # binary32 overflow -> Inf
              wl.BF16)
    out = fn(x)[0]
    assert list(out) == [BF16_INF, BF16_MAX, BF16_NINF, BF16_MAX, 0x7F7E, 0x7F7F, BF16_INF]
    # rounding at every step instead of once gets the fourth column wrong (Inf - 2^119 = Inf)
    assert wrong_bf16_per_step(x)[3] == BF16_INF


@pytest.mark.parametrize("name,fn", ORACLES)
def test_binary32_overflow_and_infinities(name, fn):
    x = _cols([[F32_MAX, F32_MAX],                # overflow -> +Inf
               [F32_MAX | 0x80000000, F32_MAX | 0x80000000],  # -> -Inf
               [F32_MAX, F32_MAX, F32_MAX | 0x80000000],      # Inf - max stays Inf
               [F32_INF, 0x3F800000],             # Inf + 1
               [0x3F800000, 0, 0, 0xFF800000],    # -Inf at the last rank
               [0x7E967699] * 4],                 # 4 x 1e38 > binary32 max: overflow at the 4th add
              wl.F32)
    out = fn(x)[0]
    assert list(out) == [F32_INF, 0xFF800000, F32_INF, F32_INF, 0xFF800000, F32_INF]
    # the same columns in descending order would give max for the third
    assert wrong_descending(x)[2] == F32_MAX


@pytest.mark.parametrize("name,fn", ORACLES)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_nan_results(name, fn, dtype):
    if dtype == wl.F32:
        cols = [[F32_INF, 0xFF800000], [0x7FC00001, 0x3F800000], [0x3F800000, 0x7F800001],
                [F32_MAX, F32_MAX, 0xFF800000]]
    else:
        cols = [[BF16_INF, BF16_NINF], [0x7FC1, 0x3F80], [0x3F80, 0x7F81], [BF16_MAX, BF16_MAX, BF16_NINF]]
    out = fn(_cols(cols, dtype))
    assert _isnan(out).all()  # Inf - Inf, quiet NaN, signalling NaN, overflow then -Inf


# ---------------------------------------------------------------- exact model
def _random_f32_bits(rng: random.Random):
    kind = rng.random()
    if kind < 0.1:
        return rng.choice([0x00000000, 0x80000000])
    if kind < 0.25:  # subnormal
        return (rng.getrandbits(1) << 31) | rng.randrange(1, 1 << 23)
    if kind < 0.5:   # small normal range, close to each other
        e = rng.randrange(120, 134)
    else:            # wide range (finite, keep clear of overflow)
        e = rng.randrange(1, 200)
    return (rng.getrandbits(1) << 31) | (e << 23) | rng.getrandbits(23)


@pytest.mark.parametrize("p", [2, 3, 4, 8])
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_oracle_matches_exact_rational_model(p, dtype):
    rng = random.Random(1000 + p + (7 if dtype == wl.BF16 else 0))
    n = 160
    cols = []
    for _ in range(n):
        col = [_random_f32_bits(rng) for _ in range(p)]
        if rng.random() < 0.3:  # force heavy cancellation in some columns
            col[-1] = col[0] ^ 0x80000000
        cols.append(col)
    x32 = np.array(cols, dtype=np.uint32).T.copy()
    if dtype == wl.F32:
        x = x32
        fmt = exactfp.BINARY32
    else:
        x = (x32 >> 16).astype(np.uint16)
        fmt = exactfp.BFLOAT16
    out_c = oracle.allreduce(x)
    out_np = npref.allreduce(x)
    for i in range(n):
        want = exactfp.reduce_sequential(fmt, [int(v) for v in x[:, i]])
        assert int(out_c[0, i]) == want, (i, [hex(int(v)) for v in x[:, i]])
        assert int(out_np[0, i]) == want
    assert np.array_equal(out_c, out_np)


def test_bf16_narrowing_matches_exact_model_and_torch():
    torch = pytest.importorskip("torch")
    rng = random.Random(5)
    words = [rng.getrandbits(32) for _ in range(20000)]
    # add halfway cases, carries into the exponent and overflow to inf
    words += [0x43808000, 0x43818000, 0x3F80FFFF, 0x7F7FFFFF, 0x7F7F8000, 0x7F7F7FFF,
              0x00008000, 0x00018000, 0x80008000, 0xFF7F8000, 0x7F800000, 0xFF800000]
    words = [w for w in words if not ((w & 0x7F800000) == 0x7F800000 and (w & 0x7FFFFF))]
    arr = np.array(words, dtype=np.uint32)
    ours_np = npref.narrow(arr.view(np.float32), np.uint16)
    ref_t = torch.from_numpy(arr.view(np.float32).copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours_np, ref_t)
    for w in words[:3000] + words[-12:]:
        h = oracle.bf16_from_f32_bits(w)
        v = exactfp.decode(exactfp.BINARY32, w)
        signed = -v.mag if (v.neg and v.mag != exactfp.INF) else v.mag
        want = exactfp.encode(exactfp.BFLOAT16, v if v.mag == exactfp.INF else exactfp.round_to(exactfp.BFLOAT16, signed, v.neg))
        assert h == want, hex(w)


def test_bf16_nan_stays_nan():
    for w in (0x7FC00000, 0x7F800001, 0xFFC12345, 0x7FFF0000):
        h = oracle.bf16_from_f32_bits(w)
        assert (h & 0x7F80) == 0x7F80 and (h & 0x7F) != 0
    x = np.array([[0x7FC0, 0x3F80], [0x3F80, 0x3F80]], dtype=np.uint16)
    out = npref.widen(oracle.allreduce(x))
    assert np.isnan(out[0, 0]) and out[0, 1] == 2.0


def test_widen_is_exact_shift():
    for h in (0x0000, 0x8000, 0x3F80, 0xC2F7, 0x0001, 0x7F7F):
        assert oracle.f32_bits_from_bf16(h) == h << 16


# ---------------------------------------------------------------- invariants
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 4, 8])
def test_every_rank_gets_the_same_result(dtype, p):
    x = wl.uniform(p, 257, dtype, seed=3)
    out = oracle.allreduce(x)
    assert all(np.array_equal(out[0], out[r]) for r in range(p))


def _gamma(k, u):
    return k * u / (1 - k * u)


def test_gamma_matches_paper_value():
    """The paper prints gamma_63 for binary32 (end of Sec. IV); the golden file
    keeps the printed number."""
    with open(os.path.join(GOLDEN, "gamma_bound.txt")) as f:
        fields = dict(line.split("=", 1) for line in f.read().splitlines() if "=" in line and not line.startswith("#"))
    printed = float(fields["gamma_63_fp32"])
    ours = _gamma(63, 2.0 ** -24)
    assert abs(ours - printed) / printed < 0.02  # the paper rounds to 2 digits


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 3, 8])
def test_within_forward_error_bound(dtype, p):
    x = wl.normal(p, 2000, dtype, sigma=3.0, seed=11) if dtype == wl.BF16 else wl.uniform(p, 2000, dtype, seed=11)
    y = npref.widen(oracle.allreduce(x)[0]).astype(np.float64)
    vals = npref.widen(x).astype(np.float64)
    u32 = 2.0 ** -24
    for i in range(x.shape[1]):
        exact = math.fsum(vals[:, i])
        bound = _gamma(p - 1, u32) * float(np.sum(np.abs(vals[:, i])))
        if dtype == wl.BF16:  # plus the one final rounding to bfloat16
            bound = bound * (1 + 2.0 ** -8) + 2.0 ** -8 * abs(exact)
        assert abs(y[i] - exact) <= bound + 1e-300


def test_bound_pin_rejects_large_errors():
    # a dropped term is far outside the bound
    x = wl.uniform(4, 100, wl.F32, seed=2)
    vals = npref.widen(x).astype(np.float64)
    dropped = vals[0] + vals[1] + vals[2]
    exact = vals.sum(axis=0)
    bound = _gamma(3, 2.0 ** -24) * np.abs(vals).sum(axis=0)
    assert np.any(np.abs(dropped - exact) > bound)


# ---------------------------------------------------------------- the two oracles
@pytest.mark.parametrize("case", [
    ("uniform", 4, 1024, wl.F32, 1.0),       # one-shot, 4 ranks, binary32
    ("normal", 8, 8192, wl.BF16, 1.0),       # 16 KiB decode step, 8 ranks
    ("normal", 8, 65536, wl.BF16, 0.5),      # slice of the 1 MiB case
    ("uniform", 8, 4099, wl.F32, 1.0),
    ("adversarial", 8, 7168, wl.BF16, 1.0),
    ("adversarial", 4, 7168, wl.BF16, 1.0),
])
def test_c_and_numpy_oracles_agree(case):
    kind, p, n, dtype, sigma = case
    x = wl.make(kind, p, n, dtype, seed=0, sigma=sigma)
    assert np.array_equal(oracle.allreduce(x), npref.allreduce(x))


@pytest.mark.parametrize("p", [4, 8])
def test_adversarial_case_is_adversarial(p):
    """Accumulating in bfloat16 would change at least 1 % of the results."""
    x = wl.adversarial(p, 7168 * 16, seed=0)
    good = oracle.allreduce(x)[0]
    bad = wrong_bf16_per_step(x)
    assert np.mean(good != bad) >= 0.01
    # and the magnitudes really are in the +-65504 range
    assert np.max(np.abs(npref.widen(x))) > 60000


# ---------------------------------------------------------------- RS and AG
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p,m", [(2, 1), (3, 5), (4, 896), (8, 896), (8, 13)])
def test_reduce_scatter_is_chunk_of_allreduce(dtype, p, m):
    x = wl.uniform(p, p * m, dtype, seed=4)
    rs = oracle.reduce_scatter(x)
    ar = oracle.allreduce(x)[0]
    for r in range(p):
        assert np.array_equal(rs[r], ar[r * m:(r + 1) * m])
    assert np.array_equal(rs, npref.reduce_scatter(x))


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p,s", [(2, 1), (3, 7), (4, 896), (8, 896)])
def test_allgather_is_concatenation(dtype, p, s):
    x = wl.uniform(p, s, dtype, seed=5)
    ag = oracle.allgather(x)
    cat = np.concatenate(list(x))
    for r in range(p):
        assert ag[r].tobytes() == cat.tobytes()
    assert np.array_equal(ag, npref.allgather(x))


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 4, 8])
def test_allgather_of_reduce_scatter_is_allreduce(dtype, p):
    m = 33
    x = wl.uniform(p, p * m, dtype, seed=6)
    rs = oracle.reduce_scatter(x)
    ag = oracle.allgather(rs)
    assert np.array_equal(ag, oracle.allreduce(x))


# ---------------------------------------------------------------- Broadcast and Reduce
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 3, 8])
def test_broadcast_is_the_roots_block_of_allgather(dtype, p):
    """Every rank's Broadcast result is block `root` of its AllGather result
    (AllGather is pinned above); with rank-index fills it is the root's index."""
    n = 77
    x = wl.uniform(p, n, dtype, seed=12)
    ag = oracle.allgather(x)
    for root in range(p):
        bc = oracle.broadcast(x, root)
        for r in range(p):
            assert bc[r].tobytes() == ag[r, root * n:(root + 1) * n].tobytes()
    idx = wl.rank_index(p, 9, dtype)
    assert np.all(npref.widen(oracle.broadcast(idx, p - 1)) == np.float32(p - 1))
    # a Broadcast that sent rank 0's data whatever the root would fail
    assert not np.array_equal(oracle.broadcast(x, p - 1), np.tile(x[0], (p, 1)))


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("p", [2, 5, 8])
def test_reduce_is_a_row_of_allreduce_for_every_root(dtype, p):
    x = wl.adversarial(p, 999, seed=3) if dtype == wl.BF16 else wl.normal(p, 999, dtype, seed=3)
    ar = oracle.allreduce(x)
    for root in range(p):
        assert np.array_equal(oracle.reduce(x, root), ar[root])


def test_broadcast_and_reduce_reject_bad_roots():
    x = wl.ones(4, 8, wl.F32)
    for fn in (oracle.broadcast, oracle.reduce):
        with pytest.raises(ValueError):
            fn(x, 4)
        with pytest.raises(ValueError):
            fn(x, -1)


def test_empty_inputs():
    for dtype in (wl.F32, wl.BF16):
        x = wl.uniform(4, 0, dtype)
        assert oracle.allreduce(x).shape == (4, 0)
        assert oracle.allgather(x).shape == (4, 0)
