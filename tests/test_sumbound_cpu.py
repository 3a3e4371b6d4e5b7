"""The bound check used for the non-deterministic atomic two-shot, pinned on
the CPU: it accepts every summation order and rejects plausible mistakes."""
from __future__ import annotations

import itertools

import numpy as np
import pytest

import oracle
from paper_2607_16100_amd import workloads as wl
from sumbound import assert_within_summation_bound, gamma


def f32_sum_in_order(x_f32: np.ndarray, order) -> np.ndarray:
    acc = x_f32[order[0]].copy()
    for q in order[1:]:
        acc = (acc + x_f32[q]).astype(np.float32)
    return acc


def test_gamma_matches_the_printed_value():
    # the paper prints gamma_63 ~ 3.8e-6 for binary32
    assert abs(gamma(63) - 3.8e-6) < 0.05e-6


@pytest.mark.parametrize("p", [3, 4])
def test_every_summation_order_is_accepted(p):
    x = wl.normal(p, 2000, "f32", seed=5)
    xf = x.view(np.float32)
    for order in itertools.permutations(range(p)):
        y = f32_sum_in_order(xf, order).view(np.uint32)
        assert_within_summation_bound(np.tile(y, (p, 1)), x, "f32", f"order {order}")


def test_ordered_oracle_is_accepted_for_both_types():
    for dtype in ("f32", "bf16"):
        x = wl.adversarial(8, 4096, seed=2) if dtype == "bf16" else wl.normal(8, 4096, "f32", seed=2)
        assert_within_summation_bound(oracle.allreduce(x), x, dtype, dtype)


def test_rejects_a_missing_contribution_disagreeing_ranks_and_a_lost_rounding():
    p, n = 8, 4096
    x = wl.normal(p, n, "f32", seed=9)
    good = oracle.allreduce(x)
    # one rank's contribution dropped
    drop = f32_sum_in_order(x.view(np.float32), list(range(p - 1))).view(np.uint32)
    with pytest.raises(AssertionError):
        assert_within_summation_bound(np.tile(drop, (p, 1)), x, "f32", "dropped")
    # ranks that do not agree
    bad = good.copy()
    bad[3, 10] ^= 1
    with pytest.raises(AssertionError):
        assert_within_summation_bound(bad, x, "f32", "disagree")
    # a result off by far more than the bound allows (a double-counted rank)
    twice = (drop.view(np.float32) + 2 * x.view(np.float32)[p - 1]).astype(np.float32).view(np.uint32)
    with pytest.raises(AssertionError):
        assert_within_summation_bound(np.tile(twice, (p, 1)), x, "f32", "double")
    # bfloat16: truncating instead of rounding stays within the bound for
    # most elements, but a result one bfloat16 ulp too far on purpose fails
    xb = wl.normal(p, n, "bf16", seed=3)
    yb = oracle.allreduce(xb)
    off = yb.copy()
    off[:, :] = (off.astype(np.uint32) + 2).astype(np.uint16)  # two ulps
    with pytest.raises(AssertionError):
        assert_within_summation_bound(off, xb, "bf16", "two ulps")
