"""The byte model behind every roofline figure, against Table I.

Table I gives the per-GPU communication volume of each low-latency AllReduce
(N ranks, message M): one-shot LL 2(N-1)M, one-shot sentinel (N-1)M, two-shot
LL 4(N-1)M/N, two-shot sentinel 2(N-1)M/N.  The HBM model counts each
transmitted byte twice (written by the sender, read by the receiver), a third
time in sentinel mode (the reset), and adds the input read and output write.
"""
from __future__ import annotations

import pytest

from paper_2607_16100_amd import bytemodel as bm


@pytest.mark.parametrize("n", [2, 4, 8])
def test_comm_volume_matches_table_one(n):
    m = 1 << 20
    assert bm.comm_volume_per_rank("oneshot", n, m, "packet8") == 2 * (n - 1) * m
    assert bm.comm_volume_per_rank("oneshot", n, m, "sentinel") == (n - 1) * m
    assert bm.comm_volume_per_rank("twoshot", n, m, "packet8") == 4 * (n - 1) * m / n
    assert bm.comm_volume_per_rank("twoshot", n, m, "sentinel") == 2 * (n - 1) * m / n


@pytest.mark.parametrize("n", [2, 4, 8])
def test_hbm_bytes_are_comm_volume_plus_local_traffic(n):
    count, es = 1 << 18, 4
    m = count * es
    for algo, base, proto, touches in [("oneshot", "oneshot", "packet8", 2), ("oneshot_line", "oneshot", "line128", 2),
                                       ("oneshot_sentinel", "oneshot", "sentinel", 3),
                                       ("twoshot", "twoshot", "packet8", 2),
                                       ("twoshot_line", "twoshot", "line128", 2),
                                       ("twoshot_sentinel", "twoshot", "sentinel", 3)]:
        want = n * (2 * m + touches * bm.comm_volume_per_rank(base, n, m, proto))
        assert bm.allreduce_bytes(algo, n, count, es) == pytest.approx(want, rel=1e-12), algo


def test_rs_ag_bytes():
    # ReduceScatter of P*c in, c out; AllGather of s in, P*s out
    p, c, es = 8, 896, 2
    b = c * es
    assert bm.reduce_scatter_bytes("sentinel", p, c, es) == p * (p * b + 3 * (p - 1) * b + b)
    assert bm.allgather_bytes("packet8", p, c, es) == p * (b + 4 * (p - 1) * b + p * b)
    assert bm.useful_bytes(p, c, es) == 2 * p * b


def test_direct_output_variants():
    p, count, es = 8, 1 << 20, 4
    m, c = count * es, count * es // p
    assert bm.allreduce_bytes("twoshot_sentinel_out", p, count, es) == p * (3 * m + 4 * (p - 1) * c)
    # atomic: input, adds (read + write of a binary32 accumulator), accumulator
    # read and reset, output, poll, fill
    assert bm.allreduce_bytes("twoshot_atomic", p, count, es) == p * (m + 2 * m + 2 * c + m + (p - 1) * c + m)
    assert bm.allreduce_bytes("twoshot_atomic", p, count, 2) == p * (count * 2 * 3 + 4 * count * 2 + 4 * c // 2
                                                                     + (p - 1) * c // 2)
