"""Algorithmic HBM bytes per call of each collective (the roofline numerator).

Counted per call over all P ranks: every byte the method itself must read or
write in HBM -- the inputs read, every packet written into a peer's slot and
read back by its owner, and the outputs written.  Packets carry 4 payload
bytes per 8 (8-byte packets) or 120 per 128 (128-byte lines).  Per rank this
is the paper's per-GPU communication volume of Table I (one-shot LL
2(N-1)M, two-shot LL 4(N-1)M/N) plus the local input reads and output
writes; the 8-byte-packet expansion factor 2 is the "halves the effective
payload bandwidth" of the LL protocol (Sec. IV).
"""
from __future__ import annotations

import math

EXPANSION = {"packet8": 2.0, "line128": 128.0 / 120.0, "sentinel": 1.0}
# bytes moved per payload byte of one packet copy: written by the sender,
# read by the receiver, and (sentinel mode) written back with the sentinel
COPY_FACTOR = {"packet8": 2 * 2.0, "line128": 2 * 128.0 / 120.0, "sentinel": 3.0}


def comm_volume_per_rank(algo: str, p: int, m: float, proto: str) -> float:
    """Bytes one rank sends to its peers (Table I, "Comm. Volume per GPU")."""
    e = EXPANSION[proto]
    if algo == "oneshot":
        return e * (p - 1) * m
    if algo == "twoshot":
        return 2 * e * (p - 1) * m / p
    raise ValueError(algo)


def _proto(algo: str) -> tuple[str, str]:
    base = {"oneshot": "oneshot", "oneshot_line": "oneshot", "oneshot_waves": "oneshot",
            "oneshot_sentinel": "oneshot", "twoshot": "twoshot", "twoshot_line": "twoshot",
            "twoshot_sentinel": "twoshot", "twoshot_waves": "twoshot", "twoshot_sentinel_waves": "twoshot",
            "oneshot_sentinel_waves": "oneshot", "oneshot_line_waves": "oneshot",
            "twoshot_line_waves": "twoshot"}[algo]
    proto = "line128" if "_line" in algo else ("sentinel" if "_sentinel" in algo else "packet8")
    return base, proto


def allreduce_bytes(algo: str, p: int, count: int, esize: int) -> float:
    """HBM bytes moved by one AllReduce call of `count` elements per rank."""
    if algo == "twoshot_atomic":
        return twoshot_atomic_bytes(p, count, esize)
    if algo == "twoshot_sentinel_out":
        return twoshot_sentinel_out_bytes(p, count, esize)
    m = count * esize
    base, proto = _proto(algo)
    f = COPY_FACTOR[proto]
    if base == "oneshot":
        # read input M; (P-1) packet copies written and read back; write output M
        per_rank = m + f * (p - 1) * m + m
    else:
        # RS: read input M, (P-1) chunk packet copies; AG: (P-1) reduced-chunk
        # packet copies; write output M
        c = math.ceil(count / p) * esize
        per_rank = m + 2 * f * (p - 1) * c + m
    return p * per_rank


def twoshot_sentinel_out_bytes(p: int, count: int, esize: int) -> float:
    """Two-shot sentinel with the AllGather stored into the peers' outputs:
    per rank, the input M, the ReduceScatter's (P-1) chunk copies (written,
    read, reset), the output M (own chunk plus the peers' direct stores), the
    poll of the (P-1) peer chunks, and the sentinel fill of the output (M)."""
    m = count * esize
    c = math.ceil(count / p) * esize
    return p * (m + COPY_FACTOR["sentinel"] * (p - 1) * c + m + (p - 1) * c + m)


def twoshot_atomic_bytes(p: int, count: int, esize: int) -> float:
    """Atomic-accumulation two-shot: per rank, read the input M; P chunk
    contributions added into binary32 accumulators (each add reads and writes
    4 bytes per element); the owner reads and zeroes its accumulator; every
    output receives M (own chunk plus the peers' direct stores), is polled
    for the (P-1) peer chunks, and was filled with the sentinel before the
    call (M)."""
    m = count * esize
    c = math.ceil(count / p) * esize
    acc = 4.0 / esize  # accumulator bytes per input byte
    per_rank = m + 2 * acc * m + 2 * acc * c + m + (p - 1) * c + m
    return p * per_rank


def reduce_scatter_bytes(proto: str, p: int, recvcount: int, esize: int) -> float:
    c = recvcount * esize
    return p * (p * c + COPY_FACTOR[proto] * (p - 1) * c + c)


def allgather_bytes(proto: str, p: int, sendcount: int, esize: int) -> float:
    s = sendcount * esize
    return p * (s + COPY_FACTOR[proto] * (p - 1) * s + p * s)


def useful_bytes(p: int, count: int, esize: int) -> float:
    """Read every input once and write every output once."""
    return 2.0 * p * count * esize
