"""Exact-arithmetic model of binary32 / bfloat16 rounding, used to pin the oracle.

Nothing here uses the machine's floating point: values are exact rationals
(``fractions.Fraction``), and rounding to a binary format is done by hand,
round to nearest, ties to even, with subnormals and overflow to infinity as
IEEE 754 defines them.  The pins compare the oracle against this model, so an
oracle built with flush-to-zero, x87 double rounding, a wrong summation order
or a wrong final rounding fails them.
"""
from __future__ import annotations

import struct
from dataclasses import dataclass
from fractions import Fraction


@dataclass(frozen=True)
class Fmt:
    prec: int   # significand bits, implicit bit included
    emin: int   # exponent of the smallest normal
    emax: int   # exponent of the largest finite
    ebits: int  # width of the exponent field
    mbits: int  # width of the stored mantissa


BINARY32 = Fmt(prec=24, emin=-126, emax=127, ebits=8, mbits=23)
BFLOAT16 = Fmt(prec=8, emin=-126, emax=127, ebits=8, mbits=7)

INF = "inf"


@dataclass(frozen=True)
class Val:
    """A finite value with the sign of zero kept, or an infinity."""
    mag: Fraction | str  # Fraction >= 0, or INF
    neg: bool


def _floor_log2(a: Fraction) -> int:
    e = a.numerator.bit_length() - a.denominator.bit_length()
    # adjust so that 2**e <= a < 2**(e+1)
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    return e


def round_to(fmt: Fmt, x: Fraction, neg_zero: bool = False) -> Val:
    """Round the exact value x to fmt (nearest, ties to even)."""
    if x == 0:
        return Val(Fraction(0), neg_zero)
    neg = x < 0
    a = -x if neg else x
    e = max(_floor_log2(a), fmt.emin)
    quantum = Fraction(2) ** (e - fmt.prec + 1)
    k = a / quantum
    n = k.numerator // k.denominator
    rem = k - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * quantum
    if r >= Fraction(2) ** (fmt.emax + 1):
        return Val(INF, neg)
    return Val(r, neg)


def add(fmt: Fmt, a: Val, b: Val) -> Val:
    """IEEE addition in fmt, round to nearest even (finite operands or inf)."""
    if a.mag == INF or b.mag == INF:
        if a.mag == INF and b.mag == INF and a.neg != b.neg:
            raise ValueError("inf - inf is NaN; not modelled")
        return a if a.mag == INF else b
    sa = -a.mag if a.neg else a.mag
    sb = -b.mag if b.neg else b.mag
    s = sa + sb
    if s == 0:
        # exact zero sum: -0 only when both operands are -0 (round-to-nearest)
        both_neg_zero = a.mag == 0 and b.mag == 0 and a.neg and b.neg
        return Val(Fraction(0), both_neg_zero)
    return round_to(fmt, s)


def decode(fmt: Fmt, bits: int) -> Val:
    sign = bits >> (fmt.ebits + fmt.mbits) & 1
    exp = (bits >> fmt.mbits) & ((1 << fmt.ebits) - 1)
    man = bits & ((1 << fmt.mbits) - 1)
    if exp == (1 << fmt.ebits) - 1:
        if man:
            raise ValueError("NaN is not a value")
        return Val(INF, bool(sign))
    bias = (1 << (fmt.ebits - 1)) - 1
    if exp == 0:
        mag = Fraction(man) * Fraction(2) ** (1 - bias - fmt.mbits)
    else:
        mag = Fraction((1 << fmt.mbits) | man) * Fraction(2) ** (exp - bias - fmt.mbits)
    return Val(mag, bool(sign))


def encode(fmt: Fmt, v: Val) -> int:
    sign = (1 << (fmt.ebits + fmt.mbits)) if v.neg else 0
    if v.mag == INF:
        return sign | (((1 << fmt.ebits) - 1) << fmt.mbits)
    if v.mag == 0:
        return sign
    bias = (1 << (fmt.ebits - 1)) - 1
    e = _floor_log2(v.mag)
    if e < fmt.emin:
        man = v.mag / Fraction(2) ** (1 - bias - fmt.mbits)
        assert man.denominator == 1
        return sign | int(man)
    man = v.mag / Fraction(2) ** (e - fmt.mbits)
    assert man.denominator == 1
    return sign | ((e + bias) << fmt.mbits) | (int(man) - (1 << fmt.mbits))


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def reduce_sequential(fmt_elem: Fmt, column_bits: list[int]) -> int:
    """Element bits of x_0 + x_1 + ... + x_{P-1}: binary32 adds, left to right,
    starting from x_0, then one rounding to the element format."""
    acc = decode(fmt_elem, column_bits[0])  # widening bfloat16 to binary32 is exact
    for b in column_bits[1:]:
        acc = add(BINARY32, acc, decode(fmt_elem, b))
    if fmt_elem is BINARY32:
        return encode(BINARY32, acc)
    if acc.mag == INF:
        return encode(fmt_elem, acc)
    signed = -acc.mag if acc.neg else acc.mag
    return encode(fmt_elem, round_to(fmt_elem, signed, acc.neg))
