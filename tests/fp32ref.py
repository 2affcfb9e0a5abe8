"""Exact binary32 helpers for tests, written from IEEE-754 (not from the oracle).

`rne32(q)` rounds an exact rational to binary32 (round to nearest, ties to
even, gradual underflow, overflow to inf). `fma32(a, b, c)` is the correctly
rounded fused multiply-add of three binary32 values, and `mul32` / `add32`
the correctly rounded product and sum. They let a test evaluate a binary32
expression exactly, independently of any C library.
"""
from __future__ import annotations

import math
import struct
from fractions import Fraction

_MAXF = Fraction((2 ** 24 - 1) * 2 ** 104)


def f32(x: float) -> float:
    return struct.unpack("<f", struct.pack("<f", x))[0]


def bits32(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def from_bits32(u: int) -> float:
    return struct.unpack("<f", struct.pack("<I", u & 0xFFFFFFFF))[0]


def rne32(q: Fraction) -> float:
    if q == 0:
        return 0.0
    sign = -1.0 if q < 0 else 1.0
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 23)
    r = a / quantum
    n = r.numerator // r.denominator
    rem = r - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    v = n * quantum
    if v > _MAXF:
        return sign * math.inf
    return sign * float(v)


def fma32(a: float, b: float, c: float) -> float:
    return rne32(Fraction(a) * Fraction(b) + Fraction(c))


def mul32(a: float, b: float) -> float:
    return rne32(Fraction(a) * Fraction(b))


def add32(a: float, b: float) -> float:
    return rne32(Fraction(a) + Fraction(b))
