"""Exact rational rounding used to pin the oracle (tests only).

Written from the IEEE 754 definition of round-to-nearest-even for a binary
format with p significant bits and minimum normal exponent emin, so that the
oracle's NumPy casts and divisions can be checked against arithmetic that
involves no floating point at all.
"""
from fractions import Fraction


def floor_log2(a: Fraction) -> int:
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    return e


def round_binary(x: Fraction, p: int, emin: int, emax: int) -> Fraction:
    """Round x to the binary format (p significant bits, normal exponents
    emin..emax, gradual underflow) with ties to even; overflow -> None."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = max(floor_log2(a), emin)
    quantum = Fraction(2) ** (e - (p - 1))
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * quantum
    max_finite = (2 - Fraction(2) ** (1 - p)) * Fraction(2) ** emax
    if r > max_finite:
        return None
    return sign * r


def to_f32(x: Fraction) -> Fraction:
    return round_binary(x, 24, -126, 127)


def to_f16(x: Fraction) -> Fraction:
    return round_binary(x, 11, -14, 15)


def to_bf16(x: Fraction) -> Fraction:
    return round_binary(x, 8, -126, 127)


def rint_even(x: Fraction) -> int:
    fl = x.numerator // x.denominator
    rem = x - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return fl
