"""Exact rational rounding for pins: values are Fractions, results the IEEE
round-to-nearest-even binary32 value as a Python float (exact in binary64)."""
from fractions import Fraction


def round_half_even(fr: Fraction) -> int:
    fl = fr.numerator // fr.denominator
    rem = fr - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        return fl + 1
    return fl


def round_to_f32(fr: Fraction) -> float:
    """binary32 nearest to fr (ties to even), subnormals included; fr must lie
    below the binary32 overflow threshold."""
    if fr == 0:
        return 0.0
    sign = -1 if fr < 0 else 1
    fr = abs(fr)
    e = fr.numerator.bit_length() - fr.denominator.bit_length()  # 2^e <= fr < 2^(e+2)
    while Fraction(2) ** (e + 1) <= fr:
        e += 1
    while Fraction(2) ** e > fr:
        e -= 1
    quantum = Fraction(2) ** (max(e, -126) - 23)  # 24 significant bits; fixed below 2^-126
    m = round_half_even(fr / quantum)
    return sign * float(m * quantum)
