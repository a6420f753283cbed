"""Exact rational arithmetic helpers for the pin tests."""
import math
from fractions import Fraction


def round_to_f32(x: Fraction) -> float:
    """Exact rational -> nearest binary32 (ties to even), by definition."""
    if x == 0:
        return 0.0
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    # choose e so that 2^23 <= a / 2^(e-23) < 2^24, clamped to the subnormal ulp
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp_exp = max(e - 23, -149)
    m = a / (Fraction(2) ** ulp_exp)
    q, rem = divmod(m.numerator, m.denominator)
    twice = 2 * rem
    if twice > m.denominator or (twice == m.denominator and q % 2 == 1):
        q += 1
    val = math.ldexp(q, ulp_exp)
    return sign * val if val < 2.0**128 else sign * math.inf
