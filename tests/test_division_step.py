"""The division step the proxy kernel uses in place of fp32 divides (its
E4M3 encodes of the proxy and of the linear-term levels): with y = RN(1/b),
q0 = RN(a y), t = RN(q0 b - a), the result RN(q0 - t y) equals RN(a / b)
(Markstein's theorem: q0 is within an ulp of a / b, so t is exact and one
correction rounds correctly).  The kernel takes this path for b in
[2^-80, 2^100]; there every quotient of magnitude >= 2^-11 must match, and
smaller ones may differ by at most an ulp (both encode to a signed zero in
E4M3).  Checked here with exact rational arithmetic."""
from fractions import Fraction

import numpy as np


def rn32(x: Fraction) -> Fraction:
    """x rounded to the nearest fp32 value, ties to even (subnormals kept)."""
    if x == 0:
        return Fraction(0)
    s = -1 if x < 0 else 1
    ax = abs(x)
    e = ax.numerator.bit_length() - ax.denominator.bit_length()
    if Fraction(2) ** e > ax:
        e -= 1
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 23)
    m = ax / quantum
    f = m.numerator // m.denominator
    r = m - f
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2 == 1):
        f += 1
    return s * f * quantum


def div_step(a: Fraction, b: Fraction) -> Fraction:
    y = rn32(1 / b)
    q0 = rn32(a * y)
    t = rn32(q0 * b - a)
    return rn32(q0 - t * y)


def f32(bits: int) -> Fraction:
    return Fraction(float(np.array([bits], dtype=np.uint32).view(np.float32)[0]))


def test_division_step_matches_rounded_quotient():
    rng = np.random.default_rng(3)
    n_checked = 0
    for i in range(3000):
        eb = int(rng.integers(127 - 80, 127 + 100))
        b = f32((eb << 23) | int(rng.integers(0, 1 << 23)))
        if i % 3 == 0:  # the encode's divisor: amax / 448, numerators up to amax
            amax = rn32(b * 448)
            a = rn32(amax * Fraction(int(rng.integers(0, 1 << 24)), 1 << 24))
        else:  # any numerator with |a / b| < 2^10, subnormals included
            ea = eb - 45 + int(rng.integers(0, 55))
            mant = int(rng.integers(0, 1 << 23))
            a = f32((max(ea, 0) << 23) | (mant >> (0 if ea > 0 else int(rng.integers(0, 23)))))
        if rng.integers(0, 2):
            a = -a
        q, ref = div_step(a, b), rn32(a / b)
        if abs(ref) >= Fraction(1, 2048):
            assert q == ref, (float(a), float(b), float(q), float(ref))
            n_checked += 1
        else:
            ulp = Fraction(2) ** -149 if ref == 0 else abs(rn32(ref * (1 + Fraction(1, 1 << 23))) - ref)
            assert abs(q - ref) <= ulp and abs(q) < Fraction(1, 1024), (float(a), float(b))
    assert n_checked > 1500
