"""The quantizers' code without a division (host check of the arithmetic, no GPU).

The code of Eq. 4 / Eq. 8 is q = clamp(rint(fp32(a / s)), 0, qmax) with a = fp32(delta - z) an fp32 value and
s an fp16 value (the metadata scale, stored in fp16).  The kernels compute it from one reciprocal per group,
rs = rcp(s) (any fp32 value within 1 ulp of 1/s), and Markstein's correction step:
    q1 = fp32(a * rs),  e = fp32(a - q1 * s) (one fma, exact),  q2 = fp32(e * rs + q1) (one fma),
then rint(q2).  The claim: rint(q2) == rint(fp32(a / s)) for every such a, s, because a / s is either exactly
a half-integer or farther than half an ulp from every half-integer (s has at most 11 significant bits), and
q2 is within |a / s| 2^-45 of a / s.  Checked here in exact rational arithmetic, with fp32 rounding written
out (round to nearest, ties to even), over random operands and the fp32 neighbours of every rounding
boundary, for every fp16 binade of s."""
from fractions import Fraction

import numpy as np
import pytest


def f32(fr: Fraction) -> Fraction:
    """fp32 round-to-nearest-even of an exact rational (normal and subnormal range; no overflow here)."""
    if fr == 0:
        return Fraction(0)
    neg = fr < 0
    x = -fr if neg else fr
    e = x.numerator.bit_length() - x.denominator.bit_length()   # 2^e <= x < 2^(e+2)
    if x < Fraction(2) ** e:
        e -= 1
    if x >= Fraction(2) ** (e + 1):
        e += 1
    ulp = Fraction(2) ** (max(e, -126) - 23)
    q = x / ulp
    n = q.numerator // q.denominator
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * ulp
    return -r if neg else r


def next_f32(x: Fraction, up: bool) -> Fraction:
    v = np.float32(float(x))
    assert Fraction(float(v)) == x
    return Fraction(float(np.nextafter(v, np.float32(np.inf if up else -np.inf))))


def rint(x: Fraction) -> int:
    n = x.numerator // x.denominator
    rem = x - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return n


def code_div(a, s, qmax):
    return min(max(rint(f32(a / s)), 0), qmax)


def code_markstein(a, s, rs, qmax):
    q1 = f32(a * rs)
    e = f32(a - q1 * s)
    q2 = f32(e * rs + q1)
    return min(max(rint(q2), 0), qmax)


def fp16_values(rng, n):
    """Positive finite fp16 values: every binade (subnormals included), random mantissas."""
    bits = rng.integers(1, 0x7C00, size=n, dtype=np.int64).astype(np.uint16)
    return [Fraction(float(b)) for b in bits.view(np.float16)]


@pytest.mark.parametrize("qmax", [3, 15, 255])
def test_markstein_code_equals_division_code(qmax):
    rng = np.random.default_rng(qmax)
    cases = 0
    for s in fp16_values(rng, 150 if qmax < 255 else 12):     # (8-bit codes: 257 boundaries per scale)
        r0 = f32(1 / s)
        recips = [r0, next_f32(r0, True), next_f32(r0, False)]
        # a in fp32 near every rounding boundary (m + 1/2) s of the code range: the boundary rounded to fp32,
        # its fp32 neighbours, and a few random values of the range
        pts = []
        for m in range(-1, qmax + 1):
            b = f32((m + Fraction(1, 2)) * s)
            if b < 0:
                continue
            pts += [b, next_f32(b, True), next_f32(b, False)]
            pts.append(next_f32(pts[-2], True))
            pts.append(next_f32(pts[-2], False))
        for x in rng.uniform(0.0, (qmax + 1) * float(s), size=8):
            pts.append(Fraction(float(np.float32(x))))
        for a in pts:
            want = code_div(a, s, qmax)
            for rs in recips:
                assert code_markstein(a, s, rs, qmax) == want, (float(a), float(s), float(rs), qmax)
                cases += 1
    assert cases > 1000


def test_exact_half_integers_tie_to_even():
    # a / s exactly m + 1/2: both forms take the even neighbour
    for s in [Fraction(1, 2), Fraction(3, 1024), Fraction(float(np.float16(0.3)))]:
        for m in range(4):
            a = (m + Fraction(1, 2)) * s
            assert f32(a) == a
            want = m if m % 2 == 0 else m + 1
            assert code_div(a, s, 255) == want
            assert code_markstein(a, s, f32(1 / s), 255) == want
