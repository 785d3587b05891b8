"""Exact rational arithmetic with IEEE-754 binary32 round-to-nearest-even.

An independent model of binary32 operations for brute-force checks on tiny
inputs: every operation is carried out exactly in rationals and then rounded
once to the nearest binary32 value (ties to even), with gradual underflow and
overflow to infinity.  It shares nothing with the C oracle.  Zero results take
IEEE-754's signs: a nonzero exact result that rounds to zero keeps its sign; an
exact zero sum is +0 under round-to-nearest unless both addends are -0; a
zero product's sign is the exclusive-or of the factors' signs.
"""
import math
from fractions import Fraction

_EMIN = -126          # smallest normal exponent
_P = 24               # significand bits
_MAX = (2 - Fraction(1, 2 ** 23)) * Fraction(2) ** 127


def rn32(q: Fraction) -> float:
    q = Fraction(q)
    if q == 0:
        return 0.0
    sign = -1 if q < 0 else 1
    a = abs(q)
    # exponent e with 2^e <= a < 2^(e+1)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    elif Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** (max(e, _EMIN) - (_P - 1))
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = fl * quantum
    if r > _MAX:
        return sign * float("inf")
    return sign * float(r)


def _neg(x) -> bool:
    return math.copysign(1.0, x) < 0


def _zero_sum(x_neg: bool, y_neg: bool) -> float:
    """Sign of an exact zero sum of two signed zeros (round to nearest)."""
    return -0.0 if (x_neg and y_neg) else 0.0


def fma(a, b, c) -> float:
    exact = Fraction(a) * Fraction(b) + Fraction(c)
    if exact != 0:
        return rn32(exact)
    if a == 0 or b == 0:  # a zero product plus c (= +-0 here)
        return _zero_sum(_neg(a) != _neg(b), _neg(c))
    return 0.0            # a nonzero product cancelled exactly by c


def add(a, b) -> float:
    exact = Fraction(a) + Fraction(b)
    if exact != 0:
        return rn32(exact)
    if a == 0 and b == 0:
        return _zero_sum(_neg(a), _neg(b))
    return 0.0


def mul(a, b) -> float:
    exact = Fraction(a) * Fraction(b)
    if exact != 0:
        return rn32(exact)
    return -0.0 if _neg(a) != _neg(b) else 0.0


def canonical_dot(a, b, k_block, fused=True) -> float:
    """The blocked left-to-right contraction, each step rounded exactly once."""
    K = len(a)
    blk = k_block if k_block > 0 else K
    acc = 0.0
    for k0 in range(0, K, blk):
        p = 0.0
        for k in range(k0, min(k0 + blk, K)):
            p = fma(a[k], b[k], p) if fused else add(p, mul(a[k], b[k]))
        acc = add(acc, p)
    return acc
