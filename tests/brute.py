"""Brute-force references for tiny inputs, in exact rational arithmetic.

These helpers are independent of the oracle: they enumerate subsets and
evaluate the App. B objectives with ``fractions.Fraction`` of the binary32 /
BF16 values, so no rounding enters the comparison.
"""
from __future__ import annotations

import itertools
import struct
from fractions import Fraction


def f32(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", bits & 0xFFFFFFFF))[0]


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def bf16_value(bits: int) -> float:
    return f32((bits & 0xFFFF) << 16)


def f32_fraction(bits: int) -> Fraction:
    """Exact value of a finite binary32 pattern, decoded from its fields."""
    bits &= 0xFFFFFFFF
    sign = -1 if bits >> 31 else 1
    ex = (bits >> 23) & 0xFF
    man = bits & 0x7FFFFF
    assert ex != 0xFF, "finite values only"
    if ex == 0:                                   # subnormal: man * 2^-149
        return sign * Fraction(man, 1 << 149)
    val = Fraction((1 << 23) | man) * (Fraction(2) ** (ex - 150))
    return sign * val


def f32_rne_bits(q: Fraction, zero_sign: int = 0) -> int:
    """binary32 pattern of the exact rational q rounded to nearest, ties to
    even (IEEE 754 roundTiesToEven), with subnormals kept.  A zero result
    takes the sign bit zero_sign (an exact zero sum is +0 unless both addends
    are -0).  Written from the format's definition; no float conversion."""
    if q == 0:
        return (zero_sign & 1) << 31
    sign = 1 if q < 0 else 0
    a = -q if sign else q
    # binade: 2^e <= a < 2^(e+1)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    assert Fraction(2) ** e <= a < Fraction(2) ** (e + 1)
    ulp_exp = max(e, -126) - 23                  # spacing of binary32 values near a
    m = a / (Fraction(2) ** ulp_exp)              # a in units of that spacing
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    # n * 2^ulp_exp is the rounded magnitude; re-normalise a carry to 2^24
    if n == 1 << 24:
        n >>= 1
        ulp_exp += 1
    if n >= 1 << 23:                              # normal
        biased = ulp_exp + 23 + 127
        assert 1 <= biased <= 254, "overflow is outside the inputs' domain"
        return (sign << 31) | (biased << 23) | (n - (1 << 23))
    return (sign << 31) | n                       # subnormal (ulp_exp = -149)


def f32_add_rne_bits(x_bits: int, y_bits: int) -> int:
    """binary32 sum x + y (round to nearest even) from the exact rational sum."""
    both_neg_zero = (x_bits & 0xFFFFFFFF) == 0x80000000 and (y_bits & 0xFFFFFFFF) == 0x80000000
    return f32_rne_bits(f32_fraction(x_bits) + f32_fraction(y_bits), 1 if both_neg_zero else 0)


def biased_scores_exact(z_bits, b) -> list:
    """s_{t,e} = z_{t,e} + b_e (Sec. 2, I_t = TopK(z_t + b)) as binary32 patterns,
    each rounded once from the exact rational sum.  z_bits: BF16 patterns
    [T][E], b: binary32 values [E].  Returns a list of rows of uint32 patterns."""
    b_bits = [f32_bits(float(v)) for v in b]
    out = []
    for row in z_bits:
        out.append([f32_add_rne_bits((int(zb) & 0xFFFF) << 16, b_bits[e]) for e, zb in enumerate(row)])
    return out


def topk_subset(s, K):
    """The valid Top-K subset preferred by the lower-index rule.

    A K-subset S is valid when every chosen score is >= every unchosen one.
    Among valid subsets the lexicographically smallest sorted index tuple is
    the one that keeps the lower indices on a boundary tie.
    """
    E = len(s)
    for S in itertools.combinations(range(E), K):       # lexicographic order
        rest = [e for e in range(E) if e not in S]
        if min(s[e] for e in S) >= max(s[e] for e in rest):
            return sorted(S, key=lambda e: (-s[e], e))     # rank order
    raise AssertionError("no valid subset")


def tau_by_threshold_identity(s, K):
    """Smallest minimiser of K*a + sum_e [s_e - a]_+ over a in {s_e} (App. B).

    The objective is convex and piecewise linear with kinks at the s_e, so its
    minimum is attained at a kink; the smallest minimiser is the (K+1)st
    largest entry.
    """
    vals = [Fraction(v) for v in s]

    def obj(a):
        return K * a + sum(max(v - a, Fraction(0)) for v in vals)

    best = min(obj(a) for a in vals)
    return min(a for a in vals if obj(a) == best)


def quantile_by_counts(keys, r):
    """The unique key v with #{k < v} < r <= #{k <= v}."""
    found = [v for v in set(keys)
             if sum(k < v for k in keys) < r <= sum(k <= v for k in keys)]
    assert len(found) == 1
    return found[0]


def quantile_by_dual(margins, r):
    """Lower endpoint of argmin_b sum_t [b - m_t]_+ - r*b over b in {m_t} (App. B)."""
    vals = [Fraction(v) for v in margins]

    def g(bb):
        return sum(max(bb - m, Fraction(0)) for m in vals) - r * bb

    best = min(g(bb) for bb in vals)
    return min(bb for bb in vals if g(bb) == best)
