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
