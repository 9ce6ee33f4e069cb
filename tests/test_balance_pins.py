"""Pins of the balance oracle (MaxVio, the closed QB loop) on the CPU.

MaxVio is pinned by closed forms, by the paper's own reading of a value
(Appendix E: a Local MaxVio of 5.96 means the most-loaded expert receives
about 6.96 times its uniform load), by exact rational arithmetic, and by
planted mistakes.  The closed loop is checked for the property Eq. 2 is
built for: after one update, fresh batches from the same skewed distribution
are routed far more evenly.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import balance_oracle as B
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "maxvio.json")


def test_maxvio_closed_forms():
    E, K, T = 64, 6, 6400
    even = np.full(E, K * T // E)
    assert B.max_violation_of(even, T, K) == 0.0
    # every token picks the same K experts: the most-loaded one holds T picks
    top = np.zeros(E, np.int64)
    top[:K] = T
    assert B.max_violation_of(top, T, K) == E / K - 1
    assert math.isnan(B.max_violation_of(np.zeros(E), 0, K))


def test_maxvio_matches_the_papers_reading():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        got = B.max_violation_of(np.asarray(c["load"]), c["tokens"], c["K"])
        assert got == pytest.approx(c["maxvio"], abs=1e-12), c["source"]


def test_maxvio_against_exact_rationals():
    rng = np.random.default_rng(5)
    for _ in range(200):
        E = int(rng.choice([8, 64, 256]))
        K = int(rng.integers(1, E))
        P = int(rng.integers(1, 6))
        sizes = rng.integers(0, 3000, size=P)
        off = np.concatenate([[0], np.cumsum(sizes)])
        load = np.stack([rng.multinomial(int(K * n), np.ones(E) / E) if n else np.zeros(E, np.int64)
                         for n in sizes])
        glob, local = B.max_violation(load, off, K)
        T = int(off[-1])
        if T:
            exact = max(Fraction(int(f), 1) / Fraction(K * T, E) - 1 for f in load.sum(0))
            assert glob == pytest.approx(float(exact), rel=1e-15, abs=1e-15)
        for p in range(P):
            n = int(sizes[p])
            if n == 0:
                assert math.isnan(local[p])
                continue
            exact = max(Fraction(int(f), 1) / Fraction(K * n, E) - 1 for f in load[p])
            assert local[p] == pytest.approx(float(exact), rel=1e-15, abs=1e-15)


def test_local_maxvio_uses_the_partition_size():
    # two partitions of different sizes with the same per-expert spread
    E, K = 8, 2
    load = np.array([[10, 10, 0, 0, 0, 0, 0, 0], [100, 100, 0, 0, 0, 0, 0, 0]])
    glob, local = B.max_violation(load, [0, 10, 110], K)
    assert local[0] == pytest.approx(10 / (2 * 10 / 8) - 1)
    assert local[1] == pytest.approx(100 / (2 * 100 / 8) - 1)
    assert glob == pytest.approx(110 / (2 * 110 / 8) - 1)


def test_qb_loop_balances_fresh_batches():
    """Eq. 2's purpose: the bias from step q balances step q+1's batch."""
    w = W.CONFIGS["skew64"].with_T(32768, 4)
    batches = [W.generate(w, batch=q)[0] for q in range(4)]
    _, _, off = W.generate(w)
    steps = B.qb_loop(batches, np.zeros(w.E, np.float32), w.K, off)
    assert steps[0]["maxvio_global"] > 1.0          # per-expert offsets N(0, 1): strongly skewed
    for s in steps[1:]:
        assert s["maxvio_global"] < 0.3, s["maxvio_global"]
        assert np.all(s["maxvio_local"] < 0.5)
    for s in steps:
        assert abs(float(np.sum(s["b_next"].astype(np.float64)))) < 1e-3   # centred
        np.testing.assert_array_equal(s["load"].sum(), w.K * w.T)


@pytest.mark.parametrize("mutant", ["global_T_for_local", "inverted_target"])
def test_maxvio_pins_catch_planted_mistakes(monkeypatch, mutant):
    orig = B.max_violation_of
    if mutant == "global_T_for_local":
        def bad(load_pe, part_off, K):
            load_pe = np.asarray(load_pe, np.int64)
            T = int(np.asarray(part_off)[-1])
            return orig(load_pe.sum(0), T, K), np.array([orig(l, T, K) for l in load_pe])
        monkeypatch.setattr(B, "max_violation", bad)
    else:
        def bad_of(load_e, n, K):
            load_e = np.asarray(load_e, np.int64)
            return float(np.float64(load_e.max() * K) / np.float64(load_e.size * n) - 1) if n else float("nan")
        monkeypatch.setattr(B, "max_violation_of", bad_of)
    failed = False
    for fn in (test_maxvio_closed_forms, test_local_maxvio_uses_the_partition_size,
               test_maxvio_matches_the_papers_reading):
        try:
            fn()
        except AssertionError:
            failed = True
    assert failed, mutant
