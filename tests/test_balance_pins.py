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


# ------------------------------------------------------ Load-Error Injection --
def _loads(rng, E, K, sizes, skew=1.0):
    w = rng.dirichlet(np.ones(E) * skew)
    return np.stack([rng.multinomial(int(K * n), w) if n else np.zeros(E, np.int64) for n in sizes])


def test_lei_residual_is_zero_centred_and_bounded():
    """The normalisation keeps rho's direction and zero mean and bounds the
    injected value by eta * c (Sec. 4, 'Stabilizing the correction')."""
    rng = np.random.default_rng(21)
    E, K, eta, c = 64, 6, 1e-4, 2.0
    sizes = [3000, 500, 0, 8000]
    off = np.concatenate([[0], np.cumsum(sizes)])
    load = _loads(rng, E, K, sizes, skew=0.3)
    raw = B.lei_residual(load, off, K, 1.0, 0.0).astype(np.float64)
    inj = B.lei_residual(load, off, K, eta, c).astype(np.float64)
    for p, n in enumerate(sizes):
        if n == 0:
            assert np.all(inj[p] == 0)
            continue
        assert abs(raw[p].sum()) < 1e-5 * E                     # sum_e rho_e = 0
        assert np.max(np.abs(inj[p])) <= eta * c * (1 + 1e-6)    # ||eta rho~||_inf = eta c tanh(xi) < eta c
        xi = np.max(np.abs(raw[p])) / c
        np.testing.assert_allclose(inj[p], eta * raw[p] * np.tanh(xi) / xi, rtol=1e-6, atol=1e-12)
        assert np.all(np.sign(inj[p]) == np.sign(raw[p]))        # direction kept


def test_lei_balanced_batch_injects_nothing_and_small_errors_pass_unscaled():
    E, K, n = 8, 2, 4000
    even = np.full((1, E), K * n // E)
    assert np.all(B.lei_residual(even, [0, n], K, 1e-3, 1.0) == 0)     # xi = 0: tanh(xi)/xi := 1
    near = even.copy()
    near[0, 0] += 1
    near[0, 1] -= 1
    raw = B.lei_residual(near, [0, n], K, 1.0, 0.0)[0].astype(np.float64)
    nrm = B.lei_residual(near, [0, n], K, 1.0, 100.0)[0].astype(np.float64)
    xi = np.max(np.abs(raw)) / 100.0
    np.testing.assert_allclose(nrm, raw, rtol=xi * xi)                 # tanh(xi)/xi = 1 - xi^2/3 + ...


def test_lei_residual_is_the_ste_gradient():
    """App. D: with the surrogate P^L_e = mean_t s_{t,e}, the straight-through
    gradient of 1/2 ||F~ - Q||^2 is (F_e - Q_e)/T for every token; LEI's
    rho_e = E (F_e - Q_e) is that gradient times E*T (autograd check)."""
    import torch
    rng = np.random.default_rng(3)
    T, E, K = 500, 16, 4
    idx = np.stack([rng.choice(E, K, replace=False, p=rng.dirichlet(np.ones(E))) for _ in range(T)])
    load = np.bincount(idx.ravel(), minlength=E)[None, :]
    s = torch.tensor(rng.random((T, E)), dtype=torch.float64, requires_grad=True)
    F = torch.tensor(load[0] / (K * T), dtype=torch.float64)
    Q = torch.full((E,), 1.0 / E, dtype=torch.float64)
    PL = s.mean(dim=0)
    Ft = PL + (F - PL).detach()
    (0.5 * ((Ft - Q) ** 2).sum()).backward()
    rho = B.lei_residual(load, [0, T], K, 1.0, 0.0)[0].astype(np.float64)
    np.testing.assert_allclose(rho, s.grad.numpy()[0] * E * T, rtol=1e-6, atol=1e-6)
    assert np.allclose(s.grad.numpy(), s.grad.numpy()[0][None, :])     # the same for every token


def test_lei_inject_adds_each_partitions_value_to_its_tokens_only():
    rng = np.random.default_rng(8)
    T, E = 37, 8
    off = np.array([0, 10, 10, 30, 37])
    g = rng.standard_normal((T, E)).astype(np.float32)
    inj = rng.standard_normal((4, E)).astype(np.float32) * 1e-3
    out = B.lei_inject(g, inj, off)
    for t in range(T):
        p = int(np.searchsorted(off, t, side="right") - 1)
        for e in range(E):
            assert out[t, e] == np.float32(g[t, e]) + np.float32(inj[p, e])


@pytest.mark.parametrize("mutant", ["l2_norm", "global_T", "sign", "no_tanh"])
def test_lei_pins_catch_planted_mistakes(monkeypatch, mutant):
    orig = B.lei_residual

    def bad(load_pe, part_off, K, eta, c):
        load_pe = np.asarray(load_pe, np.int64)
        part_off = np.asarray(part_off, np.int64)
        P, E = load_pe.shape
        out = np.zeros((P, E), np.float32)
        for p in range(P):
            n = int(part_off[p + 1] - part_off[p])
            if mutant == "global_T":
                n = int(part_off[-1])
            if n == 0:
                continue
            rho = np.array([float(f * E) / float(K * n) - 1.0 for f in load_pe[p]])
            if mutant == "sign":
                rho = -rho
            scale = 1.0
            if c > 0:
                nrm = np.sqrt((rho ** 2).sum()) if mutant == "l2_norm" else np.abs(rho).max()
                xi = nrm / c
                scale = (1.0 / xi if mutant == "no_tanh" else math.tanh(xi) / xi) if xi > 0 else 1.0
            out[p] = (eta * rho * scale).astype(np.float32)
        return out

    monkeypatch.setattr(B, "lei_residual", bad)
    failed = False
    for fn in (test_lei_residual_is_zero_centred_and_bounded,
               test_lei_balanced_batch_injects_nothing_and_small_errors_pass_unscaled,
               test_lei_residual_is_the_ste_gradient):
        try:
            fn()
        except AssertionError:
            failed = True
    assert failed, mutant
    del orig
