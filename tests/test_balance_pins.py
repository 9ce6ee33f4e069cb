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


def test_local_maxvio_is_the_mean_over_local_batches():
    """Appendix E: Local MaxVio is computed per local batch and then averaged.
    Hand case (E = 8, K = 2): partition 0 has 10 tokens (uniform load 2.5)
    and a largest load of 10, MaxVio 3; partition 1 is empty (no value);
    partition 2 has 100 tokens (uniform 25) and a largest load of 50,
    MaxVio 1.  Local MaxVio = (3 + 1) / 2 = 2, while the largest local value
    is 3 and Global MaxVio (110 tokens, largest load 60) is 60/27.5 - 1."""
    load = np.array([[10, 6, 4, 0, 0, 0, 0, 0],
                     [0, 0, 0, 0, 0, 0, 0, 0],
                     [50, 40, 30, 30, 20, 10, 10, 10]])
    off = [0, 10, 10, 110]
    glob, local = B.max_violation(load, off, 2)
    assert local[0] == 3.0 and math.isnan(local[1]) and local[2] == 1.0
    assert B.local_maxvio_mean(local) == 2.0
    assert float(Fraction(60) / Fraction(2 * 110, 8) - 1) == pytest.approx(glob, rel=1e-15)
    assert math.isnan(B.local_maxvio_mean([float("nan")]))
    # mean over many partitions against exact rationals
    rng = np.random.default_rng(12)
    vals = rng.standard_normal(37)
    want = sum(Fraction(float(v)) for v in vals) / 37
    assert B.local_maxvio_mean(vals) == pytest.approx(float(want), rel=1e-14)


@pytest.mark.parametrize("mutant", ["max", "empty_as_zero"])
def test_local_mean_pins_catch_planted_mistakes(monkeypatch, mutant):
    orig = B.local_maxvio_mean
    if mutant == "max":
        bad = lambda local: float(np.nanmax(np.asarray(local, np.float64)))
    else:
        bad = lambda local: float(np.mean(np.nan_to_num(np.asarray(local, np.float64), nan=0.0)))
    monkeypatch.setattr(B, "local_maxvio_mean", bad)
    with pytest.raises(AssertionError):
        test_local_maxvio_is_the_mean_over_local_batches()
    monkeypatch.setattr(B, "local_maxvio_mean", orig)


def test_qb_loop_balances_fresh_batches():
    """Eq. 2's purpose: the bias from step q balances step q+1's batch."""
    w = W.WORKLOADS["skew64"].with_T(32768, 4)
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


# ------------------------------------- statistics EQB is compared with --------
from oracle import eqb_oracle as O


def test_rank_average_of_one_shard_is_eqb():
    w = W.WORKLOADS["skew64"].with_T(6000, 1)
    z, b, off = W.generate(w)
    bp, avg, bn = B.rank_averaged_qb(z, b, w.K, off)
    ex = O.run_layer(z, b, w.K, off)
    np.testing.assert_array_equal(bp[0], ex["bhat"])
    np.testing.assert_array_equal(bn.view(np.uint32), ex["b_next"].view(np.uint32))


def test_rank_average_of_identical_shards_is_eqb():
    """P copies of one batch: every shard's quantile is the global one."""
    w = W.WORKLOADS["skew64"].with_T(2048, 1)        # 2048 * 6 / 64 is an integer
    z, b, _ = W.generate(w)
    zz = np.concatenate([z] * 3)
    off = np.array([0, 2048, 4096, 6144])
    bp, avg, bn = B.rank_averaged_qb(zz, b, w.K, off)
    ex = O.run_layer(zz, b, w.K, off)
    for p in range(3):
        np.testing.assert_array_equal(bp[p], ex["bhat"])
    np.testing.assert_array_equal(bn.view(np.uint32), ex["b_next"].view(np.uint32))


def test_shard_quantile_is_numpys_inverted_cdf_and_average_depends_on_the_split():
    w = W.WORKLOADS["skew64"].with_T(9000, 3)
    z, b, off = W.generate(w)
    bp, avg, _ = B.rank_averaged_qb(z, b, w.K, off)
    _, _, tau = O.route_topk(z, b, w.K)
    m = O.bf16_to_f32(O.kappa_inv(O.margin_keys(z, tau))).astype(np.float64)
    for p in range(3):
        sl = m[off[p]:off[p + 1]]
        q = np.quantile(sl, w.K / w.E, axis=0, method="inverted_cdf")
        np.testing.assert_array_equal(O.bf16_to_f32(bp[p]).astype(np.float64), q)
    np.testing.assert_array_equal(avg, (O.bf16_to_f32(bp).astype(np.float64).sum(0)) / 3)
    # another split of the same batch gives another average (Sec. 2: partition dependent)
    _, avg2, _ = B.rank_averaged_qb(z, b, w.K, [0, 1000, 9000])
    assert np.any(avg2 != avg)


def test_rank_average_skips_empty_shards():
    w = W.WORKLOADS["skew64"].with_T(4000, 2)
    z, b, _ = W.generate(w)
    bp, avg, _ = B.rank_averaged_qb(z, b, w.K, [0, 2000, 2000, 4000])
    assert np.all(bp[1] == 0x7FC0)
    np.testing.assert_array_equal(avg, (O.bf16_to_f32(bp[[0, 2]]).astype(np.float64).sum(0)) / 2)


def test_uniform_bins_against_exact_rationals():
    rng = np.random.default_rng(2)
    T, E = 300, 8
    z = O.f32_to_bf16_rne((rng.standard_normal((T, E)) * 2).astype(np.float32))
    tau = (rng.standard_normal(T) * 2).astype(np.float32)
    lo, hi, nb = -6.0, 6.0, 37
    bins = B.uniform_bins(z, tau, lo, hi, nb)
    m = (tau[:, None] - O.bf16_to_f32(z)).astype(np.float32)
    for t in range(T):
        for e in range(E):
            x = (Fraction(float(m[t, e])) - Fraction(lo)) * nb / (Fraction(hi) - Fraction(lo))
            j = min(max(math.floor(x), 0), nb - 1)
            if abs(x - round(x)) > Fraction(1, 10 ** 4):        # away from bin edges
                assert bins[t, e] == j


def test_histogram_estimate_lies_in_the_bin_of_the_exact_quantile():
    w = W.WORKLOADS["skew64"].with_T(9000, 3)
    z, b, off = W.generate(w)
    lo, hi, nb = -10.0, 10.0, 200
    counts, est, bn = B.histogram_qb(z, b, w.K, off, lo, hi, nb)
    assert np.all(counts.sum(axis=2) == np.diff(off)[:, None])
    _, _, tau = O.route_topk(z, b, w.K)
    m = np.sort((tau[:, None] - O.bf16_to_f32(z)).astype(np.float32), axis=0)
    r = O.quantile_rank(w.T, w.K, w.E)
    exact = m[r - 1].astype(np.float64)
    width = (hi - lo) / nb
    assert np.all(np.abs(est - exact) <= width)
    jb = B.uniform_bins(z, tau, lo, hi, nb)
    j = np.array([jb[np.argsort((tau - O.bf16_to_f32(z[:, e])).astype(np.float32), kind="stable")[r - 1], e]
                  for e in range(w.E)])
    assert np.all(est >= lo + j * width - 1e-12) and np.all(est <= lo + (j + 1) * width + 1e-12)
    assert abs(float(bn.astype(np.float64).sum())) < 1e-3


@pytest.mark.parametrize("mutant", ["divide_by_all_shards", "interp_after_bin"])
def test_variant_pins_catch_planted_mistakes(monkeypatch, mutant):
    if mutant == "divide_by_all_shards":
        orig = B.rank_averaged_qb

        def bad(z_bits, b, K, part_off):
            bp, avg, bn = orig(z_bits, b, K, part_off)
            P = len(part_off) - 1
            vals = np.where(bp == 0x7FC0, 0.0, O.bf16_to_f32(bp).astype(np.float64))
            avg = vals.sum(0) / P
            return bp, avg, bn
        monkeypatch.setattr(B, "rank_averaged_qb", bad)
        fns = (test_rank_average_skips_empty_shards,)
    else:
        orig_hq = B.histogram_qb

        def bad(z_bits, b, K, part_off, lo, hi, nbins):
            counts, est, bn = orig_hq(z_bits, b, K, part_off, lo, hi, nbins)
            return counts, est + (hi - lo) / nbins, bn        # reads the quantile one bin too high
        monkeypatch.setattr(B, "histogram_qb", bad)
        fns = (test_histogram_estimate_lies_in_the_bin_of_the_exact_quantile,)
    failed = False
    for fn in fns:
        try:
            fn()
        except AssertionError:
            failed = True
    assert failed, mutant


# ------------------------------------------------ router backward with LEI ---
def test_router_backward_is_the_autograd_gradient():
    """Eq. 1 and Eq. lei: the logits' gradient of sum_{t,k} g_{t,k} s_{t,idx} plus
    the injected sum_{t,e} inj_{p(t),e} s_{t,e}, by torch autograd in float64."""
    import torch
    rng = np.random.default_rng(4)
    T, E, K = 40, 16, 3
    z = O.f32_to_bf16_rne((rng.standard_normal((T, E)) * 3).astype(np.float32))
    idx = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    gs = rng.standard_normal((T, K)).astype(np.float32)
    off = np.array([0, 15, 15, 40])
    inj = (rng.standard_normal((3, E)) * 1e-2).astype(np.float32)
    zt = torch.tensor(O.bf16_to_f32(z).astype(np.float64), requires_grad=True)
    s = torch.sigmoid(zt)
    loss = (torch.tensor(gs, dtype=torch.float64) * s.gather(1, torch.tensor(idx, dtype=torch.int64))).sum()
    pid = np.searchsorted(off, np.arange(T), side="right") - 1
    loss = loss + (torch.tensor(inj.astype(np.float64)[pid]) * s).sum()
    loss.backward()
    got = B.lei_router_backward(z, idx, gs, inj, off)
    np.testing.assert_allclose(got, zt.grad.numpy(), rtol=1e-12, atol=1e-300)
    # without injection only the selected experts move
    plain = B.lei_router_backward(z, idx, gs, None, off)
    mask = np.zeros((T, E), bool)
    mask[np.repeat(np.arange(T), K), idx.ravel()] = True
    assert np.all(plain[~mask] == 0)
    assert B.lei_router_backward(np.zeros((1, 2), np.uint16), np.array([[0]]), np.array([[1.0]], np.float32),
                                 None, [0, 1])[0, 0] == 0.25          # sigmoid'(0) = 1/4
