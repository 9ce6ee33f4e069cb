"""Pins of the CPU oracle to things other than itself (CPU only).

The paper prints no numerical worked example, so the oracle is pinned by
  * library routines it must reduce to (torch's BF16 rounding, numpy's
    inverted-CDF quantile),
  * exhaustive checks of the 16-bit encoding,
  * brute force over subsets and the Appendix B objectives in exact rationals,
  * layers worked by hand (tests/golden/hand_examples.json),
  * invariants and metamorphic relations of Algorithm 1 and Eq. 2,
and a final test plants plausible mistakes in the oracle and checks that these
pins catch each one.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import brute
from oracle import eqb_oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


# ---------------------------------------------------------------- BF16 ----
def torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x32, np.float32)).to(torch.bfloat16) \
        .view(torch.int16).numpy().view(np.uint16)


def test_bf16_widening_matches_torch():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    finite = (bits & 0x7F80) != 0x7F80
    ours = O.bf16_to_f32(bits[finite])
    ref = torch.from_numpy(bits[finite].view(np.int16)).view(torch.bfloat16).float().numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_rounding_matches_torch_on_every_high_half():
    """Every finite high half with low halves at and around the tie point."""
    hi = np.arange(65536, dtype=np.uint32)
    hi = hi[(hi & 0x7F80) != 0x7F80]
    rng = np.random.default_rng(7)
    lows = [0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF]
    for low in lows + [None]:
        lo = rng.integers(0, 65536, size=hi.size, dtype=np.uint32) if low is None else np.uint32(low)
        bits = (hi << 16) | lo
        x = bits.view(np.float32)
        assert np.array_equal(O.f32_to_bf16_rne(x), torch_bf16(x)), hex(low or 0)


def test_bf16_rounding_exhaustive_against_torch():
    """Every finite float32 pattern (2^32 minus Inf/NaN), in chunks of 2^20:
    the oracle's nearest-neighbour rounding equals torch's conversion."""
    from concurrent.futures import ThreadPoolExecutor

    def chunk(c):
        s = c << 20
        bits = np.arange(s, s + (1 << 20), dtype=np.uint64).astype(np.uint32)
        bits = bits[(bits & 0x7F800000) != 0x7F800000]
        if bits.size == 0:
            return -1
        x = bits.view(np.float32)
        bad = np.flatnonzero(O.f32_to_bf16_rne(x) != torch_bf16(x))
        return int(bits[bad[0]]) if bad.size else -1

    threads = max(1, min(8, os.cpu_count() or 1))
    torch_threads = torch.get_num_threads()
    torch.set_num_threads(1)
    try:
        with ThreadPoolExecutor(threads) as ex:
            first_bad = [b for b in ex.map(chunk, range(1 << 12)) if b >= 0]
    finally:
        torch.set_num_threads(torch_threads)
    assert not first_bad, f"rounding differs at {first_bad[0]:#010x}"


def test_bf16_rounding_random_patterns():
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 1 << 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]
    x = bits.view(np.float32)
    assert np.array_equal(O.f32_to_bf16_rne(x), torch_bf16(x))


@pytest.mark.parametrize("x_bits,expect", [
    (0x3F808000, 0x3F80),   # 1 + 2^-8: tie, keep the even pattern 3F80
    (0x3F818000, 0x3F82),   # 1 + 3*2^-8: tie, round up to the even 3F82
    (0x3F808001, 0x3F81),   # just above the tie
    (0xBF808000, 0xBF80),   # negative tie
    (0x00000001, 0x0000),   # smallest binary32 subnormal underflows to +0
    (0x80000001, 0x8000),   # ... and keeps its sign
    (0x00008000, 0x0000),   # tie between 0 and the smallest BF16 subnormal -> even (0)
    (0x00018000, 0x0002),   # tie between subnormals 1 and 2 -> even (2)
    (0x7F7FFFFF, 0x7F80),   # binary32 max rounds to infinity
    (0x7F7F7FFF, 0x7F7F),   # below the overflow midpoint stays finite
])
def test_bf16_rounding_hand_values(x_bits, expect):
    x = np.array([x_bits], np.uint32).view(np.float32)
    assert int(O.f32_to_bf16_rne(x)[0]) == expect


# ---------------------------------------------------------------- kappa ---
def _total_order_rank(bits: np.ndarray) -> np.ndarray:
    """Position of each non-NaN BF16 pattern in IEEE totalOrder (-0 before +0)."""
    vals = O.bf16_to_f32(bits).astype(np.float64)
    sign = (bits >> 15).astype(np.int64)
    # numeric value first; among equal values (only +-0) the negative sign first
    order = np.lexsort((-sign, vals))
    rank = np.empty(bits.size, np.int64)
    rank[order] = np.arange(bits.size)
    return rank


def test_kappa_is_an_order_preserving_bijection():
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    keys = O.kappa(allbits)
    assert np.unique(keys).size == 65536
    assert np.array_equal(O.kappa_inv(keys), allbits)
    notnan = ~(((allbits & 0x7F80) == 0x7F80) & ((allbits & 0x7F) != 0))
    b = allbits[notnan]
    k = keys[notnan].astype(np.int64)
    rank = _total_order_rank(b)
    # key order equals totalOrder: sorting by key gives ranks 0..n-1 in order
    assert np.array_equal(rank[np.argsort(k)], np.arange(b.size))
    assert O.kappa(np.array([0x8000], np.uint16))[0] < O.kappa(np.array([0x0000], np.uint16))[0]


# ------------------------------------------------------ top-K and tau -----
def _tiny_rows(rng, T, E, grid):
    if grid:
        k = rng.integers(-3, 4, size=(T, E))
        z = O.f32_to_bf16_rne((k / 2.0).astype(np.float32))
        z[(k == 0) & (rng.random((T, E)) < 0.5)] = 0x8000
        b = (rng.integers(-2, 3, size=E) / 4.0).astype(np.float32)
        b[rng.random(E) < 0.3] = -0.0
    else:
        z = O.f32_to_bf16_rne(rng.standard_normal((T, E)).astype(np.float32))
        b = (rng.standard_normal(E) * 0.3).astype(np.float32)
    return z, b


@pytest.mark.parametrize("E", [2, 3, 4, 5, 6])
@pytest.mark.parametrize("grid", [True, False])
def test_topk_and_tau_against_brute_force(E, grid):
    rng = np.random.default_rng(100 * E + grid)
    for trial in range(4):
        z, b = _tiny_rows(rng, 12, E, grid)
        # s from the exact rational sums, rounded by the brute-force helper
        s_bits = np.array(brute.biased_scores_exact(z, b), np.uint32)
        s = s_bits.view(np.float32)
        for K in range(1, E):
            idx, score, tau = O.route_topk(z, b, K)
            for t in range(z.shape[0]):
                row = [float(v) for v in s[t]]
                want = brute.topk_subset(row, K)
                assert list(idx[t]) == want, (t, row, K)
                tau_val = brute.tau_by_threshold_identity(row, K)
                assert float(tau[t]) == float(tau_val)
                # the bit pattern is the one of the element ranked K-th (0-based)
                full = sorted(range(E), key=lambda e: (-row[e], e))
                assert tau[t].view(np.uint32) == s_bits[t, full[K]]


def test_scores_are_unbiased_sigmoid():
    rng = np.random.default_rng(5)
    z = O.f32_to_bf16_rne((rng.standard_normal((64, 16)) * 4).astype(np.float32))
    b = (rng.standard_normal(16) * 3).astype(np.float32)
    idx, score, _ = O.route_topk(z, b, 5)
    zf = O.bf16_to_f32(z)
    for t in range(64):
        for k in range(5):
            x = float(zf[t, idx[t, k]])
            ref = np.float32(0.5 * (1.0 + math.tanh(0.5 * x)))      # independent form
            assert abs(int(score[t, k].view(np.int32)) - int(ref.view(np.int32))) <= 1


def _f32(v):
    return np.float32(v)


@pytest.mark.parametrize("case", ["random", "ties", "tiny", "zeros"])
def test_biased_scores_equal_rounded_exact_sums(case):
    """Reading R1 (Sec. 2, I_t = TopK(z_t + b)): s = z + b is one binary32
    addition rounded to nearest, ties to even.  The reference rounds the
    exact rational sum itself (tests/brute.py), never a float add."""
    rng = np.random.default_rng({"random": 1, "ties": 2, "tiny": 3, "zeros": 4}[case])
    if case == "random":
        # logits of every scale, biases with full 24-bit significands
        z = rng.integers(0, 65536, size=(64, 16), dtype=np.uint32).astype(np.uint16)
        z[(z & 0x7F80) == 0x7F80] &= 0xBFFF           # keep them finite
        b = (rng.standard_normal(16) * 2.0 ** rng.integers(-30, 30, size=16)).astype(np.float32)
    elif case == "ties":
        # z = 1 + k/128 and b = (2j+1) * 2^-24 put z + b exactly halfway
        # between two binary32 neighbours: the even one must win
        z = O.f32_to_bf16_rne((1.0 + np.arange(64) / 128.0).astype(np.float32))[:, None].repeat(8, 1)
        b = ((2 * np.arange(8) + 1) * 2.0 ** -24).astype(np.float32)
        b[4:] = -b[4:]
    elif case == "tiny":
        # subnormal and smallest-normal sums
        z = np.array([[0x0000, 0x8000, 0x0080, 0x8080, 0x0001, 0x8001, 0x0081, 0x0100]] * 8, np.uint16)
        b = np.array([2.0 ** -149, -(2.0 ** -149), 2.0 ** -126, -(2.0 ** -126) + 2.0 ** -149,
                      3 * 2.0 ** -149, -(2.0 ** -127), 2.0 ** -130, -(2.0 ** -125)], np.float32)
    else:
        # signed zeros: -0 + -0 = -0, every other exact zero sum is +0
        z = np.array([[0x0000, 0x8000, 0x8000, 0x3F80, 0xBF80, 0x0000]], np.uint16)
        b = np.array([-0.0, -0.0, 0.0, -1.0, 1.0, 0.0], np.float32)
    want = np.array(brute.biased_scores_exact(z, b), np.uint32)
    got = O.biased_scores(z, b).view(np.uint32)
    assert np.array_equal(got, want)
    if case == "zeros":
        assert [hex(x) for x in want[0]] == ["0x0", "0x80000000", "0x0", "0x0", "0x0", "0x0"]


def test_topk_matches_stable_argsort_on_tie_free_rows():
    rng = np.random.default_rng(9)
    z = O.f32_to_bf16_rne(rng.standard_normal((500, 64)).astype(np.float32))
    b = (rng.standard_normal(64) * 0.1).astype(np.float32)
    idx, _, tau = O.route_topk(z, b, 6)
    s = np.array(brute.biased_scores_exact(z, b), np.uint32).view(np.float32)
    order = np.argsort(-s, axis=1, kind="stable")
    assert np.array_equal(idx, order[:, :6])
    assert np.array_equal(tau, np.sort(s, axis=1)[:, -7])


# ------------------------------------------------------------ quantile ----
@pytest.mark.parametrize("seed", range(6))
def test_quantile_against_counts_dual_and_numpy(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 24))
    k = rng.integers(-6, 7, size=n)
    bits = O.f32_to_bf16_rne((k / 8.0).astype(np.float32))
    bits[(k == 0) & (rng.random(n) < 0.5)] = 0x8000
    keys = O.kappa(bits)
    vals = O.bf16_to_f32(bits).astype(np.float64)
    for r in range(1, n + 1):
        kstar = O.select_by_sort(keys[:, None], r)[0]
        assert kstar == brute.quantile_by_counts([int(x) for x in keys], r)
        v = float(O.bf16_to_f32(O.kappa_inv(np.array([kstar], np.uint16)))[0])
        assert v == float(brute.quantile_by_dual(list(vals), r))
        assert v == np.quantile(vals, r / n, method="inverted_cdf")


def test_quantile_rank_rule():
    assert O.quantile_rank(4096, 2, 8) == 1024
    assert O.quantile_rank(4194304, 8, 256) == 131072
    assert O.quantile_rank(10, 3, 8) == 4          # 30/8 = 3.75 rounds up
    # ceil(n*q) is numpy's inverted-CDF index for q = K/E (dyadic, exact)
    x = np.arange(10.0)
    assert np.quantile(x, 3 / 8, method="inverted_cdf") == x[O.quantile_rank(10, 3, 8) - 1]


# ----------------------------------------------------- full tiny layers ---
def _brute_layer(z, b, K, part_off):
    """Everything from subsets, rationals, torch rounding and plain loops."""
    T, E = z.shape
    s = np.array(brute.biased_scores_exact(z, b), np.uint32).view(np.float32)
    zf = O.bf16_to_f32(z)
    idx = np.array([brute.topk_subset([float(v) for v in s[t]], K) for t in range(T)])
    order = [sorted(range(E), key=lambda e: (-float(s[t, e]), e)) for t in range(T)]
    tau = np.array([s[t, order[t][K]] for t in range(T)], np.float32)
    m32 = tau[:, None] - zf                         # binary32 subtraction
    mbits = torch_bf16(m32)                         # library rounding
    r = -(-T * K // E)
    # r-th smallest margin in IEEE totalOrder, per expert
    bhat = []
    for e in range(E):
        col = list(mbits[:, e])
        col.sort(key=lambda x: (brute.bf16_value(int(x)), -(int(x) >> 15)))
        bhat.append(int(col[r - 1]))
    keys = O.kappa(mbits)                           # kappa is pinned exhaustively above
    P = len(part_off) - 1
    H = np.zeros((P, E, 256), np.int64)
    for p in range(P):
        for t in range(part_off[p], part_off[p + 1]):
            for e in range(E):
                H[p, e, keys[t, e] >> 8] += 1
    Hs = H.sum(0)
    u = [min(uu for uu in range(256) if Hs[e, :uu + 1].sum() >= r) for e in range(E)]
    rho = [r - int(Hs[e, :u[e]].sum()) for e in range(E)]
    L = np.zeros((P, E, 256), np.int64)
    for p in range(P):
        for t in range(part_off[p], part_off[p + 1]):
            for e in range(E):
                if keys[t, e] >> 8 == u[e]:
                    L[p, e, keys[t, e] & 0xFF] += 1
    Ls = L.sum(0)
    v = [min(vv for vv in range(256) if Ls[e, :vv + 1].sum() >= rho[e]) for e in range(E)]
    load = np.zeros((P, E), np.int64)
    for p in range(P):
        for t in range(part_off[p], part_off[p + 1]):
            for e in idx[t]:
                load[p, e] += 1
    return dict(idx=idx, tau=tau, r=r, u=u, rho=rho, v=v, H_p=H, L_p=L, load=load,
                bhat=bhat)


def check_layer_against_brute(z, b, K, part_off):
    got = O.run_layer(z, b, K, part_off)
    want = _brute_layer(z, b, K, part_off)
    assert np.array_equal(got["idx"], want["idx"])
    assert np.array_equal(got["tau"].view(np.uint32), want["tau"].view(np.uint32))
    assert got["r"] == want["r"]
    assert np.array_equal(got["load"], want["load"])
    assert np.array_equal(got["H_p"], want["H_p"])
    assert list(got["u"]) == want["u"]
    assert list(got["rho"]) == want["rho"]
    assert np.array_equal(got["L_p"], want["L_p"])
    assert list(got["v"]) == want["v"]
    assert [int(x) for x in got["bhat"]] == want["bhat"]
    # u, v reassemble the quantile: b_hat = kappa^-1(u, v) (Algorithm 1, step 6)
    kk = (np.array(want["u"]) << 8 | np.array(want["v"])).astype(np.uint16)
    assert [int(x) for x in O.kappa_inv(kk)] == want["bhat"]


@pytest.mark.parametrize("seed", range(8))
def test_layer_against_brute_force(seed):
    rng = np.random.default_rng(1000 + seed)
    E = int(rng.integers(2, 7))
    T = int(rng.integers(1, 14))
    K = int(rng.integers(1, E))
    z, b = _tiny_rows(rng, T, E, grid=bool(seed % 2))
    cuts = np.sort(rng.integers(0, T + 1, size=int(rng.integers(0, 3))))
    part_off = np.concatenate([[0], cuts, [T]]).astype(np.int64)
    check_layer_against_brute(z, b, K, part_off)


# --------------------------------------------------------- hand-worked ----
def _hx(s):
    return int(s, 16)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_worked_examples(case):
    K = case["K"]
    if "z_bits" in case:
        z = np.array([[_hx(x) for x in row] for row in case["z_bits"]], np.uint16)
        b = np.array([_hx(x) for x in case["b_bits"]], np.uint32).view(np.float32)
    else:
        z = torch_bf16(np.array(case["z"], np.float32))
        b = np.array(case["b"], np.float32)
    got = O.run_layer(z, b, K)
    E = z.shape[1]
    assert got["idx"].tolist() == case["idx"]
    assert np.array_equal(got["score"], np.array(case["score"], np.float32))
    if "tau_bits" in case:
        assert got["tau"].view(np.uint32).tolist() == [_hx(x) for x in case["tau_bits"]]
    else:
        assert got["tau"].tolist() == case["tau"]
    assert got["load"][0].tolist() == case["load"]
    for name, arr in (("H_nonzero", got["H"]), ("L_nonzero", got["L"])):
        want = np.zeros((E, 256), np.int64)
        for e, bins in case[name].items():
            for u, c in bins.items():
                want[int(e), _hx(u)] = c
        assert np.array_equal(arr, want), name
    assert got["r"] == case["r"]
    assert got["u"].tolist() == [_hx(x) for x in case["u"]]
    assert got["rho"].tolist() == case["rho"]
    assert got["v"].tolist() == [_hx(x) for x in case["v"]]
    assert got["bhat"].tolist() == [_hx(x) for x in case["bhat_bits"]]
    if "b_next_bits" in case:
        assert got["b_next"].view(np.uint32).tolist() == [_hx(x) for x in case["b_next_bits"]]
    else:
        assert got["b_next"].tolist() == case["b_next"]


# ----------------------------------------------------------- invariants ---
def _small(name, T, P=None, seed_split=None):
    w = W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    if seed_split is not None:
        rng = np.random.default_rng(seed_split)
        cuts = np.sort(rng.integers(0, T + 1, size=w.P - 1))
        off = np.concatenate([[0], cuts, [T]]).astype(np.int64)
    return w, z, b, off


@pytest.mark.parametrize("name", W.WORKLOAD_ORDER)
def test_invariants_on_workload_shapes(name):
    w, z, b, off = _small(name, 3000, seed_split=3)
    R = O.run_layer(z, b, w.K, off)
    T, E = z.shape
    assert R["load"].sum() == w.K * T
    assert np.all(R["H"].sum(axis=1) == T)
    assert np.array_equal(R["H_p"].sum(axis=0), R["H"])
    for e in range(E):
        u = R["u"][e]
        assert R["L"][e].sum() == R["H"][e, u]
        assert 1 <= R["rho"][e] <= R["H"][e, u]
        col = R["keys"][:, e].astype(np.int64)
        kstar = int(O.kappa(R["bhat"][e:e + 1])[0])
        assert np.any(col == kstar)                               # attained
        assert (col < kstar).sum() < R["r"] <= (col <= kstar).sum()
    # centred bias: mean removed (float64 sum of float32 values is tiny)
    assert abs(float(np.sum(R["b_next"].astype(np.float64)))) < 1e-5 * E


def test_alg1_rules_and_full_histogram_agree_with_sort():
    w, z, b, off = _small("skew64", 5000)
    R = O.run_layer(z, b, w.K, off)
    r = R["r"]
    for e in range(z.shape[1]):
        c = np.cumsum(R["H"][e])
        u = int(np.argmax(c >= r))
        assert u == R["u"][e]
        assert R["rho"][e] == r - (c[u - 1] if u else 0)
        cl = np.cumsum(R["L"][e])
        assert int(np.argmax(cl >= R["rho"][e])) == R["v"][e]
        # the single-pass alternative: one 2^16-bin histogram of the whole key
        full = np.bincount(R["keys"][:, e], minlength=65536)
        k = int(np.argmax(np.cumsum(full) >= r))
        assert k == (R["u"][e] << 8 | R["v"][e])


def test_partition_invariance_including_empty_partitions():
    w, z, b, _ = _small("split128", 4000)
    one = O.run_layer(z, b, w.K, np.array([0, 4000]))
    off = np.array([0, 0, 1, 1700, 1700, 1701, 4000, 4000], np.int64)
    many = O.run_layer(z, b, w.K, off)
    for k in ("H", "L", "u", "v", "rho", "bhat", "b_next", "idx", "tau"):
        assert np.array_equal(one[k], many[k]), k
    assert np.array_equal(one["load"][0], many["load"].sum(0))
    assert many["H_p"][0].sum() == 0 and many["H_p"][1].sum() == w.E


def test_token_permutation_leaves_statistics_unchanged():
    w, z, b, _ = _small("tie64", 3000)
    R1 = O.run_layer(z, b, w.K)
    perm = np.random.default_rng(2).permutation(3000)
    R2 = O.run_layer(z[perm], b, w.K)
    for k in ("H", "L", "u", "v", "rho", "bhat", "b_next"):
        assert np.array_equal(R1[k], R2[k]), k
    assert np.array_equal(R1["load"], R2["load"])
    assert np.array_equal(R1["idx"][perm], R2["idx"])


def test_expert_permutation_permutes_outputs():
    w, z, b, _ = _small("skew64", 2000)
    R1 = O.run_layer(z, b, w.K)
    perm = np.random.default_rng(4).permutation(w.E)
    R2 = O.run_layer(z[:, perm], b[perm], w.K)
    # new column j is old expert perm[j]
    assert np.array_equal(perm[R2["idx"]], R1["idx"])     # tie-free data
    assert np.array_equal(R2["tau"], R1["tau"])
    for k in ("bhat", "b_next", "u", "v", "rho"):
        assert np.array_equal(R2[k], R1[k][perm]), k
    assert np.array_equal(R2["H"], R1["H"][perm])


def test_common_bias_shift_leaves_routing_and_centred_bias_unchanged():
    """Eq. 2: a common offset of b does not change Top-K; the quantile moves
    by the offset and the centring removes it.  On this grid every sum and
    margin is exact in binary32 and BF16, so the relation holds bit for bit."""
    rng = np.random.default_rng(8)
    T, E, K = 2048, 16, 3
    z = torch_bf16((rng.integers(-16, 17, size=(T, E)) / 4.0).astype(np.float32))
    b = (rng.integers(-4, 5, size=E) / 8.0).astype(np.float32)
    R1 = O.run_layer(z, b, K)
    R2 = O.run_layer(z, b + np.float32(0.25), K)
    assert np.array_equal(R1["idx"], R2["idx"])
    assert np.array_equal(R2["tau"], R1["tau"] + np.float32(0.25))
    bh1 = O.bf16_to_f32(R1["bhat"])
    bh2 = O.bf16_to_f32(R2["bhat"])
    assert np.array_equal(bh2, bh1 + np.float32(0.25))
    assert np.array_equal(R1["b_next"], R2["b_next"])


def test_centring_equals_exact_rational_mean_when_sums_are_exact():
    from fractions import Fraction
    rng = np.random.default_rng(12)
    for _ in range(20):
        E = int(rng.choice([8, 64, 256]))
        bh = torch_bf16((rng.standard_normal(E) * rng.choice([0.01, 1, 30])).astype(np.float32))
        got = O.centred_bias(bh)
        vals = [Fraction(float(x)) for x in O.bf16_to_f32(bh)]
        mean = sum(vals, Fraction(0)) / E
        want = np.array([np.float32(float(v - mean)) for v in vals], np.float32)
        assert np.array_equal(got, want)


def test_communication_closed_forms():
    """Sec. 3 'Communication': 2*E*256 int32 counts per layer."""
    E, layers = 256, 48
    per_layer = 2 * E * 256 * 4
    assert per_layer == 512 * 1024                       # 0.5 MiB
    assert per_layer * layers == 24 * 1024 * 1024        # 24 MiB per step
    assert (E * 2 ** 16 * 4) // per_layer == 128          # 128x below a 2^16-bin histogram


def test_load_subgradient_relation():
    """App. B: the partial derivative of Phi in b_e contains f_e(b) - r.

    For a small positive step d the one-sided slope of Phi along b_e equals
    (#tokens selecting e at b + d*1_e) - r; on tie-free data with d below the
    smallest gap this is f_e(b) - r."""
    from fractions import Fraction
    rng = np.random.default_rng(21)
    T, E, K = 40, 5, 2
    # rows of distinct values k/16, so no row has a tie at the boundary
    z = torch_bf16(np.stack([rng.permutation(np.arange(-20, 20))[:E] / 16.0
                             for _ in range(T)]).astype(np.float32))
    b = np.zeros(E, np.float32)
    R = O.run_layer(z, b, K)
    zf = O.bf16_to_f32(z).astype(np.float64)
    r = Fraction(T * K, E)

    def phi(bias):
        tot = Fraction(0)
        for t in range(T):
            row = sorted((Fraction(float(zf[t, e])) + bias[e] for e in range(E)), reverse=True)
            tot += sum(row[:K])
        return tot - r * sum(bias)

    d = Fraction(1, 1 << 20)
    base = [Fraction(0)] * E
    for e in range(E):
        step = list(base)
        step[e] += d
        slope = (phi(step) - phi(base)) / d
        assert slope == R["load"][0, e] - r


# ------------------------------------------------- planted mistakes -------
def _mut_tau_position(z_bits, b, K, chunk=1 << 15, threads=1):
    idx, score, tau = _orig_route(z_bits, b, K, chunk, threads)
    s = O.biased_scores(z_bits, b)
    return idx, score, np.sort(s, axis=1)[:, -K].astype(np.float32)   # K-th, not (K+1)st


def _mut_margin_sign(z_bits, tau, chunk=1 << 15, threads=1):
    m32 = O.bf16_to_f32(z_bits) - np.asarray(tau, np.float32)[:, None]
    return O.kappa(O.f32_to_bf16_rne(m32))


def _mut_kappa_signbit_only(bits):
    return (np.asarray(bits, np.uint16) ^ np.uint16(0x8000)).astype(np.uint16)


def _mut_rank_off_by_one(T, K, E):
    return max(1, T * K // E - 1)


def _mut_tie_higher_index(z_bits, b, K, chunk=1 << 15, threads=1):
    z_bits = np.asarray(z_bits, np.uint16)
    s = O.biased_scores(z_bits, b)
    E = s.shape[1]
    order = np.lexsort((-np.broadcast_to(np.arange(E), s.shape), -s), axis=-1)
    rows = np.arange(s.shape[0])
    idx = order[:, :K].astype(np.int32)
    tau = s[rows, order[:, K]]
    zsel = O.bf16_to_f32(z_bits[rows[:, None], order[:, :K]]).astype(np.float64)
    return idx, O.sigmoid64(zsel).astype(np.float32), tau


def _mut_biased_margin(z_bits, tau, chunk=1 << 15, threads=1):
    # uses z + b instead of the unbiased z (b of the grid test below)
    m32 = np.asarray(tau, np.float32)[:, None] - (O.bf16_to_f32(z_bits) + _PLANT_B[None, :])
    return O.kappa(O.f32_to_bf16_rne(m32))


def _mut_round_truncate(x):
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _mut_scores_rounded_to_bf16(z_bits, b):
    # s kept only to BF16 precision
    s = O.bf16_to_f32(z_bits) + np.asarray(b, np.float32)[None, :]
    return O.bf16_to_f32(O.f32_to_bf16_rne(s))


def _mut_bias_truncated_to_bf16(z_bits, b):
    # the bias cut to its top 16 bits before the addition
    bt = (np.asarray(b, np.float32).view(np.uint32) & 0xFFFF0000).view(np.float32)
    return O.bf16_to_f32(z_bits) + bt[None, :]


_orig_route = O.route_topk
_PLANT_B = np.array([0.0, 0.25, -0.5, 0.125], np.float32)


@pytest.mark.parametrize("attr,mutant", [
    ("route_topk", _mut_tau_position),
    ("margin_keys", _mut_margin_sign),
    ("kappa", _mut_kappa_signbit_only),
    ("quantile_rank", _mut_rank_off_by_one),
    ("route_topk", _mut_tie_higher_index),
    ("margin_keys", _mut_biased_margin),
    ("f32_to_bf16_rne", _mut_round_truncate),
])
def test_pins_catch_planted_mistakes(monkeypatch, attr, mutant):
    """Each plausible mistake in the oracle must make some pin above fail."""
    rng = np.random.default_rng(77)
    monkeypatch.setattr(O, attr, mutant)
    caught = False
    for trial in range(6):
        T, E, K = 9, 4, int(rng.integers(1, 4))
        z, _ = _tiny_rows(rng, T, E, grid=(trial % 2 == 0))
        if attr == "f32_to_bf16_rne":
            z = torch_bf16(rng.standard_normal((T, E)).astype(np.float32) * 3)
        off = np.array([0, 4, T], np.int64)
        try:
            check_layer_against_brute(z, _PLANT_B, K, off)
            if attr == "kappa":
                test_kappa_is_an_order_preserving_bijection()
            if attr == "f32_to_bf16_rne":
                test_bf16_rounding_random_patterns()
        except AssertionError:
            caught = True
            break
    assert caught, f"planted mistake in {attr} was not caught"


@pytest.mark.parametrize("mutant", [_mut_scores_rounded_to_bf16, _mut_bias_truncated_to_bf16])
def test_pins_catch_planted_score_mistakes(monkeypatch, mutant):
    """A mistake in the binary32 sum z + b (reading R1) must fail the pins on
    tie-free rows whose sums are inexact: the direct rounding pin and the
    brute-force layer, which takes its scores from exact rational sums."""
    monkeypatch.setattr(O, "biased_scores", mutant)
    with pytest.raises(AssertionError):
        test_biased_scores_equal_rounded_exact_sums("random")
    rng = np.random.default_rng(78)
    caught = 0
    for trial in range(4):
        T, E, K = 9, 5, int(rng.integers(1, 4))
        z = O.f32_to_bf16_rne(rng.standard_normal((T, E)).astype(np.float32))
        # full 24-bit significands: no sum is exact in BF16, and no two are equal
        b = (rng.standard_normal(E) * 0.37).astype(np.float32)
        s_exact = np.array(brute.biased_scores_exact(z, b), np.uint32)
        assert len({int(x) for x in s_exact.ravel()}) == s_exact.size        # tie-free
        assert np.all(s_exact & 0xFFFF)                                      # inexact in BF16
        try:
            check_layer_against_brute(z, b, K, np.array([0, 4, T], np.int64))
        except AssertionError:
            caught += 1
    assert caught == 4, "a planted mistake in biased_scores was not caught by the layer pin"
