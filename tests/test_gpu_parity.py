"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer outputs (Top-K indices, loads, coarse/fine counts, u, rho, v), tau,
the BF16 quantile and the centred bias are compared bit for bit; the sigmoid
scores within 1e-6 relative.  Inputs come from the seeded workload
generators; nothing the GPU computes is fed to the oracle.
"""
import functools
import os
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import eqb_oracle as O
from random_layers import random_layer_case

pytestmark = pytest.mark.gpu

SCORE_RTOL = 1e-6


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


@pytest.fixture(scope="module")
def eqb():
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2609_28053_amd import eqb as binding
    return binding


def say(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


def gpu_layer(eqb, z, b, K, part_off, fused=True):
    zt = torch.from_numpy(np.ascontiguousarray(z).view(np.int16)).cuda()
    bt = torch.from_numpy(np.ascontiguousarray(b, np.float32)).cuda()
    off = None if part_off is None else [int(x) for x in part_off]
    lay = eqb.run_layer(zt, bt, K, off, fused=fused)
    return lay.results()


def assert_parity(got, want, K, check_parts=True):
    assert got["dev_status"] == 0
    np.testing.assert_array_equal(got["idx"], want["idx"])
    np.testing.assert_array_equal(got["tau"].view(np.uint32), want["tau"].view(np.uint32))
    ws = want["score"].astype(np.float64)
    err = np.abs(got["score"].astype(np.float64) - ws)
    assert np.all(err <= SCORE_RTOL * np.abs(ws)), float(np.max(err / np.abs(ws)))
    if check_parts:
        np.testing.assert_array_equal(got["load"], want["load"])
        np.testing.assert_array_equal(got["H_p"], want["H_p"])
        np.testing.assert_array_equal(got["L_p"], want["L_p"])
    np.testing.assert_array_equal(got["load"].sum(0), want["load"].sum(0))
    np.testing.assert_array_equal(got["H"], want["H"])
    np.testing.assert_array_equal(got["L"], want["L"])
    assert got["r"] == want["r"]
    np.testing.assert_array_equal(got["u"], want["u"])
    np.testing.assert_array_equal(got["rho"], want["rho"])
    np.testing.assert_array_equal(got["v"], want["v"])
    np.testing.assert_array_equal(got["bhat"], want["bhat"])
    np.testing.assert_array_equal(got["b_next"].view(np.uint32), want["b_next"].view(np.uint32))


@functools.lru_cache(maxsize=4)
def workload(name, T=None, P=None):
    w = W.WORKLOADS[name] if T is None else W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    return w, z, b, off


@functools.lru_cache(maxsize=2)
def oracle_for(name, T=None, P=None):
    w, z, b, off = workload(name, T, P)
    return O.run_layer(z, b, w.K, off, threads=_threads())


# ------------------------------------------------- multi-tile, ragged -----
SMALL = [("tiny", 4096 + 517, 3), ("skew64", 20011, 4), ("split128", 9973, 8),
         ("tie64", 16411, 2), ("large256", 7001, 16), ("neg256", 12007, 4),
         ("signs64", 9001, 2)]


@pytest.mark.parametrize("name,T,P", SMALL, ids=[s[0] for s in SMALL])
def test_parity_small(eqb, name, T, P):
    w, z, b, off = workload(name, T, P)
    say(f"small {name} T={T} E={w.E} K={w.K} P={P}")
    want = oracle_for(name, T, P)
    assert_parity(gpu_layer(eqb, z, b, w.K, off, fused=True), want, w.K)
    assert_parity(gpu_layer(eqb, z, b, w.K, off, fused=False), want, w.K)


# ---------------------------------------------------------- full sizes ----
@pytest.mark.parametrize("name", W.WORKLOAD_ORDER)
def test_parity_full_size(eqb, name):
    w, z, b, off = workload(name)
    say(f"full {name} T={w.T} E={w.E} K={w.K} P={w.P} oracle threads={_threads()}")
    want = oracle_for(name)
    say(f"full {name}: oracle done, running GPU")
    got = gpu_layer(eqb, z, b, w.K, off)
    assert_parity(got, want, w.K)
    # partition invariance: one partition gives the same statistics
    one = gpu_layer(eqb, z, b, w.K, None)
    for k in ("H", "L", "u", "v", "rho", "bhat", "b_next", "idx", "tau"):
        np.testing.assert_array_equal(one[k], got[k])
    np.testing.assert_array_equal(one["load"][0], got["load"].sum(0))
    # the one-call layer (dynamic tails, several count slabs per partition),
    # twice on one workspace, at the size and launch configuration the bench
    # times
    say(f"full {name}: one-call layer")
    lay = eqb.Layer(w.T, w.E, w.K, w.P)
    zt = torch.from_numpy(np.ascontiguousarray(z).view(np.int16)).cuda()
    bt = torch.from_numpy(np.ascontiguousarray(b, np.float32)).cuda()
    po = eqb.PartOffsets([int(x) for x in off])
    for _ in range(2):
        lay.step(zt, bt, po, sums=True)
        res = lay.step_results()
        assert res["dev_status"] == 0 and res["workspace_zero"]
        for k in ("idx", "load", "H", "L", "bhat"):
            np.testing.assert_array_equal(np.asarray(res[k]), np.asarray(want[k]), err_msg=k)
        np.testing.assert_array_equal(res["tau"].view(np.uint32), want["tau"].view(np.uint32))
        np.testing.assert_array_equal(res["b_next"].view(np.uint32), want["b_next"].view(np.uint32))
        ws = want["score"].astype(np.float64)
        assert np.all(np.abs(res["score"].astype(np.float64) - ws) <= SCORE_RTOL * np.abs(ws))


# ------------------------------------------------------------ edge cases --
@pytest.mark.parametrize("E", [8, 16, 32, 64, 128, 256])
def test_every_E_and_K_extremes(eqb, E):
    rng = np.random.default_rng(E)
    for T in (1, 37, 2 * 1024 + 5):
        z = O.f32_to_bf16_rne((rng.standard_normal((T, E)) * 2).astype(np.float32))
        b = (rng.standard_normal(E) * 0.3).astype(np.float32)
        for K in sorted({1, E // 2, E - 1}):
            say(f"edge E={E} T={T} K={K}")
            off = np.array([0, T // 3, T // 3, T], np.int64)
            assert_parity(gpu_layer(eqb, z, b, K, off), O.run_layer(z, b, K, off), K)


@pytest.mark.parametrize("E,K", [(64, 8), (64, 6), (128, 6), (256, 8), (256, 6)])
def test_lists_run_dry(eqb, E, K):
    """Rows whose top ranks crowd into the experts of one lane.  The fast
    route kernel keeps five keys per lane at E >= 64 (lane g of a row holds
    the experts with (e >> 2) % 8 == g); a lane holding more of the top K+1
    keys runs dry, and the row is extracted again with refilled lists.  Some
    rows also carry exact ties, so dry rows meet the exact ordering of tied
    scores."""
    rng = np.random.default_rng(1000 + E + K)
    T = 3001
    x = rng.standard_normal((T, E)).astype(np.float32)
    lane = (np.arange(E) >> 2) % 8
    hot = rng.integers(0, 8, T)
    crowd = rng.random(T) < 0.6
    boost = np.where(crowd[:, None] & (lane[None, :] == hot[:, None]), np.float32(6.0), np.float32(0.0))
    x = x + boost
    tie_rows = rng.random(T) < 0.2
    x[tie_rows] = np.round(x[tie_rows] * 2) / 2          # many equal logits in these rows
    z = O.f32_to_bf16_rne(x.astype(np.float32))
    b = np.zeros(E, np.float32)
    b[rng.integers(0, E, 5)] = np.float32(0.25)
    off = np.array([0, 1000, 2001, T], np.int64)
    say(f"dry lists E={E} K={K} T={T}")
    assert_parity(gpu_layer(eqb, z, b, K, off), O.run_layer(z, b, K, off), K)


@pytest.mark.parametrize("E,K", [(64, 6), (128, 8), (256, 8), (256, 6), (256, 7)])
def test_dry_lane_next_key(eqb, E, K):
    """A lane of the fast kernel (five keys per lane at E >= 64; lane g holds
    the experts with (e >> 2) % 8 == g) that holds exactly five of the top
    K+1 keys pops its whole list; its next key is then found by a scan.
    Each row puts five experts of one lane on top and the rest of the top K+1
    in other lanes, and places that lane's sixth expert (a) far below rank
    K, (b) just below rank K, (c) on rank K's score (a tie that the lower
    index breaks), (d) just above rank K (the rounds missed it and the row is
    extracted again), or (e) two binary32 ulps below rank K's score, sharing
    its top 24 bits (the run past rank K continues)."""
    rng = np.random.default_rng(4100 + E + K)
    T = 5 * 1200 + 7
    lane = (np.arange(E) >> 2) % 8
    x = (rng.standard_normal((T, E)) * 0.5 - 3.0).astype(np.float32)
    # every expert outside lane 0 carries +2^-20: sums among them keep their
    # ties, and a lane-0 expert on the same logit scores 2 ulps lower (the
    # scores near rank K lie in [4, 8))
    b = np.where(lane == 0, np.float32(0.0), np.float32(2.0 ** -20)).astype(np.float32)
    rank_k = np.float32(6.0 - 0.5 * (K - 5))
    for t in range(T):
        c = t % 5
        h = 0 if c == 4 else int(rng.integers(1, 8))
        mine = rng.permutation(np.flatnonzero(lane == h))
        other = rng.permutation(np.flatnonzero((lane != h) & (lane != 0)))
        x[t, mine[:5]] = 8.0 + np.arange(5)[::-1]            # ranks 0..4, one lane
        x[t, other[:K - 4]] = 6.0 - 0.5 * np.arange(K - 4)   # ranks 5..K, other lanes
        x[t, mine[5]] = {0: -2.0, 1: rank_k - 0.25, 2: rank_k, 3: rank_k + 0.25, 4: rank_k}[c]
    z = O.f32_to_bf16_rne(x.astype(np.float32))
    off = np.array([0, T // 2, T], np.int64)
    say(f"dry lane next key E={E} K={K} T={T}")
    assert_parity(gpu_layer(eqb, z, b, K, off), O.run_layer(z, b, K, off), K)


# Every routing kernel the library dispatches for E >= 64: the unrolled K = 2
# kernel on an ordinary bias (its common path), the generic-K fast kernel
# (extraction loop with list refills, G = 8 lanes per row) for the K it
# serves, and the exact 64-bit kernel above K = 14 (Sec. 2 allows any
# 1 <= K < E).
ROUTE_VARIANTS = [(E, K) for E in (64, 128, 256) for K in (3, 5, 7, 10, 14)] + \
    [(64, 2), (256, 2), (256, 15), (256, 16)]


def _variant_inputs(E, K, T):
    """Skewed logits (per-expert offsets, an ordinary binary32 bias) with
    three kinds of hard rows mixed in: rows whose top ranks crowd into the
    experts of one lane of the fast kernel (lane g holds (e >> 2) % 8 == g),
    so its list runs dry; rows on a half-step grid, full of exact ties, also
    at the cutoff; and rows whose logits are all equal."""
    rng = np.random.default_rng(7000 + 17 * E + K)
    x = (rng.standard_normal((T, E)) + rng.standard_normal(E) * 0.7).astype(np.float32)
    kind = rng.random(T)
    lane = (np.arange(E) >> 2) % 8
    hot = rng.integers(0, 8, T)
    crowd = kind < 0.08
    x = x + np.where(crowd[:, None] & (lane[None, :] == hot[:, None]), np.float32(5.0), np.float32(0.0))
    grid = (kind >= 0.08) & (kind < 0.18)
    x[grid] = np.round(x[grid] * 2) / 2
    flat = kind >= 0.995
    x[flat] = np.float32(0.5)
    z = O.f32_to_bf16_rne(x.astype(np.float32))
    b = (rng.standard_normal(E) * 0.1).astype(np.float32)
    cuts = np.sort(rng.choice(np.arange(1, T), size=2, replace=False))
    off = np.array([0, cuts[0], cuts[1], T], np.int64)
    return z, b, off


@pytest.mark.parametrize("E,K", ROUTE_VARIANTS, ids=[f"E{e}-K{k}" for e, k in ROUTE_VARIANTS])
def test_route_variants(eqb, E, K):
    """Each shipped routing kernel against the oracle at the default grid and
    with one block, whose rows then span three 65,535-row segments (three LDS
    flushes of one partition, one of them across a partition boundary)."""
    T = 2 * 65535 + 31
    z, b, off = _variant_inputs(E, K, T)
    say(f"route variant E={E} K={K} T={T}: oracle")
    want = O.run_layer(z, b, K, off, threads=_threads())
    for cap in (0, 1, 5):
        say(f"route variant E={E} K={K} T={T} grid cap {cap}")
        try:
            eqb.eqb_set_max_blocks(cap)
            assert_parity(gpu_layer(eqb, z, b, K, off, fused=True), want, K)
            if cap == 0:
                assert_parity(gpu_layer(eqb, z, b, K, off, fused=False), want, K)
        finally:
            eqb.eqb_set_max_blocks(0)


@pytest.mark.parametrize("zbits", [0x3F00, 0xBF00, 0x8000], ids=["half", "minus_half", "minus_zero"])
@pytest.mark.parametrize("bzero", [0.0, -0.0], ids=["b_plus0", "b_minus0"])
def test_all_ties_constant_logits(eqb, zbits, bzero):
    for E, K in ((8, 2), (64, 6), (256, 8)):
        T = 3000
        z = np.full((T, E), zbits, np.uint16)                   # every logit equal
        b = np.full(E, bzero, np.float32)
        say(f"constant logits {zbits:#06x} b={bzero} E={E}")
        want = O.run_layer(z, b, K)
        got = gpu_layer(eqb, z, b, K, None)
        assert_parity(got, want, K)
        assert np.all(got["idx"] == np.arange(K))               # lower index wins every tie


def test_zero_scores_of_both_signs(eqb):
    # s = -0 where z = -0 meets b = -0, +0 elsewhere: every score is a zero,
    # the zeros tie, and the lower index wins
    rng = np.random.default_rng(11)
    for E, K in ((64, 4), (256, 8)):
        T = 4099
        z = np.where(rng.integers(0, 2, (T, E)).astype(bool), 0x8000, 0x0000).astype(np.uint16)
        b = np.where(rng.integers(0, 2, E).astype(bool), np.float32(-0.0), np.float32(0.0))
        say(f"signed-zero scores E={E}")
        want = O.run_layer(z, b, K)
        got = gpu_layer(eqb, z, b, K, None)
        assert_parity(got, want, K)
        assert np.all(got["idx"] == np.arange(K))


@pytest.mark.parametrize("E,K", [(64, 2), (128, 6), (256, 8), (32, 3)])
def test_huge_bias_takes_the_exact_path(eqb, E, K):
    # |b| >= 2^119 sends every row of the block through exact 64-bit keys;
    # with z at the BF16 maximum, z + b overflows to +inf for one expert
    rng = np.random.default_rng(E + K)
    T = 5003
    z = O.f32_to_bf16_rne((rng.standard_normal((T, E)) - 2.0).astype(np.float32))
    b = (rng.standard_normal(E) * 0.3).astype(np.float32)
    b[3] = np.float32(2.0 ** 120)
    say(f"bias 2^120 E={E} K={K}")
    assert_parity(gpu_layer(eqb, z, b, K, None), O.run_layer(z, b, K), K)
    b[5] = np.float32(3.0e38)
    z[::7, 5] = 0x7F7F                                            # z + b = +inf on these rows
    say(f"bias overflow E={E} K={K}")
    want = O.run_layer(z, b, K)
    assert np.isinf(want["tau"]).sum() == 0 and np.isposinf(
        O.bf16_to_f32(z[::7, 5]).astype(np.float32) + b[5]).all()
    assert_parity(gpu_layer(eqb, z, b, K, None), want, K)


def test_signed_zeros_and_subnormals(eqb):
    rng = np.random.default_rng(3)
    T, E, K = 5000, 64, 4
    pick = rng.integers(0, 6, size=(T, E))
    table = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x3F80], np.uint16)
    z = table[pick]
    b = np.where(rng.random(E) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    b[:4] = np.array([1e-40, -1e-40, 0.0, -0.0], np.float32)    # binary32 subnormals
    say("signed zeros and subnormals")
    assert_parity(gpu_layer(eqb, z, b, K, [0, 100, T]), O.run_layer(z, b, K, [0, 100, T]), K)


def test_wide_range_logits(eqb):
    rng = np.random.default_rng(4)
    T, E, K = 4000, 128, 8
    x = rng.standard_normal((T, E)) * np.exp(rng.uniform(-30, 30, size=(T, E)))
    z = O.f32_to_bf16_rne(np.clip(x, -1e30, 1e30).astype(np.float32))
    b = (rng.standard_normal(E) * 1e-3).astype(np.float32)
    say("wide-range logits")
    assert_parity(gpu_layer(eqb, z, b, K, None), O.run_layer(z, b, K), K)


def test_empty_and_single_token_partitions(eqb):
    w, z, b, _ = workload("skew64", 3001, 4)
    off = np.array([0, 0, 1, 1, 1500, 1501, 3001, 3001], np.int64)
    say("empty partitions")
    assert_parity(gpu_layer(eqb, z, b, w.K, off), O.run_layer(z, b, w.K, off), w.K)


def test_deterministic_repeat(eqb):
    w, z, b, off = workload("large256", 20000, 16)
    say("determinism")
    a = gpu_layer(eqb, z, b, w.K, off)
    c = gpu_layer(eqb, z, b, w.K, off)
    for k in a:
        np.testing.assert_array_equal(np.asarray(a[k]), np.asarray(c[k]))


def test_standalone_calls_match_fused(eqb):
    """eqb_margin_hist_pass1 and eqb_expert_load against the fused sweep."""
    w, z, b, off = workload("split128", 12345, 8)
    say("standalone pass 1 and load")
    zt = torch.from_numpy(z.view(np.int16)).cuda()
    bt = torch.from_numpy(b).cuda()
    offl = [int(x) for x in off]
    lay = eqb.run_layer(zt, bt, w.K, offl, fused=True)
    H1 = torch.zeros_like(lay.hist_hi)
    eqb.eqb_margin_hist_pass1(zt, lay.tau, H1, offl)
    ld = torch.zeros_like(lay.load)
    eqb.eqb_expert_load(lay.topk_idx, w.E, ld, offl)
    torch.cuda.synchronize()
    assert torch.equal(H1, lay.hist_hi)
    assert torch.equal(ld, lay.load)


def test_select_reports_rank_beyond_counts(eqb):
    E = 8
    say("select error status")
    hist = torch.zeros((1, E, 256), dtype=torch.int32, device="cuda")
    hist[0, :, 3] = 4                                   # four margins per expert
    sel = torch.empty(E, dtype=torch.int32, device="cuda")
    rib = torch.empty(E, dtype=torch.int64, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    eqb.eqb_select_quantile(1, hist, 4, sel, rib, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == 0 and torch.all(sel == 3) and torch.all(rib == 4)
    eqb.eqb_select_quantile(1, hist, 5, sel, rib, dev_status=st)
    torch.cuda.synchronize()
    assert st.item() == eqb.EQB_DEV_RANK_EXCEEDS_COUNT and torch.all(sel == -1)


def test_bf16_rounding_of_every_high_half_through_both_passes(eqb):
    """Margins tau - 0 = tau cover every finite high half with low halves at,
    around and away from the tie point; the coarse counts and the fine counts
    for every selected high byte must equal the oracle's, i.e. the device's
    BF16 rounding and key agree with the oracle on this whole set."""
    hi = np.arange(65536, dtype=np.uint32)
    hi = hi[(hi & 0x7F80) < 0x7F00]                    # keep tau - 0 far from overflow
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x4000, 0xC000], np.uint32)
    tau = ((hi[:, None] << 16) | lows[None, :]).ravel().view(np.float32)
    T, E = tau.size, 8
    z = np.zeros((T, E), np.uint16)
    z[:, 1] = 0x8000                                   # -0: tau - (-0) = tau as well
    keys = O.margin_keys(z, tau)
    say(f"rounding sweep T={T}")
    zt = torch.from_numpy(z.view(np.int16)).cuda()
    tt = torch.from_numpy(tau).cuda()
    H = torch.zeros((1, E, 256), dtype=torch.int32, device="cuda")
    eqb.eqb_margin_hist_pass1(zt, tt, H)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(H.cpu().numpy()[0], O.count_high(keys, [0, T])[0])
    L = torch.zeros((1, E, 256), dtype=torch.int32, device="cuda")
    for u in range(256):
        sel = torch.full((E,), u, dtype=torch.int32, device="cuda")
        L.zero_()
        eqb.eqb_margin_hist_pass2(zt, tt, sel, L)
        torch.cuda.synchronize()
        want = O.count_low(keys[:, :2], np.array([u, u]), [0, T])[0]
        np.testing.assert_array_equal(L.cpu().numpy()[0, :2], want, err_msg=f"u={u}")


def test_device_rounding_exhaustive_through_both_passes(eqb):
    """Every finite float32 value tau (2^32 minus Inf/NaN) is a margin tau - 0;
    its coarse count and its fine count inside every populated coarse bin must
    equal the oracle's, chunk by chunk (2^24 consecutive patterns per chunk).
    Counts aggregate, so one rounding error would need another that cancels it
    in the same bin of the same chunk to go unseen."""
    from concurrent.futures import ThreadPoolExecutor
    E, Tc = 8, 1 << 24

    def n_finite(c):
        return Tc // 2 if (c & 0x7F) == 0x7F else Tc      # exponent 0xFF above the midpoint

    def expected(c):
        bits = np.arange(c << 24, (c << 24) + n_finite(c), dtype=np.uint64).astype(np.uint32)
        keys = O.kappa(O.f32_to_bf16_rne(bits.view(np.float32)))
        hi = (keys >> 8).astype(np.int64)
        coarse = np.bincount(hi, minlength=256)
        fine = {int(u): np.bincount((keys[hi == u] & 0xFF).astype(np.int64), minlength=256)
                for u in np.flatnonzero(coarse)}
        return coarse, fine

    z = torch.zeros((Tc, E), dtype=torch.int16, device="cuda")
    H = torch.zeros((1, E, 256), dtype=torch.int32, device="cuda")
    L = torch.zeros((1, E, 256), dtype=torch.int32, device="cuda")
    with ThreadPoolExecutor(_threads()) as ex:
        for c, (coarse, fine) in zip(range(256), ex.map(expected, range(256))):
            if c % 32 == 0:
                say(f"device rounding chunk {c:#04x}")
            n = n_finite(c)
            start = (c << 24) - (1 << 32 if c >= 0x80 else 0)
            tau = torch.arange(start, start + n, dtype=torch.int32, device="cuda").view(torch.float32)
            zc = z[:n]
            H.zero_()
            eqb.eqb_margin_hist_pass1(zc, tau, H)
            got = H.cpu().numpy()[0]
            for e in range(E):
                np.testing.assert_array_equal(got[e], coarse, err_msg=f"coarse chunk {c:#x}")
            us = sorted(fine)
            for i in range(0, len(us), E):
                group = us[i:i + E]
                sel = torch.tensor(group + [group[0]] * (E - len(group)), dtype=torch.int32, device="cuda")
                L.zero_()
                eqb.eqb_margin_hist_pass2(zc, tau, sel, L)
                got = L.cpu().numpy()[0]
                for j, u in enumerate(group):
                    np.testing.assert_array_equal(got[j], fine[u], err_msg=f"fine chunk {c:#x} u={u:#x}")


# ------------------------------------------------- forced grid shapes (T7) --
@pytest.mark.parametrize("cap", [1, 3, 7])
def test_forced_grid_shapes(eqb, cap):
    """One block, or a few blocks whose row ranges do not divide T, must give
    the oracle's results: catches missing LDS barriers and flush races."""
    cases = [("skew64", 70001, 4), ("large256", 30011, 16), ("tiny", 5000, 3)]
    try:
        eqb.eqb_set_max_blocks(cap)
        for name, T, P in cases:
            w, z, b, off = workload(name, T, P)
            say(f"grid cap {cap}: {name} T={T} P={P}")
            want = oracle_for(name, T, P)
            assert_parity(gpu_layer(eqb, z, b, w.K, off, fused=True), want, w.K)
            assert_parity(gpu_layer(eqb, z, b, w.K, off, fused=False), want, w.K)
    finally:
        eqb.eqb_set_max_blocks(0)


def test_token_permutation_on_gpu(eqb):
    """Permuting the tokens of one partition permutes I and tau and leaves
    the loads and every EQB statistic unchanged."""
    w, z, b, _ = workload("large256", 20000, 16)
    perm = np.random.default_rng(9).permutation(w.T)
    say("token permutation")
    a = gpu_layer(eqb, z, b, w.K, None)
    c = gpu_layer(eqb, np.ascontiguousarray(z[perm]), b, w.K, None)
    np.testing.assert_array_equal(c["idx"], a["idx"][perm])
    np.testing.assert_array_equal(c["tau"].view(np.uint32), a["tau"][perm].view(np.uint32))
    for k in ("load", "H", "L", "u", "v", "rho", "bhat"):
        np.testing.assert_array_equal(c[k], a[k])
    np.testing.assert_array_equal(c["b_next"].view(np.uint32), a["b_next"].view(np.uint32))


def test_expert_permutation_on_gpu(eqb):
    """Permuting the experts (columns of z together with b) permutes every
    per-expert statistic; the cutoffs do not move (tau is a value of the row)."""
    w, z, b, off = workload("large256", 30011, 4)
    perm = np.random.default_rng(11).permutation(w.E)
    say("expert permutation")
    a = gpu_layer(eqb, z, b, w.K, off)
    c = gpu_layer(eqb, np.ascontiguousarray(z[:, perm]), np.ascontiguousarray(b[perm]), w.K, off)
    np.testing.assert_array_equal(c["tau"].view(np.uint32), a["tau"].view(np.uint32))
    np.testing.assert_array_equal(c["H_p"], a["H_p"][:, perm])
    np.testing.assert_array_equal(c["L_p"], a["L_p"][:, perm])
    for k in ("u", "rho", "v", "bhat"):
        np.testing.assert_array_equal(c[k], a[k][perm])
    np.testing.assert_array_equal(c["b_next"].view(np.uint32), a["b_next"][perm].view(np.uint32))
    # the selected experts are the same set (and loads follow them) wherever
    # the row has no tie at the cutoff, which the index rule would break
    # differently after the permutation
    zf = (z.astype(np.uint32) << 16).view(np.float32)
    s = zf + b[None, :]
    tau = a["tau"]
    untied = (s == tau[:, None]).sum(1) == 1
    sel_a = np.sort(a["idx"][untied], axis=1)
    sel_c = np.sort(perm[c["idx"][untied]], axis=1)
    np.testing.assert_array_equal(sel_c, sel_a)
    assert untied.mean() > 0.9


def test_common_bias_shift_on_gpu(eqb):
    """With logits and bias on the quarter-step grid every sum and every
    margin is exact (margins stay within BF16's 8 significant bits): adding
    1/4 to every bias leaves the routing unchanged, moves tau and the
    quantile by exactly 1/4, and leaves the centred bias unchanged (Eq. 2:
    only differences of b matter)."""
    w, z, _, off = workload("tie64", 50021, 2)
    b = (np.random.default_rng(5).integers(-4, 5, size=w.E) / 4).astype(np.float32)
    say("common bias shift")
    a = gpu_layer(eqb, z, b, w.K, off)
    c = gpu_layer(eqb, z, (b + np.float32(0.25)).astype(np.float32), w.K, off)
    np.testing.assert_array_equal(c["idx"], a["idx"])
    np.testing.assert_array_equal(c["load"], a["load"])
    np.testing.assert_array_equal(c["tau"], a["tau"] + np.float32(0.25))
    qa = (a["bhat"].astype(np.uint32) << 16).view(np.float32)
    qc = (c["bhat"].astype(np.uint32) << 16).view(np.float32)
    np.testing.assert_array_equal(qc, qa + np.float32(0.25))
    np.testing.assert_array_equal(c["b_next"], a["b_next"])


# ------------------------------------------------------ random shapes -----
@pytest.mark.parametrize("i", range(24))
def test_random_shapes_calls(eqb, i):
    """The separate calls (fused pass 1 and the standalone pass-1 kernel) on
    the seeded random layers of the one-call layer's test, per-partition
    counts included, under each case's grid cap."""
    w, z, b, off, cap = random_layer_case(i)
    say(f"random calls {i}: T={w.T} E={w.E} K={w.K} P={w.P} kind={w.kind} cuts={off.tolist()} cap={cap}")
    want = O.run_layer(z, b, w.K, off, threads=_threads())
    try:
        eqb.eqb_set_max_blocks(cap)
        for fused in (True, False):
            assert_parity(gpu_layer(eqb, z, b, w.K, off, fused=fused), want, w.K)
    finally:
        eqb.eqb_set_max_blocks(0)
