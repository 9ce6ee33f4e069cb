"""GPU parity of the one-call layer (eqb_layer) against the CPU oracle.

eqb_layer chains the route kernel, both selections and the fine pass with a
caller-owned workspace whose counter part must be zero when a layer starts
and is left zero when it ends (each selection clears the counts it has
summed); the rest is scratch for the fine pass's per-block count images.
Every layer below runs twice on the same workspace: the second run can only
match the oracle if the first left the counters zeroed.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import eqb_oracle as O
from random_layers import random_layer_case

pytestmark = pytest.mark.gpu

SCORE_RTOL = 1e-6


@pytest.fixture(scope="module")
def eqb():
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2609_28053_amd import eqb as binding
    return binding


def say(msg):
    print(f"[gpu-layer] {msg}", flush=True)
    sys.stdout.flush()


def check(got, want, K):
    assert got["dev_status"] == 0
    assert got["workspace_zero"], "the layer must leave its workspace counters zeroed"
    np.testing.assert_array_equal(got["idx"], want["idx"])
    np.testing.assert_array_equal(got["tau"].view(np.uint32), want["tau"].view(np.uint32))
    ws = want["score"].astype(np.float64)
    assert np.all(np.abs(got["score"] - ws) <= SCORE_RTOL * np.abs(ws))
    np.testing.assert_array_equal(got["load"], want["load"])
    np.testing.assert_array_equal(got["H"], want["H"])
    np.testing.assert_array_equal(got["L"], want["L"])
    np.testing.assert_array_equal(got["bhat"], want["bhat"])
    np.testing.assert_array_equal(got["b_next"].view(np.uint32), want["b_next"].view(np.uint32))


def run_twice(eqb, z, b, K, off, cap=0):
    T, E = z.shape
    P = 1 if off is None else len(off) - 1
    zt = torch.from_numpy(np.ascontiguousarray(z).view(np.int16)).cuda()
    bt = torch.from_numpy(np.ascontiguousarray(b, np.float32)).cuda()
    po = None if off is None else eqb.PartOffsets([int(x) for x in off])
    lay = eqb.Layer(T, E, K, P)
    out = []
    try:
        eqb.eqb_set_max_blocks(cap)
        for _ in range(2):
            lay.step(zt, bt, po, sums=True)
            out.append(lay.step_results())
    finally:
        eqb.eqb_set_max_blocks(0)
    return out


CASES = [("tiny", None, None), ("skew64", 20011, 4), ("split128", 9973, 8), ("tie64", 16411, 2),
         ("large256", 7001, 16), ("neg256", 12007, 4), ("signs64", 9001, 2), ("rank256", None, None)]


@pytest.mark.parametrize("name,T,P", CASES, ids=[c[0] for c in CASES])
def test_layer_matches_oracle(eqb, name, T, P):
    w = W.WORKLOADS[name] if T is None else W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    say(f"layer {name} T={w.T} E={w.E} K={w.K} P={w.P}")
    want = O.run_layer(z, b, w.K, off, threads=8)
    for got in run_twice(eqb, z, b, w.K, off):
        check(got, want, w.K)


def test_layer_empty_partitions_and_one_block(eqb):
    w = W.WORKLOADS["skew64"].with_T(70001, 1)
    z, b, _ = W.generate(w)
    off = np.array([0, 0, 1, 1, 35000, 70001, 70001], np.int64)
    want = O.run_layer(z, b, w.K, off, threads=8)
    for cap in (0, 1):
        say(f"layer empty partitions, grid cap {cap}")
        for got in run_twice(eqb, z, b, w.K, off, cap):
            check(got, want, w.K)


def test_layer_equals_the_call_sequence(eqb):
    """eqb_layer against the five separate calls on the full large workload."""
    w = W.WORKLOADS["large256"]
    z, b, off = W.generate(w)
    zt = torch.from_numpy(z.view(np.int16)).cuda()
    bt = torch.from_numpy(b).cuda()
    offl = [int(x) for x in off]
    say("layer vs call sequence, large256")
    ref = eqb.run_layer(zt, bt, w.K, offl).results()
    lay = eqb.Layer(w.T, w.E, w.K, w.P)
    lay.step(zt, bt, eqb.PartOffsets(offl), sums=True)
    got = lay.step_results()
    assert got["dev_status"] == 0 and got["workspace_zero"]
    for k in ("idx", "load", "H", "L", "bhat"):
        np.testing.assert_array_equal(got[k], ref[k])
    for k in ("tau", "score", "b_next"):
        np.testing.assert_array_equal(got[k].view(np.uint32), ref[k].view(np.uint32))


# The one-call layer's route sweep takes its last rows as dynamic tails
# (chunks that each block's waves claim once their own range is done) when a
# block's range is long; a grid cap makes the ranges long at sizes the oracle
# finishes quickly.  Groups of up to 8 blocks per partition, one or several
# groups, partitions of unequal size and the hard rows (dry lanes, ties,
# equal logits) of the routing tests.
DYNAMIC = [("large256", 131072, 1, 16), ("large256", 262144, 1, 40), ("large256", 196608, 5, 24),
           ("skew64", 262144, 3, 24), ("split128", 262144, 2, 34)]
CUTS = {2: [0.58], 3: [0.30, 0.71], 5: [0.13, 0.41, 0.62, 0.85]}   # unequal partitions


@pytest.mark.parametrize("name,T,P,cap", DYNAMIC, ids=[f"{d[0]}-P{d[2]}-cap{d[3]}" for d in DYNAMIC])
def test_layer_dynamic_tails(eqb, name, T, P, cap):
    w = W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    if P > 1:
        off = np.array([0] + [int(T * f) for f in CUTS[P]] + [T], np.int64)
    say(f"dynamic tails {name} T={T} E={w.E} K={w.K} P={P} grid cap {cap}")
    want = O.run_layer(z, b, w.K, off, threads=8)
    for got in run_twice(eqb, z, b, w.K, off, cap=cap):
        check(got, want, w.K)


def test_layer_scratch_contents_do_not_matter(eqb):
    """Past eqb_layer_workspace_zero_bytes the workspace is scratch for the
    fine pass's per-block count images: filled with ones before each call,
    the layer still matches the oracle and leaves its counters zero."""
    w = W.WORKLOADS["split128"].with_T(40009, 3)
    z, b, off = W.generate(w)
    want = O.run_layer(z, b, w.K, off, threads=8)
    zt = torch.from_numpy(z.view(np.int16)).cuda()
    bt = torch.from_numpy(b).cuda()
    po = eqb.PartOffsets([int(x) for x in off])
    lay = eqb.Layer(w.T, w.E, w.K, w.P)
    lay._layer_buffers()
    n = eqb.eqb_layer_workspace_zero_bytes(w.E, w.P)
    assert 0 < n < lay.workspace.numel()
    for i in range(2):
        say(f"scratch filled with ones, call {i}")
        lay.workspace[n:].fill_(0xFF)
        lay.step(zt, bt, po, sums=True)
        check(lay.step_results(), want, w.K)


@pytest.mark.parametrize("P", [1, 3])
def test_layer_long_blocks_add_fine_counts_to_slabs(eqb, P):
    """With more than 65,535 rows per block (a grid cap of 2) a block cannot
    hold its fine counts in 16-bit LDS counters to its end: the fine pass adds
    them to the partition slabs after each segment, as the separate calls
    do, and the fine selection sums the slabs."""
    w = W.WORKLOADS["skew64"].with_T(140001, P)
    z, b, off = W.generate(w)
    if P > 1:
        off = np.array([0] + [int(w.T * f) for f in CUTS[P]] + [w.T], np.int64)
    say(f"long blocks {w.T} rows, P={P}, grid cap 2")
    want = O.run_layer(z, b, w.K, off, threads=8)
    for got in run_twice(eqb, z, b, w.K, off, cap=2):
        check(got, want, w.K)


# The layer's route sweep adds its coarse counts to 16-bit slab counters where
# no slab can take more than 65,535 rows.  A grid cap of 96 gives 12 blocks per
# slab (8 slabs per partition at P = 1, 4 at P = 2) and no dynamic tails; with
# 5,461 rows per block a slab takes 65,532 rows (16-bit counters), with 5,462
# it takes 65,544 (the 32-bit form).  Every column is one value, so each
# expert's rows all land in one bin and that counter reaches its bound.
LIMIT = [(5461, 1), (5462, 1), (5461, 2), (5462, 2)]


@pytest.mark.parametrize("rpb,P", LIMIT, ids=[f"rows{c[0]}-P{c[1]}" for c in LIMIT])
def test_layer_coarse_counts_at_the_16bit_bound(eqb, rpb, P):
    T, E, K = 96 * rpb, 64, 4
    rng = np.random.default_rng(rpb + P)
    col = W._to_bf16_bits(rng.normal(0.0, 1.0, E).astype(np.float32))
    z = np.broadcast_to(col, (T, E)).copy()
    b = np.zeros(E, np.float32)
    off = None if P == 1 else np.array([0, T // 2, T], np.int64)
    say(f"one value per column, T={T} E={E} K={K} P={P}, grid cap 96")
    want = O.run_layer(z, b, K, off, threads=8)
    assert want["H"].max() == T
    for got in run_twice(eqb, z, b, K, off, cap=96):
        check(got, want, K)


@pytest.mark.parametrize("P", [1, 3])
def test_layer_runs_of_equal_rows(eqb, P):
    """A run of 1,500 equal rows puts a few blocks' rows into one fine bin of
    some experts: those blocks' images hold counts far above the others'."""
    w = W.WORKLOADS["skew64"].with_T(40000, P)
    z, b, off = W.generate(w)
    z[10000:11500] = z[10000]
    if P > 1:
        off = np.array([0] + [int(w.T * f) for f in CUTS[P]] + [w.T], np.int64)
    say(f"run of equal rows, T={w.T} P={P}")
    want = O.run_layer(z, b, w.K, off, threads=8)
    assert want["L"].max() >= 1500   # the run lands in one fine bin of some expert
    for got in run_twice(eqb, z, b, w.K, off):
        check(got, want, w.K)


# Small layers of every expert count: a single row, a few rows (fewer than
# one block step, so every block of the fine pass stores an image of almost
# nothing), K up to E - 1 (the generic route kernel past K = 14), several
# partitions.
SMALL = [(8, 1, 1, 1), (8, 7, 17, 2), (16, 3, 1, 1), (16, 9, 2, 1), (16, 15, 4099, 3),
         (32, 5, 3, 2), (32, 31, 1001, 3), (64, 1, 1, 1), (64, 14, 65, 4), (256, 255, 3, 1),
         (256, 16, 777, 2)]


@pytest.mark.parametrize("E,K,T,P", SMALL, ids=[f"E{c[0]}-K{c[1]}-T{c[2]}-P{c[3]}" for c in SMALL])
def test_layer_small_shapes(eqb, E, K, T, P):
    w = dataclasses.replace(W.WORKLOADS["skew64"], name=f"small{E}", E=E, K=K, T=T, P=P, seed=100 + E + K)
    z, b, off = W.generate(w)
    say(f"small layer E={E} K={K} T={T} P={P}")
    want = O.run_layer(z, b, K, off, threads=8)
    for got in run_twice(eqb, z, b, K, off):
        check(got, want, K)


# Seeded random layers: every expert count, K up to E - 1, batch sizes over
# five decades, unequal partitions with empty ones, grid caps, every data kind.
@pytest.mark.parametrize("i", range(24))
def test_layer_random_shapes(eqb, i):
    w, z, b, off, cap = random_layer_case(i)
    say(f"random layer {i}: T={w.T} E={w.E} K={w.K} P={w.P} kind={w.kind} cuts={off.tolist()} cap={cap}")
    want = O.run_layer(z, b, w.K, off, threads=8)
    for got in run_twice(eqb, z, b, w.K, off, cap=cap):
        check(got, want, w.K)


@pytest.mark.parametrize("P", [1, 4])
def test_layer_beyond_4gib_of_logits(eqb, P):
    """131 copies of a 65,536-token batch (E = 256): 8,585,216 tokens and
    4.4 GB of logits, so offsets into z pass 2^32 bytes (dynamic tails and
    per-block fine images at that size).  Each row's routing is its copy's,
    every count is 131 times the copy's (a partition's loads: its copies
    times the copy's), and the r-th largest key of 131 copies, r = 131 r_M, is
    the r_M-th of one copy: the quantile and the centred bias are the copy's,
    which the oracle gives on one copy.  The same for the separate calls."""
    M, n = 65536, 131
    w = W.WORKLOADS["large256"].with_T(M, 1)
    z, b, _ = W.generate(w)
    want = O.run_layer(z, b, w.K, None, threads=8)
    T, K = n * M, w.K
    copies = {1: [n], 4: [17, 43, 1, 70]}[P]
    off = np.concatenate([[0], np.cumsum(copies) * M]).astype(np.int64)
    say(f"{n} copies of {M} tokens, T={T} P={P}")
    zt = torch.from_numpy(z.view(np.int16)).cuda().repeat(n, 1)
    assert zt.numel() * 2 > 2 ** 32
    bt = torch.from_numpy(b).cuda()
    po = eqb.PartOffsets([int(x) for x in off])
    lay = eqb.Layer(T, w.E, K, P)
    want_idx = torch.from_numpy(np.ascontiguousarray(want["idx"], np.int32)).cuda()
    want_tau = torch.from_numpy(want["tau"].view(np.int32)).cuda()
    for _ in range(2):
        lay.step(zt, bt, po, sums=True)
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0 and lay.counters_zero()
        assert torch.equal(lay.topk_idx.view(n, M, K), want_idx.expand(n, M, K))
        assert torch.equal(lay.tau.view(torch.int32).view(n, M), want_tau.expand(n, M))
        score = lay.topk_score.view(n, M, K)
        assert torch.equal(score, score[:1].expand(n, M, K))
        ws = want["score"].astype(np.float64)
        assert np.all(np.abs(score[0].cpu().numpy() - ws) <= SCORE_RTOL * np.abs(ws))
        load = lay.load_out.cpu().numpy()
        np.testing.assert_array_equal(load, np.array(copies)[:, None] * want["load"][0][None, :])
        np.testing.assert_array_equal(lay.H.cpu().numpy(), n * want["H"])
        np.testing.assert_array_equal(lay.L.cpu().numpy(), n * want["L"])
        np.testing.assert_array_equal(lay.q_bf16.cpu().numpy().view(np.uint16), want["bhat"])
        np.testing.assert_array_equal(lay.b_next.cpu().numpy().view(np.uint32), want["b_next"].view(np.uint32))
    del lay
    # the separate calls on the same logits: per-partition counts are the
    # partition's copies times the copy's
    c = np.array(copies)[:, None, None]
    for fused in (True, False):
        say(f"separate calls, fused={fused}")
        sep = eqb.run_layer(zt, bt, K, [int(x) for x in off], fused=fused)
        torch.cuda.synchronize()
        assert int(sep.dev_status.item()) == 0
        assert torch.equal(sep.topk_idx.view(n, M, K), want_idx.expand(n, M, K))
        assert torch.equal(sep.tau.view(torch.int32).view(n, M), want_tau.expand(n, M))
        np.testing.assert_array_equal(sep.load.cpu().numpy(), c[:, :, 0] * want["load"][0][None, :])
        np.testing.assert_array_equal(sep.hist_hi.cpu().numpy(), c * want["H_p"][0][None])
        np.testing.assert_array_equal(sep.hist_lo.cpu().numpy(), c * want["L_p"][0][None])
        np.testing.assert_array_equal(sep.q_bf16.cpu().numpy().view(np.uint16), want["bhat"])
        np.testing.assert_array_equal(sep.b_next.cpu().numpy().view(np.uint32), want["b_next"].view(np.uint32))
        del sep
    del zt
    torch.cuda.empty_cache()
