"""GPU parity of the statistics EQB is compared with (Sec. 2): rank-averaged
QB (per-shard exact quantiles through the two passes, averaged) and the
fixed-resolution histogram estimate, through the C ABI, against the CPU
oracle, bit for bit."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import balance_oracle as B
from random_layers import random_layer_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def eqb():
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2609_28053_amd import eqb as binding
    return binding


def say(msg):
    print(f"[gpu-variants] {msg}", flush=True)
    sys.stdout.flush()


def dev(z, b):
    return torch.from_numpy(np.ascontiguousarray(z).view(np.int16)).cuda(), torch.from_numpy(b).cuda()


CASES = [("skew64", 20011, 4, None), ("large256", 9001, 16, None), ("split128", 30011, 8, None),
         ("tie64", 16411, 2, None), ("skew64", 12000, 5, [0, 3000, 3000, 7000, 7001, 12000]),
         ("skew64", 262144, 4, None)]


@pytest.mark.parametrize("name,T,P,cuts", CASES)
def test_rank_averaged_qb_matches_oracle(eqb, name, T, P, cuts):
    w = W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    if cuts is not None:
        off = np.array(cuts, np.int64)
    say(f"rank-averaged {name} T={T} P={len(off) - 1}")
    want_bp, want_avg, want_b = B.rank_averaged_qb(z, b, w.K, off)
    zt, bt = dev(z, b)
    got = eqb.rank_averaged_qb(zt, bt, w.K, [int(x) for x in off])
    assert got["dev_status"] == 0
    np.testing.assert_array_equal(got["bhat_p"], want_bp)
    np.testing.assert_array_equal(got["b_avg"].view(np.uint64), want_avg.view(np.uint64))
    np.testing.assert_array_equal(got["b_next"].view(np.uint32), want_b.view(np.uint32))


@pytest.mark.parametrize("name,T,P,lo,hi,nbins", [("skew64", 20011, 4, -8.0, 8.0, 256),
                                                  ("large256", 9001, 16, -6.0, 10.0, 37),
                                                  ("tie64", 16411, 2, -8.0, 8.0, 64),
                                                  ("split128", 30011, 8, -1.0, 1.0, 256),
                                                  ("skew64", 262144, 4, -10.0, 10.0, 200)])
def test_histogram_qb_matches_oracle(eqb, name, T, P, lo, hi, nbins):
    w = W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    say(f"histogram {name} T={T} P={P} [{lo},{hi}) nbins={nbins}")
    want_c, want_est, want_b = B.histogram_qb(z, b, w.K, off, lo, hi, nbins)
    zt, bt = dev(z, b)
    got = eqb.histogram_qb(zt, bt, w.K, lo, hi, nbins, [int(x) for x in off])
    assert got["dev_status"] == 0
    np.testing.assert_array_equal(got["counts"], want_c)
    np.testing.assert_array_equal(got["est"].view(np.uint64), want_est.view(np.uint64))
    np.testing.assert_array_equal(got["b_next"].view(np.uint32), want_b.view(np.uint32))


# The seeded random layers of the layer tests (every expert count, K up to
# E - 1, unequal partitions with empty ones, grid caps, every data kind), with
# a random histogram range and bin count for the fixed-resolution estimate.
@pytest.mark.parametrize("i", range(16))
def test_variants_on_random_shapes(eqb, i):
    w, z, b, off, cap = random_layer_case(i)
    rng = np.random.default_rng(9000 + i)
    lo = float(np.float32(rng.uniform(-10.0, 0.0)))
    hi = float(np.float32(lo + rng.uniform(0.5, 16.0)))
    nbins = int(rng.integers(1, 257))
    say(f"variants random {i}: T={w.T} E={w.E} K={w.K} cuts={off.tolist()} cap={cap} "
        f"[{lo},{hi}) nbins={nbins}")
    want_bp, want_avg, want_b = B.rank_averaged_qb(z, b, w.K, off)
    want_c, want_est, want_hb = B.histogram_qb(z, b, w.K, off, lo, hi, nbins)
    zt, bt = dev(z, b)
    offl = [int(x) for x in off]
    try:
        eqb.eqb_set_max_blocks(cap)
        got = eqb.rank_averaged_qb(zt, bt, w.K, offl)
        hist = eqb.histogram_qb(zt, bt, w.K, lo, hi, nbins, offl)
    finally:
        eqb.eqb_set_max_blocks(0)
    assert got["dev_status"] == 0 and hist["dev_status"] == 0
    np.testing.assert_array_equal(got["bhat_p"], want_bp)
    np.testing.assert_array_equal(got["b_avg"].view(np.uint64), want_avg.view(np.uint64))
    np.testing.assert_array_equal(got["b_next"].view(np.uint32), want_b.view(np.uint32))
    np.testing.assert_array_equal(hist["counts"], want_c)
    np.testing.assert_array_equal(hist["est"].view(np.uint64), want_est.view(np.uint64))
    np.testing.assert_array_equal(hist["b_next"].view(np.uint32), want_hb.view(np.uint32))
