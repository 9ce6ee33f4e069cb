"""GPU parity of the balance quantities: MaxVio and the closed QB loop,
through the C ABI, against the CPU oracle (bit for bit)."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import balance_oracle as B

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def eqb():
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2609_28053_amd import eqb as binding
    return binding


def say(msg):
    print(f"[gpu-balance] {msg}", flush=True)
    sys.stdout.flush()


def same_f64(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.array_equal(a.view(np.uint64), b.view(np.uint64))


@pytest.mark.parametrize("E,P", [(8, 1), (64, 5), (256, 16), (256, 256)])
def test_max_violation_matches_oracle(eqb, E, P):
    rng = np.random.default_rng(E * 1000 + P)
    K = max(1, E // 32)
    sizes = rng.integers(0, 5000, size=P)
    sizes[rng.integers(0, P)] = 0 if P > 1 else sizes[0]      # an empty partition when P > 1
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    T = int(off[-1])
    weights = rng.dirichlet(np.ones(E) * 0.5)
    load = np.stack([rng.multinomial(int(K * n), weights) for n in sizes]).astype(np.int32)
    say(f"maxvio E={E} P={P} T={T}")
    lt = torch.from_numpy(load).cuda()
    g = torch.empty(1, dtype=torch.float64, device="cuda")
    l = torch.empty(P, dtype=torch.float64, device="cuda")
    eqb.eqb_max_violation(lt, T, K, g, l, [int(x) for x in off])
    torch.cuda.synchronize()
    want_g, want_l = B.max_violation(load, off, K)
    assert same_f64(g.cpu().numpy(), [want_g])
    assert same_f64(l.cpu().numpy(), want_l)


def check_loop(got, want):
    assert len(got) == len(want)
    for q, (a, b) in enumerate(zip(got, want)):
        assert a["dev_status"] == 0
        np.testing.assert_array_equal(a["b"].view(np.uint32), b["b"].view(np.uint32), err_msg=f"step {q}")
        np.testing.assert_array_equal(a["load"], b["load"], err_msg=f"step {q}")
        assert same_f64([a["maxvio_global"]], [b["maxvio_global"]]), q
        assert same_f64(a["maxvio_local"], b["maxvio_local"]), q
        np.testing.assert_array_equal(a["bhat"], b["bhat"], err_msg=f"step {q}")
        np.testing.assert_array_equal(a["b_next"].view(np.uint32), b["b_next"].view(np.uint32))


@pytest.mark.parametrize("name,T,P,steps", [("skew64", 20011, 4, 3), ("large256", 9001, 16, 2),
                                            ("skew64", 262144, 4, 3)])
def test_qb_loop_matches_oracle(eqb, name, T, P, steps):
    w = W.CONFIGS[name].with_T(T, P)
    _, b0, off = W.generate(w)
    batches = [W.generate(w, batch=q)[0] for q in range(steps)]
    say(f"qb loop {name} T={T} P={P} steps={steps}")
    want = B.qb_loop(batches, b0, w.K, off, threads=8)
    zs = [torch.from_numpy(z.view(np.int16)).cuda() for z in batches]
    got = eqb.qb_loop(zs, torch.from_numpy(b0), w.K, [int(x) for x in off])
    check_loop(got, want)
