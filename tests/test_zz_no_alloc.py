"""eqb_layer_noalloc (the layer for callers that cannot allocate) against
eqb_layer with a caller workspace: the same outputs bit for bit, on calls in
a row that share the library's scratch array, the second one smaller than
the first, and a clear error for a layer that needs more scratch."""
import sys

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def eqb():
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2609_28053_amd import eqb as binding
    return binding


def say(msg):
    print(f"[gpu-noalloc] {msg}", flush=True)
    sys.stdout.flush()


def outputs(eqb, T, E, K, P, dev):
    i32 = dict(dtype=torch.int32, device=dev)
    return dict(idx=torch.empty((T, K), **i32), score=torch.empty((T, K), dtype=torch.float32, device=dev),
                tau=torch.empty(T, dtype=torch.float32, device=dev), load=torch.empty((P, E), **i32),
                q=torch.empty(E, dtype=torch.int16, device=dev), b_next=torch.empty(E, dtype=torch.float32, device=dev),
                H=torch.empty((E, 256), **i32), L=torch.empty((E, 256), **i32), status=torch.full((1,), -7, **i32))


def host(o):
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in o.items()}


def run_both(eqb, name, T, P):
    w = W.WORKLOADS[name].with_T(T, P)
    z, b, off = W.generate(w)
    dev = torch.device("cuda:0")
    zt = torch.from_numpy(z.view(np.int16)).to(dev)
    bt = torch.from_numpy(b).to(dev)
    po = eqb.PartOffsets([int(x) for x in off])
    ref = outputs(eqb, w.T, w.E, w.K, w.P, dev)
    ws = torch.zeros(eqb.eqb_layer_workspace_size(w.E, w.P), dtype=torch.uint8, device=dev)
    eqb.eqb_layer(zt, bt, w.K, ref["idx"], ref["score"], ref["tau"], ref["load"], ref["q"], ref["b_next"],
                  ref["status"], ws, po, ref["H"], ref["L"])
    got = outputs(eqb, w.T, w.E, w.K, w.P, dev)
    say(f"noalloc {name} T={w.T} E={w.E} K={w.K} P={w.P}")
    eqb.eqb_layer_noalloc(zt, bt, w.K, got["idx"], got["score"], got["tau"], got["load"], got["q"], got["b_next"],
                          got["status"], po, got["H"], got["L"])
    return host(ref), host(got)


def test_noalloc_layer_matches_the_workspace_layer(eqb):
    # two calls in a row on the shared scratch: a large layer, then a smaller
    # one (fewer partitions and experts), then the large one again
    for name, T, P in (("large256", 30011, 16), ("skew64", 7001, 4), ("large256", 20011, 16)):
        ref, got = run_both(eqb, name, T, P)
        assert int(ref["status"][0]) == 0 and int(got["status"][0]) == 0
        for k in ref:
            np.testing.assert_array_equal(got[k].view(np.uint8), ref[k].view(np.uint8), err_msg=f"{name} {k}")


def test_noalloc_layer_with_dynamic_tails(eqb):
    # a grid of 16 blocks makes each block's range long enough for the route
    # sweep's dynamic tails (claim counters in the scratch array, which the
    # coarse selection resets); one partition, so 16 count slabs per
    # partition; then a smaller layer and the first one again
    try:
        eqb.eqb_set_max_blocks(16)
        for name, T, P in (("large256", 131072, 1), ("skew64", 7001, 4), ("large256", 131072, 1)):
            ref, got = run_both(eqb, name, T, P)
            assert int(ref["status"][0]) == 0 and int(got["status"][0]) == 0
            for k in ref:
                np.testing.assert_array_equal(got[k].view(np.uint8), ref[k].view(np.uint8), err_msg=f"{name} {k}")
    finally:
        eqb.eqb_set_max_blocks(0)


def test_noalloc_layer_rejects_a_layer_beyond_its_scratch(eqb):
    w = W.WORKLOADS["large256"].with_T(4096, 17)        # P * E = 4352 > 4096
    z, b, off = W.generate(w)
    dev = torch.device("cuda:0")
    zt = torch.from_numpy(z.view(np.int16)).to(dev)
    bt = torch.from_numpy(b).to(dev)
    o = outputs(eqb, w.T, w.E, w.K, w.P, dev)
    assert eqb.eqb_layer_workspace_zero_bytes(w.E, w.P) > eqb.EQB_NOALLOC_SCRATCH_BYTES
    with pytest.raises(eqb.EqbError) as ex:
        eqb.eqb_layer_noalloc(zt, bt, w.K, o["idx"], o["score"], o["tau"], o["load"], o["q"], o["b_next"],
                              o["status"], [int(x) for x in off])
    assert ex.value.status == eqb.EQB_ERR_SCRATCH
    torch.cuda.synchronize()
    assert int(o["status"].item()) == -7                  # nothing was enqueued
