"""The C ABI without a GPU: the library loads, exports every declared entry
point, and rejects bad arguments before it touches the HIP runtime."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eqb.h")
LIB = os.environ.get("EQB_LIB", os.path.join(ROOT, "paper_2609_28053_amd", "libeqb.so"))

OK, INVALID, UNSUPPORTED, RANK = 0, 1, 2, 3


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eqb_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libeqb.so is not built (run paper_2609_28053_amd/build.py)")
    lib = ctypes.CDLL(LIB)
    V, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.eqb_route_topk.argtypes = [V, V, i64, i32, i32, V, V, V, V, i32, V, V, V]
    lib.eqb_margin_hist_pass1.argtypes = [V, V, i64, i32, V, i32, V, V]
    lib.eqb_margin_hist_pass2.argtypes = [V, V, i64, i32, V, V, i32, V, V]
    lib.eqb_select_quantile.argtypes = [i32, V, i32, i32, i64, V, V, V, V, V, V, V, V]
    lib.eqb_expert_load.argtypes = [V, i64, i32, i32, V, i32, V, V]
    lib.eqb_max_violation.argtypes = [V, i64, i32, i32, V, i32, V, V, V, V]
    lib.eqb_lei_residual.argtypes = [V, i64, i32, i32, V, i32, ctypes.c_double, ctypes.c_double, V, V]
    lib.eqb_lei_inject.argtypes = [V, V, i64, i32, V, i32, V]
    lib.eqb_lei_router_backward.argtypes = [V, V, V, V, i64, i32, i32, V, i32, V, V]
    lib.eqb_layer_workspace_size.argtypes = [i32, i32]
    lib.eqb_layer_workspace_size.restype = ctypes.c_size_t
    lib.eqb_layer_workspace_zero_bytes.argtypes = [i32, i32]
    lib.eqb_layer_workspace_zero_bytes.restype = ctypes.c_size_t
    lib.eqb_layer.argtypes = [V, V, i64, i32, i32, V, i32] + [V] * 10 + [ctypes.c_size_t, V, V]
    lib.eqb_set_max_blocks.argtypes = [i32]
    lib.eqb_get_max_blocks.argtypes = []
    lib.eqb_rank.argtypes = [i64, i32, i32]
    lib.eqb_rank.restype = i64
    lib.eqb_status_string.argtypes = [i32]
    lib.eqb_status_string.restype = ctypes.c_char_p
    return lib


def test_header_declares_the_five_calls():
    names = declared_functions()
    for n in ("eqb_route_topk", "eqb_margin_hist_pass1", "eqb_margin_hist_pass2",
              "eqb_select_quantile", "eqb_expert_load"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_exports_match_header():
    src = open(os.path.join(ROOT, "paper_2609_28053_amd", "eqb.py")).read()
    for name in declared_functions():
        assert f'"{name}"' in src


FAKE = ctypes.c_void_p(0x10000)     # never dereferenced: every call below fails its checks first


def offs(*v):
    arr = (ctypes.c_int64 * len(v))(*v)
    return ctypes.cast(arr, ctypes.c_void_p), arr


def route(lib, T=64, E=8, K=2, z=FAKE, po=None, P=1):
    return lib.eqb_route_topk(z, FAKE, T, E, K, FAKE, FAKE, FAKE, po, P, None, None, None)


def test_route_argument_checks(lib):
    assert route(lib, K=0) == INVALID
    assert route(lib, K=8) == INVALID            # K >= E
    assert route(lib, T=-1) == INVALID
    assert route(lib, E=12, K=2) == UNSUPPORTED
    assert route(lib, E=512, K=2) == UNSUPPORTED
    assert route(lib, z=ctypes.c_void_p(0x10002)) == UNSUPPORTED   # z not 16-byte aligned
    assert lib.eqb_route_topk(None, FAKE, 64, 8, 2, FAKE, FAKE, FAKE, None, 1, None, None, None) == INVALID
    assert lib.eqb_route_topk(FAKE, FAKE, 64, 8, 2, None, FAKE, FAKE, None, 1, None, None, None) == INVALID
    assert route(lib, T=0) == OK                 # empty batch: nothing to do
    assert lib.eqb_route_topk(None, None, 0, 8, 2, None, None, None, None, 1, None, None, None) == OK


def test_partition_table_checks(lib):
    po, keep = offs(0, 10, 5, 64)                 # decreasing
    assert route(lib, po=po, P=3) == INVALID
    po, keep = offs(0, 10, 63)                    # does not end at T
    assert route(lib, po=po, P=2) == INVALID
    po, keep = offs(1, 10, 64)                    # does not start at 0
    assert route(lib, po=po, P=2) == INVALID
    assert route(lib, po=None, P=2) == INVALID    # NULL table means exactly one partition
    po, keep = offs(0, 64)
    assert route(lib, po=po, P=0) == INVALID
    big = [0] * 258
    big[-1] = 64
    po, keep = offs(*big)
    assert route(lib, po=po, P=257) == INVALID    # beyond EQB_MAX_PARTITIONS
    po, keep = offs(0, 0, 0)
    assert route(lib, T=0, po=po, P=2) == OK      # all partitions empty


def test_pass_and_load_checks(lib):
    f = lib.eqb_margin_hist_pass1
    assert f(FAKE, FAKE, 10, 12, None, 1, FAKE, None) == UNSUPPORTED
    assert f(FAKE, None, 10, 8, None, 1, FAKE, None) == INVALID
    assert f(FAKE, FAKE, 10, 8, None, 1, None, None) == INVALID
    assert f(FAKE, FAKE, 0, 8, None, 1, FAKE, None) == OK
    g = lib.eqb_margin_hist_pass2
    assert g(FAKE, FAKE, 10, 8, None, None, 1, FAKE, None) == INVALID     # no sel_hi
    assert g(ctypes.c_void_p(0x10008), FAKE, 10, 8, FAKE, None, 1, FAKE, None) == UNSUPPORTED
    h = lib.eqb_expert_load
    assert h(FAKE, 10, 0, 8, None, 1, FAKE, None) == INVALID
    assert h(FAKE, 10, 2, 8, None, 1, None, None) == INVALID
    assert h(FAKE, 10, 2, 7, None, 1, FAKE, None) == UNSUPPORTED


def test_select_checks(lib):
    s = lib.eqb_select_quantile
    assert s(3, FAKE, 1, 8, 10, FAKE, FAKE, None, None, None, None, None, None) == INVALID
    assert s(1, FAKE, 0, 8, 10, FAKE, FAKE, None, None, None, None, None, None) == INVALID
    assert s(1, FAKE, 1, 9, 10, FAKE, FAKE, None, None, None, None, None, None) == UNSUPPORTED
    assert s(1, FAKE, 1, 8, 0, FAKE, FAKE, None, None, None, None, None, None) == RANK
    assert s(1, None, 1, 8, 5, FAKE, FAKE, None, None, None, None, None, None) == INVALID
    assert s(2, FAKE, 1, 8, 5, FAKE, FAKE, None, FAKE, None, None, None, None) == INVALID  # no sel_lo


def test_max_violation_checks(lib):
    m = lib.eqb_max_violation
    assert m(FAKE, 64, 0, 8, None, 1, FAKE, None, None, None) == INVALID        # K < 1
    assert m(FAKE, 64, 8, 8, None, 1, FAKE, None, None, None) == INVALID        # K >= E
    assert m(FAKE, 64, 2, 12, None, 1, FAKE, None, None, None) == UNSUPPORTED
    assert m(None, 64, 2, 8, None, 1, FAKE, None, None, None) == INVALID
    assert m(FAKE, 64, 2, 8, None, 1, None, None, None, None) == INVALID        # no global output
    po, keep = offs(0, 10, 5, 64)
    assert m(FAKE, 64, 2, 8, po, 3, FAKE, FAKE, None, None) == INVALID          # decreasing offsets
    assert m(FAKE, 0, 2, 8, None, 1, FAKE, None, None, None) == OK              # empty batch


def test_lei_checks(lib):
    r = lib.eqb_lei_residual
    assert r(FAKE, 64, 2, 8, None, 1, 1e-5, 2.0, None, None) == INVALID     # no output
    assert r(None, 64, 2, 8, None, 1, 1e-5, 2.0, FAKE, None) == INVALID
    assert r(FAKE, 64, 8, 8, None, 1, 1e-5, 2.0, FAKE, None) == INVALID     # K >= E
    assert r(FAKE, 64, 2, 24, None, 1, 1e-5, 2.0, FAKE, None) == UNSUPPORTED
    assert r(FAKE, 64, 2, 8, None, 1, float("nan"), 2.0, FAKE, None) == INVALID
    assert r(FAKE, 64, 2, 8, None, 1, 1e-5, float("nan"), FAKE, None) == INVALID
    i = lib.eqb_lei_inject
    assert i(None, FAKE, 64, 8, None, 1, None) == INVALID
    assert i(FAKE, None, 64, 8, None, 1, None) == INVALID
    assert i(ctypes.c_void_p(0x10004), FAKE, 64, 8, None, 1, None) == UNSUPPORTED   # misaligned
    assert i(FAKE, FAKE, 64, 12, None, 1, None) == UNSUPPORTED
    po, keep = offs(0, 10, 63)
    assert i(FAKE, FAKE, 64, 8, po, 2, None) == INVALID
    assert i(FAKE, FAKE, 0, 8, None, 1, None) == OK


def test_router_backward_checks(lib):
    f = lib.eqb_lei_router_backward
    assert f(None, FAKE, FAKE, None, 64, 8, 2, None, 1, FAKE, None) == INVALID
    assert f(FAKE, FAKE, FAKE, None, 64, 8, 2, None, 1, None, None) == INVALID
    assert f(FAKE, FAKE, FAKE, None, 64, 8, 8, None, 1, FAKE, None) == INVALID      # K >= E
    assert f(FAKE, FAKE, FAKE, None, 64, 24, 2, None, 1, FAKE, None) == UNSUPPORTED
    assert f(ctypes.c_void_p(0x10002), FAKE, FAKE, None, 64, 8, 2, None, 1, FAKE, None) == UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, None, 64, 8, 2, None, 1, ctypes.c_void_p(0x10004), None) == UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, None, 0, 8, 2, None, 1, FAKE, None) == OK


def test_set_max_blocks(lib):
    assert lib.eqb_set_max_blocks(-1) == INVALID
    assert lib.eqb_set_max_blocks(3) == OK
    assert lib.eqb_set_max_blocks(0) == OK


def test_rank_and_status_strings(lib):
    assert lib.eqb_rank(4096, 2, 8) == 1024
    assert lib.eqb_rank(4194304, 8, 256) == 131072
    assert lib.eqb_rank(10, 3, 8) == 4
    assert lib.eqb_rank(10, 8, 8) == -1
    assert lib.eqb_rank(-1, 2, 8) == -1
    assert lib.eqb_status_string(0) == b"EQB_OK"
    assert lib.eqb_status_string(3) == b"EQB_ERR_RANK"
    assert lib.eqb_status_string(99) == b"EQB_ERR_UNKNOWN"


def layer(lib, T=64, E=8, K=2, ws=ctypes.c_void_p(0x10000), ws_bytes=1 << 30, po=None, P=1, z=FAKE):
    return lib.eqb_layer(z, FAKE, T, E, K, po, P, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE,
                         ws, ws_bytes, None, None)


def test_layer_workspace_size(lib):
    # Counters: two sets of [P,nsub,E,256] int32 count slabs (nsub = 8 // P
    # slabs per partition below 8 partitions, else 1), the [P,E] loads and
    # three [E] selections, each rounded up to 256 bytes, and 1,024 claim
    # counters of the route sweep's dynamic tails, 128 bytes apart.  Then the
    # fine pass's per-block images, E/2 * 256 words each, for one block per
    # compute unit on 256 compute units.
    for E, P in ((8, 1), (64, 4), (128, 3), (256, 1), (256, 16), (256, 17), (256, 256)):
        nsub = 1 if P >= 8 else 8 // P
        zero = (2 * P * nsub * E * 1024 + -(-4 * P * E // 256) * 256 + 2 * -(-4 * E // 256) * 256
                + -(-8 * E // 256) * 256 + 1024 * 128)
        assert lib.eqb_layer_workspace_zero_bytes(E, P) == zero
        assert lib.eqb_layer_workspace_size(E, P) == zero + 256 * (E // 2) * 256 * 4
    assert lib.eqb_layer_workspace_size(256, 1) - lib.eqb_layer_workspace_zero_bytes(256, 1) == 32 << 20
    for E, P in ((12, 1), (8, 0), (8, 257)):
        assert lib.eqb_layer_workspace_size(E, P) == 0
        assert lib.eqb_layer_workspace_zero_bytes(E, P) == 0


def test_layer_argument_checks(lib):
    assert layer(lib, T=0) == RANK                                 # no margins, no quantile
    assert layer(lib, K=8) == INVALID
    assert layer(lib, E=12) == UNSUPPORTED
    assert layer(lib, ws=None) == INVALID
    assert layer(lib, ws=ctypes.c_void_p(0x10010)) == UNSUPPORTED   # not 256-byte aligned
    assert layer(lib, ws_bytes=lib.eqb_layer_workspace_size(8, 1) - 1) == INVALID
    assert layer(lib, z=ctypes.c_void_p(0x10002)) == UNSUPPORTED
    po, keep = offs(0, 10, 64)
    assert layer(lib, po=po, P=2, ws_bytes=lib.eqb_layer_workspace_size(8, 2) - 1) == INVALID   # one byte short
    bad, keep2 = offs(0, 70, 64)
    assert layer(lib, po=bad, P=2) == INVALID


def test_grid_cap_is_per_thread(lib):
    """A cap set on one host thread leaves other threads' grids alone."""
    import threading
    assert lib.eqb_set_max_blocks(3) == OK
    seen = {}

    def other():
        seen["before"] = lib.eqb_get_max_blocks()
        lib.eqb_set_max_blocks(7)
        seen["after"] = lib.eqb_get_max_blocks()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    try:
        assert seen == {"before": 0, "after": 7}
        assert lib.eqb_get_max_blocks() == 3
    finally:
        assert lib.eqb_set_max_blocks(0) == OK
    assert lib.eqb_set_max_blocks(-1) == INVALID



def test_noalloc_layer_rejects_before_any_hip_call(lib):
    """The scratch limit and the argument checks come before the library
    touches the runtime (this container has no GPU)."""
    f = lib.eqb_layer_noalloc
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_void_p, ctypes.c_int32] + [ctypes.c_void_p] * 10
    SCRATCH = 5
    po, keep = offs(*range(0, 18 * 64, 64)[:18])           # 17 partitions
    assert f(FAKE, FAKE, 17 * 64 - 64, 256, 8, po, 17, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE,
             None) == SCRATCH                               # 17 * 256 > 4096
    assert lib.eqb_status_string(SCRATCH) == b"EQB_ERR_SCRATCH"
    assert f(FAKE, FAKE, 64, 8, 8, None, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE, None) == INVALID
    assert f(FAKE, FAKE, 64, 12, 2, None, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE, None) == UNSUPPORTED
    assert f(FAKE, FAKE, 0, 8, 2, None, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE, None) == RANK
    assert f(FAKE, FAKE, 64, 8, 2, None, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None) == INVALID
