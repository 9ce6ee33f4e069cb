"""ctypes binding of libeqb.so: argument marshalling only.

Every function takes torch tensors that live on the GPU (except ``part_off``,
a host sequence of P+1 token offsets) and passes their device pointers and the
current HIP stream to the C ABI of the same name.  All computation happens in
the library's kernels; torch only provides device memory and streams.  A
missing or unloadable library raises ImportError: there is no fallback.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("EQB_LIB", os.path.join(_HERE, "libeqb.so"))

EQB_OK = 0
EQB_ERR_INVALID_ARG = 1
EQB_ERR_UNSUPPORTED = 2
EQB_ERR_RANK = 3
EQB_ERR_HIP = 4
EQB_ERR_SCRATCH = 5
EQB_NOALLOC_SCRATCH_BYTES = (8 << 20) + (192 << 10)
EQB_NBINS = 256
EQB_MAX_PARTITIONS = 256
EQB_DEV_RANK_EXCEEDS_COUNT = 1

EXPORTS = (
    "eqb_route_topk",
    "eqb_margin_hist_pass1",
    "eqb_select_quantile",
    "eqb_margin_hist_pass2",
    "eqb_expert_load",
    "eqb_select_quantile_local",
    "eqb_margin_hist_pass2_local",
    "eqb_rank_average",
    "eqb_margin_hist_uniform",
    "eqb_select_uniform",
    "eqb_max_violation",
    "eqb_lei_residual",
    "eqb_lei_inject",
    "eqb_lei_router_backward",
    "eqb_layer_workspace_size",
    "eqb_layer_workspace_zero_bytes",
    "eqb_layer",
    "eqb_layer_noalloc",
    "eqb_set_max_blocks",
    "eqb_get_max_blocks",
    "eqb_rank",
    "eqb_status_string",
)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libeqb.so not built at {LIB_PATH}; run paper_2609_28053_amd/build.py")
    try:
        lib = ctypes.CDLL(LIB_PATH)
    except OSError as exc:  # pragma: no cover - depends on the ROCm install
        raise ImportError(f"cannot load {LIB_PATH}: {exc}") from exc
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    sig = {
        "eqb_route_topk": [P, P, i64, i32, i32, P, P, P, P, i32, P, P, P],
        "eqb_margin_hist_pass1": [P, P, i64, i32, P, i32, P, P],
        "eqb_select_quantile": [i32, P, i32, i32, i64, P, P, P, P, P, P, P, P],
        "eqb_margin_hist_pass2": [P, P, i64, i32, P, P, i32, P, P],
        "eqb_expert_load": [P, i64, i32, i32, P, i32, P, P],
        "eqb_select_quantile_local": [i32, P, i64, i32, i32, P, i32, P, P, P, P, P, P],
        "eqb_margin_hist_pass2_local": [P, P, i64, i32, P, P, i32, P, P],
        "eqb_rank_average": [P, i64, i32, P, i32, P, P, P],
        "eqb_margin_hist_uniform": [P, P, i64, i32, P, i32, ctypes.c_float, ctypes.c_float, i32, P, P],
        "eqb_select_uniform": [P, i32, i32, i32, i64, ctypes.c_float, ctypes.c_float, P, P, P, P],
        "eqb_max_violation": [P, i64, i32, i32, P, i32, P, P, P, P],
        "eqb_lei_residual": [P, i64, i32, i32, P, i32, ctypes.c_double, ctypes.c_double, P, P],
        "eqb_lei_inject": [P, P, i64, i32, P, i32, P],
        "eqb_lei_router_backward": [P, P, P, P, i64, i32, i32, P, i32, P, P],
        "eqb_layer_workspace_size": [i32, i32],
        "eqb_layer_workspace_zero_bytes": [i32, i32],
        "eqb_layer": [P, P, i64, i32, i32, P, i32, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P, P],
        "eqb_layer_noalloc": [P, P, i64, i32, i32, P, i32, P, P, P, P, P, P, P, P, P, P],
        "eqb_set_max_blocks": [i32],
        "eqb_get_max_blocks": [],
        "eqb_rank": [i64, i32, i32],
        "eqb_status_string": [i32],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = i32
    lib.eqb_rank.restype = i64
    lib.eqb_layer_workspace_size.restype = ctypes.c_size_t
    lib.eqb_layer_workspace_zero_bytes.restype = ctypes.c_size_t
    lib.eqb_status_string.restype = ctypes.c_char_p
    return lib


lib = _load()


class EqbError(RuntimeError):
    def __init__(self, name: str, status: int):
        self.status = status
        super().__init__(f"{name} returned {lib.eqb_status_string(status).decode()} ({status})")


def _check(name: str, status: int) -> None:
    if status != EQB_OK:
        raise EqbError(name, status)


def _ptr(t: Optional[torch.Tensor], dtype=None, numel=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class PartOffsets:
    """A partition table converted once for repeated calls: P+1 token
    offsets held as an int64 array with its pointer ready for the C ABI."""

    __slots__ = ("arr", "ptr", "P")

    def __init__(self, part_off: Sequence[int]):
        self.arr = np.ascontiguousarray(np.asarray(part_off, dtype=np.int64))
        self.ptr = self.arr.ctypes.data_as(ctypes.c_void_p)
        self.P = self.arr.size - 1


def _offsets(part_off, T: int):
    if part_off is None:
        return None, 1, None
    if isinstance(part_off, PartOffsets):
        return part_off.ptr, part_off.P, part_off
    arr = np.ascontiguousarray(np.asarray(part_off, dtype=np.int64))
    P = arr.size - 1
    return arr.ctypes.data_as(ctypes.c_void_p), P, arr     # keep arr alive


_Z = (torch.int16, torch.uint16) if hasattr(torch, "uint16") else (torch.int16,)


def eqb_route_topk(z, b, K, topk_idx, topk_score, tau, part_off=None, load=None, hist_hi=None,
                   stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_route_topk", lib.eqb_route_topk(
        _ptr(z, _Z, name="z"), _ptr(b, torch.float32, E, "b"), T, E, K,
        _ptr(topk_idx, torch.int32, T * K, "topk_idx"), _ptr(topk_score, torch.float32, T * K, "topk_score"),
        _ptr(tau, torch.float32, T, "tau"), po, P,
        _ptr(load, torch.int32, P * E, "load"), _ptr(hist_hi, torch.int32, P * E * EQB_NBINS, "hist_hi"),
        _stream(stream)))
    del keep


def eqb_margin_hist_pass1(z, tau, hist_hi, part_off=None, stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_margin_hist_pass1", lib.eqb_margin_hist_pass1(
        _ptr(z, _Z, name="z"), _ptr(tau, torch.float32, T, "tau"), T, E, po, P,
        _ptr(hist_hi, torch.int32, P * E * EQB_NBINS, "hist_hi"), _stream(stream)))
    del keep


def eqb_select_quantile(pass_, hist, r, sel_hi, rank_in_bin, sel_lo=None, q_bf16=None, b_next=None,
                        hist_sum=None, dev_status=None, stream=None):
    P, E, nb = hist.shape
    assert nb == EQB_NBINS
    _check("eqb_select_quantile", lib.eqb_select_quantile(
        pass_, _ptr(hist, torch.int32, name="hist"), P, E, r,
        _ptr(sel_hi, torch.int32, E, "sel_hi"), _ptr(rank_in_bin, torch.int64, E, "rank_in_bin"),
        _ptr(sel_lo, torch.int32, E, "sel_lo"), _ptr(q_bf16, _Z, E, "q_bf16"),
        _ptr(b_next, torch.float32, E, "b_next"), _ptr(hist_sum, torch.int32, E * EQB_NBINS, "hist_sum"),
        _ptr(dev_status, torch.int32, 1, "dev_status"), _stream(stream)))


def eqb_margin_hist_pass2(z, tau, sel_hi, hist_lo, part_off=None, stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_margin_hist_pass2", lib.eqb_margin_hist_pass2(
        _ptr(z, _Z, name="z"), _ptr(tau, torch.float32, T, "tau"), T, E,
        _ptr(sel_hi, torch.int32, E, "sel_hi"), po, P,
        _ptr(hist_lo, torch.int32, P * E * EQB_NBINS, "hist_lo"), _stream(stream)))
    del keep


def eqb_expert_load(topk_idx, E, load, part_off=None, stream=None):
    T, K = topk_idx.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_expert_load", lib.eqb_expert_load(
        _ptr(topk_idx, torch.int32, T * K, "topk_idx"), T, K, E, po, P,
        _ptr(load, torch.int32, P * E, "load"), _stream(stream)))
    del keep


def eqb_select_quantile_local(pass_, hist, T, K, sel_hi, rank_in_bin, sel_lo=None, q_bf16=None,
                              part_off=None, dev_status=None, stream=None):
    P, E, nb = hist.shape
    assert nb == EQB_NBINS
    po, Pn, keep = _offsets(part_off, T)
    if Pn != P:
        raise ValueError(f"hist has {P} partitions, part_off describes {Pn}")
    _check("eqb_select_quantile_local", lib.eqb_select_quantile_local(
        pass_, _ptr(hist, torch.int32, name="hist"), T, K, E, po, P,
        _ptr(sel_hi, torch.int32, P * E, "sel_hi"), _ptr(rank_in_bin, torch.int64, P * E, "rank_in_bin"),
        _ptr(sel_lo, torch.int32, P * E, "sel_lo"), _ptr(q_bf16, _Z, P * E, "q_bf16"),
        _ptr(dev_status, torch.int32, 1, "dev_status"), _stream(stream)))
    del keep


def eqb_margin_hist_pass2_local(z, tau, sel_hi, hist_lo, part_off=None, stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_margin_hist_pass2_local", lib.eqb_margin_hist_pass2_local(
        _ptr(z, _Z, name="z"), _ptr(tau, torch.float32, T, "tau"), T, E,
        _ptr(sel_hi, torch.int32, P * E, "sel_hi"), po, P,
        _ptr(hist_lo, torch.int32, P * E * EQB_NBINS, "hist_lo"), _stream(stream)))
    del keep


def eqb_rank_average(q_bf16, T, b_next, b_avg=None, part_off=None, stream=None):
    P, E = q_bf16.shape
    po, Pn, keep = _offsets(part_off, T)
    if Pn != P:
        raise ValueError(f"q_bf16 has {P} partitions, part_off describes {Pn}")
    _check("eqb_rank_average", lib.eqb_rank_average(
        _ptr(q_bf16, _Z, P * E, "q_bf16"), T, E, po, P, _ptr(b_avg, torch.float64, E, "b_avg"),
        _ptr(b_next, torch.float32, E, "b_next"), _stream(stream)))
    del keep


def eqb_margin_hist_uniform(z, tau, lo, hi, hist, part_off=None, stream=None):
    T, E = z.shape
    P, E2, nbins = hist.shape
    po, Pn, keep = _offsets(part_off, T)
    if Pn != P or E2 != E:
        raise ValueError("hist must be [P, E, nbins]")
    _check("eqb_margin_hist_uniform", lib.eqb_margin_hist_uniform(
        _ptr(z, _Z, name="z"), _ptr(tau, torch.float32, T, "tau"), T, E, po, P, float(lo), float(hi), nbins,
        _ptr(hist, torch.int32, P * E * nbins, "hist"), _stream(stream)))
    del keep


def eqb_select_uniform(hist, r, lo, hi, est, b_next=None, dev_status=None, stream=None):
    P, E, nbins = hist.shape
    _check("eqb_select_uniform", lib.eqb_select_uniform(
        _ptr(hist, torch.int32, name="hist"), P, E, nbins, r, float(lo), float(hi),
        _ptr(est, torch.float64, E, "est"), _ptr(b_next, torch.float32, E, "b_next"),
        _ptr(dev_status, torch.int32, 1, "dev_status"), _stream(stream)))


def eqb_max_violation(load, T, K, maxvio_global, maxvio_local=None, part_off=None, maxvio_local_mean=None,
                      stream=None):
    P, E = load.shape
    po, Pn, keep = _offsets(part_off, T)
    if Pn != P:
        raise ValueError(f"load has {P} partitions, part_off describes {Pn}")
    _check("eqb_max_violation", lib.eqb_max_violation(
        _ptr(load, torch.int32, P * E, "load"), T, K, E, po, P,
        _ptr(maxvio_global, torch.float64, 1, "maxvio_global"),
        _ptr(maxvio_local, torch.float64, P, "maxvio_local"),
        _ptr(maxvio_local_mean, torch.float64, 1, "maxvio_local_mean"), _stream(stream)))
    del keep


def eqb_lei_residual(load, T, K, eta, c, inj, part_off=None, stream=None):
    P, E = load.shape
    po, Pn, keep = _offsets(part_off, T)
    if Pn != P:
        raise ValueError(f"load has {P} partitions, part_off describes {Pn}")
    _check("eqb_lei_residual", lib.eqb_lei_residual(
        _ptr(load, torch.int32, P * E, "load"), T, K, E, po, P, float(eta), float(c),
        _ptr(inj, torch.float32, P * E, "inj"), _stream(stream)))
    del keep


def eqb_lei_inject(grad_s, inj, part_off=None, stream=None):
    T, E = grad_s.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_lei_inject", lib.eqb_lei_inject(
        _ptr(grad_s, torch.float32, T * E, "grad_s"), _ptr(inj, torch.float32, P * E, "inj"), T, E,
        po, P, _stream(stream)))
    del keep


def eqb_lei_router_backward(z, topk_idx, grad_score, grad_z, inj=None, part_off=None, stream=None):
    T, E = z.shape
    K = topk_idx.shape[1]
    po, P, keep = _offsets(part_off, T)
    _check("eqb_lei_router_backward", lib.eqb_lei_router_backward(
        _ptr(z, _Z, name="z"), _ptr(topk_idx, torch.int32, T * K, "topk_idx"),
        _ptr(grad_score, torch.float32, T * K, "grad_score"), _ptr(inj, torch.float32, P * E, "inj"),
        T, E, K, po, P, _ptr(grad_z, torch.float32, T * E, "grad_z"), _stream(stream)))
    del keep


def eqb_layer_workspace_size(E: int, P: int) -> int:
    return int(lib.eqb_layer_workspace_size(E, P))


def eqb_layer_workspace_zero_bytes(E: int, P: int) -> int:
    """Leading bytes of a layer workspace that hold its counters (zero
    before and after every call); the rest is the fine pass's scratch."""
    return int(lib.eqb_layer_workspace_zero_bytes(E, P))


def layer_marks(events):
    """The marks argument of eqb_layer from five torch.cuda.Event objects (or
    None entries).  An event's handle exists once it has been recorded, so
    each is recorded once here first."""
    handles = []
    for ev in events:
        if ev is None:
            handles.append(None)
            continue
        if not ev.cuda_event:
            ev.record()
        handles.append(ev.cuda_event)
    return (ctypes.c_void_p * 5)(*handles)


def eqb_layer(z, b, K, topk_idx, topk_score, tau, load, q_bf16, b_next, dev_status, workspace,
              part_off=None, hist_hi_sum=None, hist_lo_sum=None, marks=None, stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_layer", lib.eqb_layer(
        _ptr(z, _Z, name="z"), _ptr(b, torch.float32, E, "b"), T, E, K, po, P,
        _ptr(topk_idx, torch.int32, T * K, "topk_idx"), _ptr(topk_score, torch.float32, T * K, "topk_score"),
        _ptr(tau, torch.float32, T, "tau"), _ptr(load, torch.int32, P * E, "load"),
        _ptr(q_bf16, _Z, E, "q_bf16"), _ptr(b_next, torch.float32, E, "b_next"),
        _ptr(hist_hi_sum, torch.int32, E * EQB_NBINS, "hist_hi_sum"),
        _ptr(hist_lo_sum, torch.int32, E * EQB_NBINS, "hist_lo_sum"),
        _ptr(dev_status, torch.int32, 1, "dev_status"), _ptr(workspace, torch.uint8, name="workspace"),
        workspace.numel(), marks, _stream(stream)))
    del keep


def eqb_layer_noalloc(z, b, K, topk_idx, topk_score, tau, load, q_bf16, b_next, dev_status, part_off=None,
                      hist_hi_sum=None, hist_lo_sum=None, stream=None):
    T, E = z.shape
    po, P, keep = _offsets(part_off, T)
    _check("eqb_layer_noalloc", lib.eqb_layer_noalloc(
        _ptr(z, _Z, name="z"), _ptr(b, torch.float32, E, "b"), T, E, K, po, P,
        _ptr(topk_idx, torch.int32, T * K, "topk_idx"), _ptr(topk_score, torch.float32, T * K, "topk_score"),
        _ptr(tau, torch.float32, T, "tau"), _ptr(load, torch.int32, P * E, "load"),
        _ptr(q_bf16, _Z, E, "q_bf16"), _ptr(b_next, torch.float32, E, "b_next"),
        _ptr(hist_hi_sum, torch.int32, E * EQB_NBINS, "hist_hi_sum"),
        _ptr(hist_lo_sum, torch.int32, E * EQB_NBINS, "hist_lo_sum"),
        _ptr(dev_status, torch.int32, 1, "dev_status"), _stream(stream)))
    del keep


def eqb_set_max_blocks(max_blocks: int) -> None:
    """Test control: caps the streaming kernels' grids for calls made later
    from the calling thread only."""
    _check("eqb_set_max_blocks", lib.eqb_set_max_blocks(int(max_blocks)))


def eqb_get_max_blocks() -> int:
    return int(lib.eqb_get_max_blocks())


def eqb_rank(T_total: int, K: int, E: int) -> int:
    return int(lib.eqb_rank(T_total, K, E))


class Layer:
    """Device buffers for one layer's routing + EQB statistics, reused across calls."""

    def __init__(self, T: int, E: int, K: int, P: int = 1, device="cuda"):
        self.T, self.E, self.K, self.P = T, E, K, P
        dev = torch.device(device)
        i32 = dict(dtype=torch.int32, device=dev)
        self.topk_idx = torch.empty((T, K), **i32)
        self.topk_score = torch.empty((T, K), dtype=torch.float32, device=dev)
        self.tau = torch.empty(T, dtype=torch.float32, device=dev)
        # counters that are zeroed before every pass, kept in one buffer so a
        # single fill clears them all
        n_load, n_hist = P * E, P * E * EQB_NBINS
        self._counts = torch.empty(n_load + 2 * n_hist + 1, **i32)
        self.load = self._counts[:n_load].view(P, E)
        self.hist_hi = self._counts[n_load:n_load + n_hist].view(P, E, EQB_NBINS)
        self.hist_lo = self._counts[n_load + n_hist:n_load + 2 * n_hist].view(P, E, EQB_NBINS)
        self.dev_status = self._counts[-1:]
        self.H = torch.empty((E, EQB_NBINS), **i32)
        self.L = torch.empty((E, EQB_NBINS), **i32)
        self.sel_hi = torch.empty(E, **i32)
        self.sel_lo = torch.empty(E, **i32)
        self.rank_in_bin = torch.empty(E, dtype=torch.int64, device=dev)
        self.q_bf16 = torch.empty(E, dtype=torch.int16, device=dev)
        self.b_next = torch.empty(E, dtype=torch.float32, device=dev)

    def _layer_buffers(self):
        """Buffers of the one-call layer (eqb_layer): a workspace, zeroed once
        here and left zeroed by every call, and the outputs it writes."""
        if getattr(self, "workspace", None) is None:
            dev = self.topk_idx.device
            n = eqb_layer_workspace_size(self.E, self.P)
            self.workspace = torch.zeros(n, dtype=torch.uint8, device=dev)
            self.load_out = torch.empty((self.P, self.E), dtype=torch.int32, device=dev)
            self.status = torch.empty(1, dtype=torch.int32, device=dev)

    def step(self, z, b, part_off=None, sums=False, marks=None, stream=None):
        """One layer through eqb_layer: one C call, five kernels, no fill of
        counters (the workspace comes back zeroed).  Writes topk_idx,
        topk_score, tau, load_out, q_bf16, b_next, status and, with sums=True,
        the summed counts H and L.  marks: see layer_marks."""
        self._layer_buffers()
        eqb_layer(z, b, self.K, self.topk_idx, self.topk_score, self.tau, self.load_out, self.q_bf16,
                  self.b_next, self.status, self.workspace, part_off,
                  self.H if sums else None, self.L if sums else None, marks, stream)
        return self

    def step_results(self) -> dict:
        """Host copies of the one-call layer's outputs (synchronises)."""
        torch.cuda.synchronize()
        g = lambda t: t.cpu().numpy()
        return dict(idx=g(self.topk_idx), score=g(self.topk_score), tau=g(self.tau), load=g(self.load_out),
                    H=g(self.H), L=g(self.L), bhat=g(self.q_bf16).view(np.uint16), b_next=g(self.b_next),
                    dev_status=int(self.status.item()), workspace_zero=self.counters_zero())

    def counters_zero(self) -> bool:
        """Whether the counter part of the layer workspace is all zero (as
        every call must leave it)."""
        n = eqb_layer_workspace_zero_bytes(self.E, self.P)
        return bool((self.workspace[:n] == 0).all().item())

    def run(self, z, b, part_off=None, fused=True, stream=None):
        """One layer: route (+ coarse counts), select 1, fine counts, select 2."""
        r = eqb_rank(self.T, self.K, self.E)
        self._counts.zero_()
        if fused:
            eqb_route_topk(z, b, self.K, self.topk_idx, self.topk_score, self.tau, part_off,
                           self.load, self.hist_hi, stream)
        else:
            eqb_route_topk(z, b, self.K, self.topk_idx, self.topk_score, self.tau, part_off,
                           None, None, stream)
            eqb_expert_load(self.topk_idx, self.E, self.load, part_off, stream)
            eqb_margin_hist_pass1(z, self.tau, self.hist_hi, part_off, stream)
        eqb_select_quantile(1, self.hist_hi, r, self.sel_hi, self.rank_in_bin,
                            hist_sum=self.H, dev_status=self.dev_status, stream=stream)
        eqb_margin_hist_pass2(z, self.tau, self.sel_hi, self.hist_lo, part_off, stream)
        eqb_select_quantile(2, self.hist_lo, r, self.sel_hi, self.rank_in_bin, self.sel_lo,
                            self.q_bf16, self.b_next, hist_sum=self.L, dev_status=self.dev_status,
                            stream=stream)
        return self

    def results(self) -> dict:
        """Copy every output to host numpy arrays (synchronises)."""
        torch.cuda.synchronize()
        g = lambda t: t.cpu().numpy()
        return dict(idx=g(self.topk_idx), score=g(self.topk_score), tau=g(self.tau), load=g(self.load),
                    H_p=g(self.hist_hi), H=g(self.H), u=g(self.sel_hi), rho=g(self.rank_in_bin),
                    L_p=g(self.hist_lo), L=g(self.L), v=g(self.sel_lo),
                    bhat=g(self.q_bf16).view(np.uint16), b_next=g(self.b_next),
                    dev_status=int(self.dev_status.item()), r=eqb_rank(self.T, self.K, self.E))


def run_layer(z: torch.Tensor, b: torch.Tensor, K: int, part_off=None, fused=True, stream=None) -> Layer:
    T, E = z.shape
    P = 1 if part_off is None else len(part_off) - 1
    return Layer(T, E, K, P, device=z.device).run(z, b, part_off, fused, stream)


def qb_loop(batches, b0, K: int, part_off=None, stream=None):
    """The closed QB loop (Eq. 2) on the GPU: batch q is routed with b^(q),
    its EQB statistics give b^(q+1), which routes batch q+1.  The bias never
    leaves the device between steps.  Returns one dict per step with host
    copies of the bias used (b), the loads [P,E], Global and Local MaxVio
    (Sec. 5) of that routing, b_hat (BF16 bits) and the next bias.  Work is
    enqueued on ``stream`` (default: the current stream)."""
    batches = list(batches)
    if not batches:
        return []
    T, E = batches[0].shape
    P = 1 if part_off is None else len(part_off) - 1
    dev = batches[0].device
    ctx = torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()
    steps = []
    with ctx:
        lay = Layer(T, E, K, P, device=dev)
        mv_g = torch.empty(1, dtype=torch.float64, device=dev)
        mv_l = torch.empty(P, dtype=torch.float64, device=dev)
        mv_m = torch.empty(1, dtype=torch.float64, device=dev)
        b = b0.detach().to(device=dev, dtype=torch.float32).clone()
        for z in batches:
            if tuple(z.shape) != (T, E):
                raise ValueError("every batch of the loop has the same shape")
            lay.run(z, b, part_off)
            eqb_max_violation(lay.load, T, K, mv_g, mv_l, part_off, mv_m)
            b_used = b.clone()
            b.copy_(lay.b_next)
            steps.append(dict(b=b_used.cpu().numpy(), load=lay.load.cpu().numpy(),
                              maxvio_global=float(mv_g.item()), maxvio_local=mv_l.cpu().numpy(),
                              maxvio_local_mean=float(mv_m.item()),
                              bhat=lay.q_bf16.cpu().numpy().view(np.uint16), b_next=b.cpu().numpy(),
                              dev_status=int(lay.dev_status.item())))
    return steps


def _mark(marks, name):
    """Record an event on the current stream after a stage, if asked."""
    if marks is not None:
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()
        marks.append((name, ev))


def rank_averaged_qb(z, b, K: int, part_off=None, stream=None, marks=None) -> dict:
    """Rank-averaged QB (Sec. 2): every shard's exact K/E quantile of its own
    margins, averaged over the shards and centred.  Returns host copies of
    the shards' quantiles (BF16 bits [P,E]), the average (binary64 [E]) and
    the centred bias.  ``marks``, a list, receives (stage, event) pairs
    recorded after each device stage."""
    T, E = z.shape
    P = 1 if part_off is None else len(part_off) - 1
    ctx = torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()
    with ctx:
        dev = z.device
        i32 = dict(dtype=torch.int32, device=dev)
        idx = torch.empty((T, K), **i32)
        score = torch.empty((T, K), dtype=torch.float32, device=dev)
        tau = torch.empty(T, dtype=torch.float32, device=dev)
        hist = torch.zeros((2, P, E, EQB_NBINS), **i32)
        status = torch.zeros(1, **i32)
        sel_hi = torch.empty((P, E), **i32)
        sel_lo = torch.empty((P, E), **i32)
        rib = torch.empty((P, E), dtype=torch.int64, device=dev)
        q = torch.empty((P, E), dtype=torch.int16, device=dev)
        b_avg = torch.empty(E, dtype=torch.float64, device=dev)
        b_next = torch.empty(E, dtype=torch.float32, device=dev)
        _mark(marks, "start")
        eqb_route_topk(z, b, K, idx, score, tau, part_off, None, hist[0])
        _mark(marks, "route_hist1")
        eqb_select_quantile_local(1, hist[0], T, K, sel_hi, rib, part_off=part_off, dev_status=status)
        _mark(marks, "select1_local")
        eqb_margin_hist_pass2_local(z, tau, sel_hi, hist[1], part_off)
        _mark(marks, "hist2_local")
        eqb_select_quantile_local(2, hist[1], T, K, sel_hi, rib, sel_lo, q, part_off, status)
        _mark(marks, "select2_local")
        eqb_rank_average(q, T, b_next, b_avg, part_off)
        _mark(marks, "rank_average")
        return dict(bhat_p=q.cpu().numpy().view(np.uint16), b_avg=b_avg.cpu().numpy(),
                    b_next=b_next.cpu().numpy(), dev_status=int(status.item()))


def histogram_qb(z, b, K: int, lo: float, hi: float, nbins: int, part_off=None, stream=None,
                 marks=None) -> dict:
    """Fixed-resolution histogram QB (Sec. 2): margin counts over nbins
    uniform bins of [lo, hi), summed over the shards, the K/E quantile read
    off the sum by linear interpolation within its bin, then centred.
    Returns host copies of the counts [P,E,nbins], the estimate (binary64 [E])
    and the centred bias.  ``marks`` as for rank_averaged_qb."""
    T, E = z.shape
    P = 1 if part_off is None else len(part_off) - 1
    ctx = torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()
    with ctx:
        dev = z.device
        idx = torch.empty((T, K), dtype=torch.int32, device=dev)
        score = torch.empty((T, K), dtype=torch.float32, device=dev)
        tau = torch.empty(T, dtype=torch.float32, device=dev)
        hist = torch.zeros((P, E, nbins), dtype=torch.int32, device=dev)
        status = torch.zeros(1, dtype=torch.int32, device=dev)
        est = torch.empty(E, dtype=torch.float64, device=dev)
        b_next = torch.empty(E, dtype=torch.float32, device=dev)
        _mark(marks, "start")
        eqb_route_topk(z, b, K, idx, score, tau, part_off)
        _mark(marks, "route")
        eqb_margin_hist_uniform(z, tau, lo, hi, hist, part_off)
        _mark(marks, "uniform_hist")
        eqb_select_uniform(hist, eqb_rank(T, K, E), lo, hi, est, b_next, status)
        _mark(marks, "select_uniform")
        return dict(counts=hist.cpu().numpy(), est=est.cpu().numpy(), b_next=b_next.cpu().numpy(),
                    dev_status=int(status.item()))
