"""Benchmark: one MoE layer's routing + Exact Quantile Balancing statistics.

A step is the whole path over one batch already resident in HBM, one call of
eqb_layer (five kernels, no counter fill: the workspace is left zeroed):
  route_topk + loads + coarse counts -> select pass 1 (clears the coarse
  counts) -> fine counts (pass 2) -> select pass 2 (clears the fine counts)
  -> centred bias and status.

    python bench.py [--gpus 1] [--steps 100] [--warmup 30] [--workload large256]
    python bench.py --all-configs        # one line per smaller workload instead

Prints one JSON line.  ``value`` is tokens/s of the whole step; ``roofline``
describes the dominant kernel (route + coarse pass), timed live with HIP
events that eqb_layer records around it on its stream; ``cpu_baseline`` times
the CPU oracle on a bounded slice of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0                     # MI355X HBM3E, vendor figure
METRIC = "routing+EQB tokens/s per MoE layer; achieved HBM GB/s vs peak"
CSRC = os.path.join(ROOT, "paper_2609_28053_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "route_hist1_large256_traffic.txt")
VALU_FILE = os.path.join(ROOT, "profiles", "route_fine_large256_valu_counters.txt")
# Vector issue peak: 256 CUs x 4 SIMDs, a wave64 instruction occupies a
# 16-lane SIMD for 4 cycles, 2.4 GHz: 256 * 4 * 16 * 2.4e9 lane-operations/s
# (the vendor's 157.3 TFLOP/s FP32 figure counts an FMA as two and packed
# FP32 as two more).
VALU_PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9


def route_bytes_per_token(E, K):
    """Algorithmic bytes of route + coarse pass: read z row, write idx, score, tau."""
    return 2 * E + 4 * K + 4 * K + 4


def pass_bytes_per_token(E, K):
    """Algorithmic bytes of the whole step: z twice, idx, score, tau written and read back."""
    return 4 * E + 8 * K + 8


ROUTE_SOURCES = [os.path.join(CSRC, f) for f in ("route.hip", "eqb_device.hpp", "eqb_internal.hpp")] + \
    [os.path.join(ROOT, "include", "eqb.h")]


def source_hash():
    """Hash of the route kernel's sources; counters taken on other sources are stale."""
    h = hashlib.sha256()
    for path in ROUTE_SOURCES:
        with open(path, "rb") as f:
            h.update(os.path.basename(path).encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def read_traffic(T):
    """Measured HBM bytes per launch of the route kernel from a committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_sha256_16") != source_hash() or int(vals.get("T", -1)) != T:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def read_valu_per_element(T):
    """Issued VALU instructions per (token, expert) of the route kernel, from
    the committed SQ_INSTS_VALU summary, if it was taken on the current kernel
    source and the same token count."""
    if not os.path.exists(VALU_FILE):
        return None
    lines = open(VALU_FILE).read().splitlines()
    head = " ".join(l for l in lines if l.startswith("#"))
    m_hash = re.search(r"sources sha256\[:16\] = ([0-9a-f]{16})", head)
    m_t = re.search(r"\bT=(\d+)", head)
    if not m_hash or m_hash.group(1) != source_hash() or not m_t or int(m_t.group(1)) != T:
        return None
    section = None
    for line in lines:
        if line.startswith("## "):
            section = line
        elif section and "route_fast" in section and line.startswith("valu_per_element"):
            return float(line.split("=", 1)[1])
    return None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(w, rows, threads=1):
    import workloads as W
    from oracle import eqb_oracle as O
    sub = w.with_T(rows, 1)
    z, b, off = W.generate(sub)
    t0 = time.perf_counter()
    O.run_layer(z, b, sub.K, off, threads=threads)
    dt = time.perf_counter() - t0
    return {"value": rows / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"first {rows} tokens of {w.name} (E={w.E}, K={w.K}, one partition), "
                      f"full oracle layer (row sorts, margins, column sorts, counts) in "
                      f"{dt:.1f} s on {threads} thread(s) of {os.cpu_count()} visible cores ({cpu_model()})"}


def qb_loop_leg(w, eqb, torch, steps, dev, part_off):
    """The closed QB loop (Eq. 2) over fresh batches of the same distribution,
    starting from b = 0: Global and Local MaxVio (Sec. 5) of every step."""
    import workloads as W
    zs = []
    for q in range(1, steps + 1):
        z, _, _ = W.generate(w, batch=q)
        zs.append(torch.from_numpy(z.view(np.int16)).to(dev))
        del z
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = eqb.qb_loop(zs, torch.zeros(w.E, dtype=torch.float32), w.K, part_off)
    dt = time.perf_counter() - t0
    del zs
    return {"batches": f"fresh draws 1..{steps} of {w.name} (same per-expert offsets), b^(0) = 0",
            "maxvio_global": [r["maxvio_global"] for r in res],
            "maxvio_local": [r["maxvio_local_mean"] for r in res],
            "maxvio_local_note": "Local MaxVio as Appendix E reports it: per partition, averaged over the "
                                 "partitions; maxvio_local_max is the largest partition's value",
            "maxvio_local_max": [float(np.nanmax(r["maxvio_local"])) for r in res],
            "ms_per_step_wall": dt * 1e3 / steps,
            "dev_status": max(r["dev_status"] for r in res)}


def lei_leg(w, eqb, torch, lay, load, zt, part_off, stream, reps=10):
    """Load-Error Injection (Sec. 4) after the step: the residual from the
    step's per-partition loads, the injection into a [T,E] binary32
    score-gradient buffer (read and written once: 8 bytes per score), and the
    fused router backward (reads z and the [T,K] mixture gradients, writes the
    binary32 logit gradient: 6E + 8K bytes per token)."""
    dev = load.device
    inj = torch.empty((w.P, w.E), dtype=torch.float32, device=dev)
    grad = torch.zeros((w.T, w.E), dtype=torch.float32, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    with torch.cuda.stream(stream):
        for _ in range(2):
            eqb.eqb_lei_residual(load, w.T, w.K, 2e-5, 1.0, inj, part_off, stream)
            eqb.eqb_lei_inject(grad, inj, part_off, stream)
        ev[0].record(stream)
        for _ in range(reps):
            eqb.eqb_lei_residual(load, w.T, w.K, 2e-5, 1.0, inj, part_off, stream)
        ev[1].record(stream)
        for _ in range(reps):
            eqb.eqb_lei_inject(grad, inj, part_off, stream)
        ev[2].record(stream)
    torch.cuda.synchronize()
    inject_ms = ev[1].elapsed_time(ev[2]) / reps
    gbs = 8.0 * w.T * w.E / (inject_ms * 1e-3) / 1e9
    # fused router backward: the step's scores stand in for the mixture gradients
    gz = grad
    bw = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    with torch.cuda.stream(stream):
        eqb.eqb_lei_router_backward(zt, lay.topk_idx, lay.topk_score, gz, inj, part_off, stream)
        bw[0].record(stream)
        for _ in range(reps):
            eqb.eqb_lei_router_backward(zt, lay.topk_idx, lay.topk_score, gz, inj, part_off, stream)
        bw[1].record(stream)
    torch.cuda.synchronize()
    bwd_ms = bw[0].elapsed_time(bw[1]) / reps
    bwd_bytes = (6 * w.E + 8 * w.K) * w.T
    bwd_gbs = bwd_bytes / (bwd_ms * 1e-3) / 1e9
    del grad, gz
    return {"residual_us": ev[0].elapsed_time(ev[1]) * 1e3 / reps, "inject_ms": inject_ms,
            "inject_bytes": 8 * w.T * w.E, "inject_gbs": gbs, "inject_frac_of_peak": gbs / HBM_PEAK_GBS,
            "router_backward_ms": bwd_ms, "router_backward_bytes": bwd_bytes, "router_backward_gbs": bwd_gbs,
            "router_backward_frac_of_peak": bwd_gbs / HBM_PEAK_GBS, "eta": 2e-5, "c": 1.0}


STAGES = ("route_hist1", "select1", "margin_hist2", "select2_center")
ROUTE_EVENT_EVERY = 5        # timed steps per pair of route-kernel events


def make_events(torch, n, k=5):
    return [[torch.cuda.Event(enable_timing=True) for _ in range(k)] for _ in range(n)]


def signs_leg(eqb, torch, zt, bt, po, lay, stream, reps=10, shift=4.0):
    """The whole step on the step's logits shifted down by `shift`, which
    makes every cutoff negative: a sigmoid router's logits sit mostly below
    zero, and the path should not depend on the sign of tau.  The shifted copy
    is made on the device by torch (input preparation, finished before the
    timed steps).  Shifted and unshifted steps alternate, so both see the
    same clock and thermal state; stage times come from the events eqb_layer
    records."""
    zs = (zt.view(torch.bfloat16).float() - shift).to(torch.bfloat16).view(torch.int16)
    torch.cuda.synchronize()
    evs = {name: make_events(torch, reps) for name in ("shifted", "unshifted")}
    marks = {name: [eqb.layer_marks(e) for e in evs[name]] for name in evs}
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(3):
            lay.step(zs, bt, po, stream=stream)
            lay.step(zt, bt, po, stream=stream)
        for i in range(reps):
            lay.step(zs, bt, po, marks=marks["shifted"][i], stream=stream)
            lay.step(zt, bt, po, marks=marks["unshifted"][i], stream=stream)
        torch.cuda.synchronize()
        lay.step(zs, bt, po, stream=stream)
    torch.cuda.synchronize()
    frac = float((lay.tau <= 0).float().mean().item())
    del zs
    out = {"shift": -shift, "tau_nonpositive_frac": frac}
    for name, e in evs.items():
        out[name] = {"route_hist1_ms": float(np.median([x[0].elapsed_time(x[1]) for x in e])),
                     "margin_hist2_ms": float(np.median([x[2].elapsed_time(x[3]) for x in e])),
                     "step_ms_median": float(np.median([x[0].elapsed_time(x[4]) for x in e]))}
    return out


def per_rank_leg(eqb, torch, stream, steps=400, event_steps=100):
    """The whole step at one data-parallel rank's share of the paper's
    training step (rank256: 147,456 tokens of E = 256, K = 6, App. E):
    the wall clock over `steps` back-to-back eqb_layer calls, and the device
    time of one step from the events eqb_layer records at its start and end
    (a separate run, so the wall-clock loop records no events)."""
    import workloads as W
    w = W.WORKLOADS["rank256"]
    z, b, off = W.generate(w)
    dev = torch.device("cuda:0")
    zt = torch.from_numpy(z.view(np.int16)).to(dev)
    bt = torch.from_numpy(b).to(dev)
    po = eqb.PartOffsets([int(x) for x in off])
    lay = eqb.Layer(w.T, w.E, w.K, w.P, device=dev)
    evs = make_events(torch, event_steps)
    marks = [eqb.layer_marks([e[0], None, None, None, e[4]]) for e in evs]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(50):
            lay.step(zt, bt, po, stream=stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            lay.step(zt, bt, po, stream=stream)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        for i in range(event_steps):
            lay.step(zt, bt, po, marks=marks[i], stream=stream)
        torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    dev_ms = float(np.median([e[0].elapsed_time(e[4]) for e in evs]))
    gbs = pass_bytes_per_token(w.E, w.K) * w.T / (ms * 1e-3) / 1e9
    return {"workload": w.name, "T": w.T, "E": w.E, "K": w.K, "steps": steps, "ms_per_step": ms,
            "device_ms_per_step_median": dev_ms, "wall_over_device": ms / dev_ms,
            "tokens_per_s": w.T / (ms * 1e-3), "pass_hbm_gbs": gbs, "pass_frac_of_peak": gbs / HBM_PEAK_GBS,
            "note": "z is 72 MiB here, so part of it can be served from the 256 MB memory-side cache"}


def variants_leg(w, eqb, torch, zt, bt, lay, part_off):
    """The statistics EQB is compared with (Sec. 2), on the same batch: the
    rank-averaged quantile (P shards, and P/4 shards to show that it depends
    on the split) and the fixed-resolution histogram estimate (256 bins on
    [-8, 8)), each against EQB's exact global quantile b_hat."""
    exact = (lay.q_bf16.to(torch.int32).cpu().numpy().astype(np.uint32) << 16).view(np.float32)
    exact = exact.astype(np.float64)
    out = {}

    def stage_ms(marks):
        """Device time of each stage from the events the driver recorded."""
        return {marks[i + 1][0]: marks[i][1].elapsed_time(marks[i + 1][1]) for i in range(len(marks) - 1)}

    eqb.rank_averaged_qb(zt, bt, w.K, part_off)                 # warm-up (allocations)
    marks = []
    ra = eqb.rank_averaged_qb(zt, bt, w.K, part_off, marks=marks)
    out["rank_avg_stage_ms"] = stage_ms(marks)
    coarse = [part_off[i] for i in range(0, len(part_off), 4)]
    if coarse[-1] != part_off[-1]:
        coarse.append(part_off[-1])
    ra4 = eqb.rank_averaged_qb(zt, bt, w.K, coarse)
    eqb.histogram_qb(zt, bt, w.K, -8.0, 8.0, 256, part_off)
    marks = []
    hq = eqb.histogram_qb(zt, bt, w.K, -8.0, 8.0, 256, part_off, marks=marks)
    out["histogram_stage_ms"] = stage_ms(marks)
    d = lambda a: np.abs(a - exact)
    out.update({
        "rank_avg_P": len(part_off) - 1,
        "rank_avg_max_abs_err": float(d(ra["b_avg"]).max()),
        "rank_avg_mean_abs_err": float(d(ra["b_avg"]).mean()),
        "rank_avg_split_dependence_max_abs": float(np.abs(ra["b_avg"] - ra4["b_avg"]).max()),
        "rank_avg_coarse_P": len(coarse) - 1,
        "histogram_bins": 256, "histogram_range": [-8.0, 8.0],
        "histogram_max_abs_err": float(d(hq["est"]).max()),
        "histogram_mean_abs_err": float(d(hq["est"]).mean()),
        "dev_status": max(ra["dev_status"], ra4["dev_status"], hq["dev_status"]),
    })
    return out


def roofline_of(w, route_ms, vpe, traffic):
    """The dominant kernel against the limit that binds it.  Its algorithmic
    bytes over its live duration give the HBM view; its issued VALU
    instructions (from committed counters, when they were taken on the current
    sources) over the same duration give the vector-issue view.  The view with
    the larger fraction of its peak is the binding one and fills the
    top-level fields."""
    route_bytes = route_bytes_per_token(w.E, w.K) * w.T
    route_gbs = route_bytes / (route_ms * 1e-3) / 1e9
    hbm = {"achieved": route_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": route_gbs / HBM_PEAK_GBS,
           "algorithmic_bytes": route_bytes}
    out = {"kernel": "route_hist1", "launch_ms": route_ms, "traffic": traffic, "hbm": hbm, "alu": None}
    if vpe is not None:
        ops = vpe * w.T * w.E / (route_ms * 1e-3)
        out["alu"] = {"achieved": ops / 1e12, "peak": VALU_PEAK_LANE_OPS / 1e12, "unit": "T VALU lane-op/s",
                      "frac": ops / VALU_PEAK_LANE_OPS, "valu_per_element": vpe,
                      "source": os.path.relpath(VALU_FILE, ROOT)}
    bind = out["alu"] if out["alu"] is not None and out["alu"]["frac"] > hbm["frac"] else hbm
    out.update({"bound": "alu" if bind is out["alu"] else "hbm", "achieved": bind["achieved"],
                "peak": bind["peak"], "unit": bind["unit"], "frac": bind["frac"]})
    if out["alu"] is None:
        out["alu_note"] = "no VALU counters for the current sources; bound taken from HBM"
    return out


def stats(x):
    x = np.asarray(x, np.float64)
    return {"median": float(np.median(x)), "max": float(x.max()), "min": float(x.min()),
            "mean": float(x.mean())}


def time_layer(eqb, torch, w, zt, bt, po, stream, steps, warmup, min_warmup_s, stage_steps=20):
    """Warm up, time `steps` back-to-back layers on the wall clock (events
    only around the route kernel), then a separate stage run with an event
    between every kernel and host timestamps around every call."""
    lay = eqb.Layer(w.T, w.E, w.K, w.P, device=zt.device)
    lay._layer_buffers()
    # Route-kernel events on every ROUTE_EVENT_EVERY-th step of the timed
    # region: each event record costs the queue a few microseconds.
    rev = make_events(torch, (steps + ROUTE_EVENT_EVERY - 1) // ROUTE_EVENT_EVERY, 2)
    rmarks = [eqb.layer_marks([a, b, None, None, None]) for a, b in rev]
    sev = make_events(torch, stage_steps)
    smarks = [eqb.layer_marks(e) for e in sev]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        # Warm-up, untimed: at least `warmup` steps and at least min_warmup_s
        # seconds of them.  Per-dispatch traces show the route kernel's time
        # falling by about a quarter over the first ~30 steps after the set-up
        # (input generation and the 2 GiB upload leave the GPU idle).
        warmup_run = 0
        t_w = time.perf_counter()
        while warmup_run < warmup or time.perf_counter() - t_w < min_warmup_s:
            lay.step(zt, bt, po, stream=stream)
            warmup_run += 1
            if warmup_run % 10 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()
        # Timed region: exactly `steps` layers; the only events in it are the
        # two eqb_layer records around the route kernel on its own stream, on
        # every ROUTE_EVENT_EVERY-th step.
        t0 = time.perf_counter()
        for i in range(steps):
            m = rmarks[i // ROUTE_EVENT_EVERY] if i % ROUTE_EVENT_EVERY == 0 else None
            lay.step(zt, bt, po, marks=m, stream=stream)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        # Stage breakdown: a separate run with an event after every kernel.
        host = []
        for i in range(stage_steps):
            h0 = time.perf_counter()
            lay.step(zt, bt, po, marks=smarks[i], stream=stream)
            host.append((time.perf_counter() - h0) * 1e3)
        torch.cuda.synchronize()
    assert int(lay.status.item()) == 0, "device reported a rank beyond the counts"
    route = [a.elapsed_time(b) for a, b in rev]
    stage = {n: [e[j].elapsed_time(e[j + 1]) for e in sev] for j, n in enumerate(STAGES)}
    step_dev = [e[0].elapsed_time(e[4]) for e in sev]
    gaps = [sev[i][4].elapsed_time(sev[i + 1][0]) for i in range(stage_steps - 1)]
    # An outlier stage either follows a host stall (the GPU caught up with the
    # host and waited: the call that enqueued it took long, or the device sat
    # idle before the step) or is the device's own.
    med = {n: float(np.median(v)) for n, v in stage.items()}
    outliers = []
    for i in range(stage_steps):
        for n in STAGES:
            if stage[n][i] > 1.5 * med[n] + 0.02:
                outliers.append({"step": i, "stage": n, "ms": stage[n][i], "host_enqueue_ms": host[i],
                                 "idle_before_ms": gaps[i - 1] if i > 0 else None,
                                 "cause": "host" if host[i] > 1.0 or (i > 0 and gaps[i - 1] > 0.05) else "device"})
    breakdown = {"stage_ms": {n: stats(v) for n, v in stage.items()},
                 "step_ms": dict(stats(step_dev), p90=float(np.percentile(step_dev, 90))),
                 "host_enqueue_ms": stats(host), "device_idle_between_steps_ms": stats(gaps),
                 "outliers": outliers, "steps": stage_steps,
                 "note": "a separate run with an event after every kernel (eqb_layer marks)"}
    route_stats = dict(stats(route), launches=len(route), of_timed_steps=f"every {ROUTE_EVENT_EVERY}th")
    return lay, elapsed * 1e3 / steps, warmup_run, float(np.mean(route)), route_stats, breakdown


def bench_line(w, ms_per_step, warmup_args, route_ms, route_stats, breakdown):
    steps, warmup, warmup_run = warmup_args
    tokens_per_s = w.T / (ms_per_step * 1e-3)
    pass_gbs = pass_bytes_per_token(w.E, w.K) * w.T / (ms_per_step * 1e-3) / 1e9
    traffic = read_traffic(w.T)
    vpe = read_valu_per_element(w.T)
    roof = roofline_of(w, route_ms, vpe, traffic)
    roof["launch_ms_stats"] = route_stats
    return {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "warmup_steps_run": warmup_run,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "T": w.T, "E": w.E, "K": w.K, "P": w.P,
                   "logits": LOGITS.get(w.name, w.kind),
                   "parallelism": "single GPU; P partitions summed on device"},
        "pass_hbm_gbs": pass_gbs,
        "pass_frac_of_peak": pass_gbs / HBM_PEAK_GBS,
        "stages": breakdown,
        "roofline": roof,
    }


LOGITS = {
    "large256": "bf16 N(0,1) + per-expert N(0,0.7) offset, 5% tokens +3 on one expert",
    "tiny": "bf16 N(0,1) + per-expert N(0,0.5) offset",
    "skew64": "bf16 N(0,1) + per-expert N(0,1) offset",
    "split128": "bf16 N(0,1.5), b = 0, random partition sizes",
    "tie64": "33 BF16 values k/4 in [-4,4] (both zeros), b bf16 N(0,0.05)",
}
SMALL_CONFIGS = ("tiny", "skew64", "split128", "tie64")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--min-warmup-s", type=float, default=0.3,
                    help="keep warming up (untimed) until this many seconds of steps have run: after the "
                         "host-side set-up the GPU takes a few tens of milliseconds to reach steady clocks")
    ap.add_argument("--workload", default="large256")
    ap.add_argument("--all-configs", action="store_true",
                    help="instead of the main line, one line per smaller workload (tiny, skew64, split128, "
                         "tie64), each with its own single-thread oracle time")
    ap.add_argument("--cpu-rows", type=int, default=1048576,
                    help="tokens in the CPU-oracle baseline slice (0 disables it)")
    ap.add_argument("--qb-steps", type=int, default=4,
                    help="steps of the closed QB loop over fresh batches (0 disables it)")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the LEI and comparison-variant legs (for counter collection)")
    ap.add_argument("--print-source-hash", action="store_true", help="print the kernel source hash and exit")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy a device buffer of this size three times "
                         "(a plain copy of known size, used to scale HBM counters)")
    args = ap.parse_args()
    if args.print_source_hash:
        print(source_hash())
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(the per-rank all-reduce of Algorithm 1 is reproduced as a sum of partition "
              "histograms on one device). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    from paper_2609_28053_amd import eqb

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=dev)     # default priority
    names = SMALL_CONFIGS if args.all_configs else (args.workload,)
    for name in names:
        w = W.WORKLOADS[name]
        t0 = time.time()
        z, b, off = W.generate(w)
        print(f"[bench] generated {w.name} T={w.T} E={w.E} K={w.K} P={w.P} in {time.time() - t0:.1f}s",
              file=sys.stderr, flush=True)
        zt = torch.from_numpy(z.view(np.int16)).to(dev)
        bt = torch.from_numpy(b).to(dev)
        del z
        part_off = [int(x) for x in off]
        po = eqb.PartOffsets(part_off)
        lay, ms_per_step, warmup_run, route_ms, route_stats, breakdown = time_layer(
            eqb, torch, w, zt, bt, po, stream, args.steps, args.warmup, args.min_warmup_s)
        out = bench_line(w, ms_per_step, (args.steps, args.warmup, warmup_run), route_ms, route_stats, breakdown)
        if args.all_configs:
            out["note"] = ("z is at most 256 MiB here, so part of it can be served from the 256 MB "
                           "memory-side cache: the HBM fraction is context, not a bound")
            rows = min(w.T, 262144)
            out["cpu_baseline"] = cpu_baseline(w, rows) if args.cpu_rows > 0 else None
            print(json.dumps(out), flush=True)
            del zt, lay
            continue
        if not args.no_legs:
            out["lei"] = lei_leg(w, eqb, torch, lay, lay.load_out, zt, part_off, stream)
            out["variants"] = variants_leg(w, eqb, torch, zt, bt, lay, part_off)
            out["cutoff_signs"] = signs_leg(eqb, torch, zt, bt, po, lay, stream)
            out["per_rank"] = per_rank_leg(eqb, torch, stream)
        if args.qb_steps > 0:
            del zt
            out["qb_loop"] = qb_loop_leg(w, eqb, torch, args.qb_steps, dev, part_off)
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_rows) if args.cpu_rows > 0 else None
        if args.copy_calibration_mib > 0:
            n = args.copy_calibration_mib << 20
            src = torch.ones(n // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            for _ in range(3):
                dst.copy_(src)
            torch.cuda.synchronize()
            print(f"[bench] copied {n} bytes three times for counter calibration", file=sys.stderr)
        print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
