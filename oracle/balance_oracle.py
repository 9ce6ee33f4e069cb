"""CPU oracle for the load-balance quantities around the EQB step.

TEST INFRASTRUCTURE ONLY.  Like ``eqb_oracle``, this module exists to check
the GPU library: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import it, and it shares no code, constant
table or helper with the HIP path.

Written from arXiv 2609.28053:

* MaxVio (Sec. 5 and Appendix E, "Balance metrics"): for a token batch B,
  MaxVio(B) = max_e [ f_e(B) / fbar(B) - 1 ] with the uniform target
  fbar(B) = K|B|/E (Sec. 2).  Global MaxVio takes the loads of the whole
  batch; Local MaxVio is computed on each local batch (a partition here) and
  then averaged over the local batches.
* The closed QB loop (Eq. 2): the statistics of step q give the bias
  b^(q+1) that routes the batch of step q+1.
* Load-Error Injection (Sec. 4, Eq. lei and the normalisation that bounds
  it): for a local batch, rho_e = f_e/fbar - 1 = E (F_e - Q_e); optionally
  rho~ = rho tanh(xi)/xi with xi = ||rho||_inf / c (and tanh(xi)/xi := 1 at
  xi = 0); the router-score gradient of every token of that local batch gets
  grad_{s_{t,e}} += eta rho~_e.
* The router backward with LEI (Sec. 2 Eq. 1; Sec. 4 Eq. lei): with
  s_{t,e} = sigmoid(z_{t,e}) weighting the selected experts, the gradient of
  the loss w.r.t. the logits is (g_{t,e} + eta rho~_{p(t),e}) * s (1 - s),
  where g_{t,e} is the mixture-weight gradient of a selected expert (zero for
  the others) and the injected term reaches every expert of every token of
  the local batch.
* The two distributed QB statistics EQB is compared with (Sec. 2, after
  Eq. 2; Sec. 3): the rank-averaged quantile, where each rank takes the K/E
  quantile of its own shard and the ranks average them, and the
  fixed-resolution histogram estimate, where the ranks all-reduce margin
  counts over fixed bins and read the quantile off the summed histogram.

Readings taken where the paper is silent:
  * MaxVio is evaluated in binary64 as (max_e f_e) * E / (K |B|) - 1: the
    maximum over the integer loads is exact, then one division and one
    subtraction, each rounded to nearest even.  (The maximum of
    f_e/fbar - 1 over e is attained at the largest f_e because the map is
    increasing.)
  * An empty batch has no uniform target; its MaxVio is NaN.
  * LEI's injected value eta * rho~_e is computed in binary64 as
    rho = (f E)/(K |B|) - 1, xi = max|rho| / c, rho~ = rho * (tanh(xi)/xi),
    value = eta * rho~, and rounded once to binary32; c <= 0 means the
    unnormalised form (rho~ = rho).  An empty local batch injects 0.
  * The injection itself is one binary32 addition per score, rounded to
    nearest even.
  * Router backward: sigmoid'(z) = e / (1 + e)^2 with e = exp(-|z|), in
    binary64; the selected experts' gradients arrive as [T,K] with their
    indices; the result is compared with the device's binary32 within a
    tolerance (the device evaluates exp in binary32).
  * Rank-averaged QB: shard p's quantile is its exact r_p-th smallest BF16
    margin, r_p = ceil(|B_p| K/E); the average over the non-empty shards is a
    binary64 sum in ascending p divided by their number; the result is
    centred like Eq. 2 (binary64 mean over e, one rounding to binary32).
  * Fixed-resolution histogram: the margin is the binary32 difference
    tau - z (no BF16 rounding); with w = hi - lo and s = nbins / w, both
    binary32, its bin is floor((m - lo) * s) in binary32, clamped to
    [0, nbins-1].  The r-th smallest is read as lo + (j + (r - C_{j-1}) / H_j)
    * (hi - lo) / nbins in binary64 (j the first bin whose running count C_j
    reaches r, linear within the bin), then centred like Eq. 2.
"""
from __future__ import annotations

import math

import numpy as np

from . import eqb_oracle as _eqb


# --------------------------------------------------------------------------
# MaxVio (Sec. 5; Appendix E "Balance metrics")
# --------------------------------------------------------------------------
def max_violation_of(load_e, n_tokens: int, K: int) -> float:
    """MaxVio of one batch from its per-expert loads f_e (length E)."""
    load_e = np.asarray(load_e, dtype=np.int64)
    E = load_e.size
    if n_tokens == 0:
        return float("nan")
    fmax = int(load_e.max())
    return float(np.float64(fmax * E) / np.float64(K * n_tokens) - np.float64(1.0))


def max_violation(load_pe, part_off, K: int):
    """(global MaxVio, [P] local MaxVio) from per-partition loads [P,E]."""
    load_pe = np.asarray(load_pe, dtype=np.int64)
    part_off = np.asarray(part_off, dtype=np.int64)
    sizes = np.diff(part_off)
    glob = max_violation_of(load_pe.sum(axis=0), int(part_off[-1]), K)
    local = np.array([max_violation_of(load_pe[p], int(sizes[p]), K) for p in range(load_pe.shape[0])])
    return glob, local


def local_maxvio_mean(local) -> float:
    """Local MaxVio as Appendix E reports it: the per-local-batch values
    averaged over the local batches (empty partitions, which have no value,
    are left out).  Binary64 sum in ascending partition order, divided by the
    number of values; NaN when there is none."""
    vals = [float(v) for v in np.asarray(local, np.float64) if not math.isnan(float(v))]
    if not vals:
        return float("nan")
    acc = 0.0
    for v in vals:
        acc = acc + v
    return acc / len(vals)


# --------------------------------------------------------------------------
# The closed QB loop (Eq. 2)
# --------------------------------------------------------------------------
def qb_loop(batches, b0, K: int, part_off=None, threads: int = 1):
    """Route batch q with b^(q), take its EQB statistics, and carry the
    centred bias b^(q+1) to batch q+1.  Returns one dict per step with the
    bias used (b), the loads [P,E], the global and local MaxVio of that
    routing, and the next bias (b_next)."""
    b = np.asarray(b0, dtype=np.float32).copy()
    steps = []
    for z in batches:
        T = z.shape[0]
        off = np.array([0, T], np.int64) if part_off is None else np.asarray(part_off, np.int64)
        res = _eqb.run_layer(z, b, K, off, threads=threads)
        glob, local = max_violation(res["load"], off, K)
        steps.append(dict(b=b.copy(), load=res["load"], maxvio_global=glob, maxvio_local=local,
                          maxvio_local_mean=local_maxvio_mean(local), bhat=res["bhat"], b_next=res["b_next"]))
        b = res["b_next"].astype(np.float32)
    return steps


# --------------------------------------------------------------------------
# Load-Error Injection (Sec. 4, Eq. lei and its normalisation)
# --------------------------------------------------------------------------
def lei_residual(load_pe, part_off, K: int, eta: float, c: float) -> np.ndarray:
    """The value each partition injects into its router-score gradients,
    eta * rho~_{p,e}, as binary32 [P,E]."""
    load_pe = np.asarray(load_pe, dtype=np.int64)
    part_off = np.asarray(part_off, dtype=np.int64)
    P, E = load_pe.shape
    out = np.zeros((P, E), np.float32)
    for p in range(P):
        n = int(part_off[p + 1] - part_off[p])
        if n == 0:
            continue
        rho = [float(f * E) / float(K * n) - 1.0 for f in load_pe[p]]
        scale = 1.0
        if c > 0:
            xi = max(abs(v) for v in rho) / float(c)
            scale = math.tanh(xi) / xi if xi > 0 else 1.0
        out[p] = np.array([float(eta) * (v * scale) for v in rho], dtype=np.float64).astype(np.float32)
    return out


def lei_inject(grad_s, inj, part_off) -> np.ndarray:
    """grad_{s_{t,e}} + eta rho~_{p(t),e} for every token t of partition p,
    one binary32 addition each."""
    grad_s = np.asarray(grad_s, dtype=np.float32)
    part_off = np.asarray(part_off, dtype=np.int64)
    out = grad_s.copy()
    for p in range(len(part_off) - 1):
        r0, r1 = int(part_off[p]), int(part_off[p + 1])
        out[r0:r1] = (grad_s[r0:r1] + inj[p][None, :]).astype(np.float32)
    return out


def lei_router_backward(z_bits, topk_idx, grad_score, inj, part_off) -> np.ndarray:
    """d loss / d z [T,E] in binary64: (g_{t,e} + inj[p(t),e]) * sigmoid'(z_{t,e}),
    g_{t,e} the mixture-weight gradient of selected experts (from [T,K]); inj
    may be None (no injection)."""
    zf = _eqb.bf16_to_f32(z_bits).astype(np.float64)
    T, E = zf.shape
    part_off = np.asarray(part_off, np.int64)
    g = np.zeros((T, E), np.float64)
    rows = np.repeat(np.arange(T), np.asarray(topk_idx).shape[1])
    g[rows, np.asarray(topk_idx).ravel()] = np.asarray(grad_score, np.float32).astype(np.float64).ravel()
    if inj is not None:
        for p in range(part_off.size - 1):
            g[part_off[p]:part_off[p + 1]] += np.asarray(inj[p], np.float32).astype(np.float64)[None, :]
    e = np.exp(-np.abs(zf))
    return g * (e / (1.0 + e) ** 2)


# --------------------------------------------------------------------------
# The statistics EQB is compared with (Sec. 2, after Eq. 2; Sec. 3)
# --------------------------------------------------------------------------
def _centre64(vals64) -> np.ndarray:
    vals64 = [float(v) for v in vals64]
    total = 0.0
    for v in vals64:
        total += v
    mean = total / len(vals64)
    return np.array([np.float32(v - mean) for v in vals64], dtype=np.float32)


def rank_averaged_qb(z_bits, b, K: int, part_off):
    """Each shard's exact K/E quantile of its own margins, averaged over the
    non-empty shards, then centred.  Returns (bhat_p BF16 bits [P,E], a NaN
    pattern for empty shards; the average [E] binary64; the centred bias)."""
    z_bits = np.asarray(z_bits, np.uint16)
    T, E = z_bits.shape
    part_off = np.asarray(part_off, np.int64)
    P = part_off.size - 1
    _, _, tau = _eqb.route_topk(z_bits, b, K)
    keys = _eqb.margin_keys(z_bits, tau)
    bhat_p = np.full((P, E), 0x7FC0, np.uint16)      # an empty shard has no quantile (NaN)
    vals = []
    for p in range(P):
        r0, r1 = int(part_off[p]), int(part_off[p + 1])
        if r1 == r0:
            continue
        r_p = _eqb.quantile_rank(r1 - r0, K, E)
        kstar = _eqb.select_by_sort(keys[r0:r1], r_p)
        bhat_p[p] = _eqb.kappa_inv(kstar)
        vals.append(_eqb.bf16_to_f32(bhat_p[p]).astype(np.float64))
    avg = np.zeros(E, np.float64)
    for e in range(E):
        total = 0.0
        for v in vals:
            total += float(v[e])
        avg[e] = total / len(vals)
    return bhat_p, avg, _centre64(avg)


def uniform_bins(z_bits, tau, lo: float, hi: float, nbins: int) -> np.ndarray:
    """Bin index [T,E] of every binary32 margin tau_t - z_{t,e}."""
    zf = _eqb.bf16_to_f32(z_bits)
    m = (np.asarray(tau, np.float32)[:, None] - zf).astype(np.float32)
    lo32, hi32 = np.float32(lo), np.float32(hi)
    scale = np.float32(np.float32(nbins) / np.float32(hi32 - lo32))
    x = ((m - lo32).astype(np.float32) * scale).astype(np.float32)
    return np.clip(np.floor(x), 0, nbins - 1).astype(np.int64)


def histogram_qb(z_bits, b, K: int, part_off, lo: float, hi: float, nbins: int):
    """Fixed-resolution global-histogram estimate of the K/E quantile.
    Returns (per-partition counts [P,E,nbins], estimate [E] binary64, the
    centred bias)."""
    z_bits = np.asarray(z_bits, np.uint16)
    T, E = z_bits.shape
    part_off = np.asarray(part_off, np.int64)
    P = part_off.size - 1
    _, _, tau = _eqb.route_topk(z_bits, b, K)
    bins = uniform_bins(z_bits, tau, lo, hi, nbins)
    counts = np.zeros((P, E, nbins), np.int64)
    for p in range(P):
        r0, r1 = int(part_off[p]), int(part_off[p + 1])
        for e in range(E):
            counts[p, e] = np.bincount(bins[r0:r1, e], minlength=nbins)
    total = counts.sum(axis=0)
    r = _eqb.quantile_rank(T, K, E)
    lo64 = float(np.float32(lo))
    width = (float(np.float32(hi)) - lo64) / nbins
    est = np.zeros(E, np.float64)
    for e in range(E):
        run = np.cumsum(total[e])
        j = int(np.searchsorted(run, r))          # first bin whose running count reaches r
        before = int(run[j - 1]) if j > 0 else 0
        est[e] = lo64 + (j + (r - before) / int(total[e, j])) * width
    return counts, est, _centre64(est)
