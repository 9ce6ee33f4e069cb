"""CPU oracle for the load-balance quantities around the EQB step.

TEST INFRASTRUCTURE ONLY.  Like ``eqb_oracle``, this module exists to check
the GPU library: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import it, and it shares no code, constant
table or helper with the HIP path.

Written from arXiv 2609.28053:

* MaxVio (Sec. 5 and Appendix E, "Balance metrics"): for a token batch B,
  MaxVio(B) = max_e [ f_e(B) / fbar(B) - 1 ] with the uniform target
  fbar(B) = K|B|/E (Sec. 2).  Global MaxVio takes the loads of the whole
  batch, Local MaxVio those of one local batch (a partition here).
* The closed QB loop (Eq. 2): the statistics of step q give the bias
  b^(q+1) that routes the batch of step q+1.
* Load-Error Injection (Sec. 4, Eq. lei and the normalisation that bounds
  it): for a local batch, rho_e = f_e/fbar - 1 = E (F_e - Q_e); optionally
  rho~ = rho tanh(xi)/xi with xi = ||rho||_inf / c (and tanh(xi)/xi := 1 at
  xi = 0); the router-score gradient of every token of that local batch gets
  grad_{s_{t,e}} += eta rho~_e.

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
                          bhat=res["bhat"], b_next=res["b_next"]))
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
