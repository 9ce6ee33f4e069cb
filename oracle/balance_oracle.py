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

Readings taken where the paper is silent:
  * MaxVio is evaluated in binary64 as (max_e f_e) * E / (K |B|) - 1: the
    maximum over the integer loads is exact, then one division and one
    subtraction, each rounded to nearest even.  (The maximum of
    f_e/fbar - 1 over e is attained at the largest f_e because the map is
    increasing.)
  * An empty batch has no uniform target; its MaxVio is NaN.
"""
from __future__ import annotations

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
