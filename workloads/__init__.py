"""Seeded synthetic router-logit workloads shaped like the paper's MoE layers.

This module only draws random numbers.  It holds none of the routing or
quantile arithmetic, so both the CPU oracle tests and the GPU path can take
their inputs from here without sharing any of the method's code.

The paper trains a 7.5B MoE with E=256 routed experts and K=6 (Appendix E,
"Model, training, and evaluation"); its router logits come from trained
weights on a pretraining corpus that is not available.  The recipes below
stand in for those logits with normal draws plus a per-expert offset (expert
skew), a few boosted tokens, and a tie-heavy grid.  A sigmoid router's logits
sit mostly below zero (its selected experts score well under 1/2), so one
workload is shifted down until the cutoffs straddle zero, and one puts a grid
of non-positive logits under a bias of signed zeros.

Every array is produced deterministically from (config, seed):
  * a main generator ``default_rng(seed)`` draws, in this order, the
    per-expert offsets, the bias b, and the partition cut points;
  * the logits are drawn in row chunks of 2**18 tokens, chunk c using its own
    generator ``default_rng([seed, c])``, so chunks can be produced in any
    order or in parallel threads and the result does not change;
  * further batches of the same distribution (same offsets, bias and
    partitions; fresh logits) use ``default_rng([seed, batch, c])`` for
    batch >= 1, so batch 0 is the workload itself;
  * float32 values are rounded to BF16 by torch's CPU conversion
    (round-to-nearest-even), a library routine independent of both the
    oracle and the kernels.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Optional

import numpy as np

CHUNK_ROWS = 1 << 18


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int
    E: int
    K: int
    P: int
    seed: int
    kind: str            # "normal", "tie", "boost", "negtie"
    z_sigma: float = 1.0
    z_mean: float = 0.0
    off_sigma: float = 0.0
    b_sigma: float = 0.0
    b_bf16: bool = False
    split: str = "equal"  # "equal" or "random"
    boost_frac: float = 0.0
    boost: float = 0.0

    def with_T(self, T: int, P: Optional[int] = None) -> "Workload":
        return dataclasses.replace(self, T=T, P=self.P if P is None else P)

    @property
    def r(self) -> int:
        """Rank of the balanced quantile, r = T*K/E rounded up."""
        return -(-self.T * self.K // self.E)


# tiny (E=8), skewed E=64, random split E=128, tie-heavy grid E=64, the large
# E=256 layer with boosted tokens and one rank's share of it, logits centred
# below zero (cutoffs of both signs), and non-positive ties under a bias of
# +0 and -0.
WORKLOADS = {
    "tiny": Workload("tiny", T=4096, E=8, K=2, P=1, seed=0, kind="normal",
                     z_sigma=1.0, off_sigma=0.5, b_sigma=0.1),
    "skew64": Workload("skew64", T=262144, E=64, K=6, P=4, seed=1, kind="normal",
                       z_sigma=1.0, off_sigma=1.0, b_sigma=0.2),
    "split128": Workload("split128", T=1048576, E=128, K=8, P=8, seed=2, kind="normal",
                         z_sigma=1.5, off_sigma=0.0, b_sigma=0.0, split="random"),
    "tie64": Workload("tie64", T=1048576, E=64, K=4, P=2, seed=3, kind="tie",
                      b_sigma=0.05, b_bf16=True),
    "large256": Workload("large256", T=4194304, E=256, K=8, P=16, seed=4, kind="boost",
                         z_sigma=1.0, off_sigma=0.7, b_sigma=0.1,
                         boost_frac=0.05, boost=3.0),
    # one data-parallel rank's share of the paper's optimizer step: 576 sequences
    # of 16,384 tokens over 64 ranks, E = 256, K = 6 (Appendix E)
    "rank256": Workload("rank256", T=147456, E=256, K=6, P=1, seed=5, kind="boost",
                        z_sigma=1.0, off_sigma=0.7, b_sigma=0.1,
                        boost_frac=0.05, boost=3.0),
    # logits of a sigmoid router, shifted down by 2.375: about two thirds of
    # the cutoffs are negative, and most rows mix scores of both signs
    "neg256": Workload("neg256", T=1048576, E=256, K=8, P=4, seed=6, kind="boost",
                       z_sigma=1.0, z_mean=-2.375, off_sigma=0.7, b_sigma=0.1,
                       boost_frac=0.05, boost=3.0),
    # z uniform over k/4, k = -16..0, zero's sign a fair coin; b is +0 or -0
    # per expert: exact ties on non-positive scores, zero cutoffs of both signs
    "signs64": Workload("signs64", T=262144, E=64, K=4, P=2, seed=7, kind="negtie"),
}
WORKLOAD_ORDER = ["tiny", "skew64", "split128", "tie64", "large256", "rank256", "neg256", "signs64"]

TIE_GRID_STEPS = 16   # values k/4 for k = -16..16: 33 distinct BF16 values in [-4, 4]


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def partition_offsets(w: Workload, rng: np.random.Generator) -> np.ndarray:
    """Contiguous token partitions [off[p], off[p+1]) standing in for P ranks."""
    if w.split == "random" and w.P > 1 and w.T > w.P:
        cuts = np.sort(rng.choice(w.T - 1, w.P - 1, replace=False) + 1)
        return np.concatenate([[0], cuts, [w.T]]).astype(np.int64)
    base = np.linspace(0, w.T, w.P + 1)
    off = np.floor(base).astype(np.int64)
    off[-1] = w.T
    return off


def _z_chunk(w: Workload, c: int, rows: int, off: np.ndarray, batch: int = 0) -> np.ndarray:
    g = np.random.default_rng([w.seed, c] if batch == 0 else [w.seed, batch, c])
    if w.kind in ("tie", "negtie"):
        top = TIE_GRID_STEPS if w.kind == "tie" else 0
        k = g.integers(-TIE_GRID_STEPS, top + 1, size=(rows, w.E))
        neg = g.integers(0, 2, size=(rows, w.E)).astype(bool)
        bits = _to_bf16_bits(k.astype(np.float32) / 4.0)
        bits[(k == 0) & neg] = 0x8000     # zero's sign is a fair coin: -0 and +0 both occur
        return bits
    x = g.standard_normal((rows, w.E), dtype=np.float32)
    if w.z_sigma != 1.0:
        x *= np.float32(w.z_sigma)
    if w.z_mean != 0.0:
        x += np.float32(w.z_mean)
    if w.off_sigma != 0.0:
        x += off[None, :]
    if w.kind == "boost":
        mask = g.random(rows) < w.boost_frac
        cols = g.integers(0, w.E, size=rows)
        ridx = np.nonzero(mask)[0]
        x[ridx, cols[ridx]] += np.float32(w.boost)
    return _to_bf16_bits(x)


def generate(w: Workload, threads: Optional[int] = None, batch: int = 0):
    """Return (z_bits uint16 [T,E], b float32 [E], part_off int64 [P+1]).

    ``batch`` selects a fresh draw of the logits from the same distribution;
    b and part_off do not depend on it."""
    if batch < 0:
        raise ValueError("batch must be non-negative")
    rng = np.random.default_rng(w.seed)
    off = (rng.standard_normal(w.E, dtype=np.float32) * np.float32(w.off_sigma)
           if w.off_sigma else np.zeros(w.E, np.float32))
    if w.b_sigma:
        b = rng.standard_normal(w.E, dtype=np.float32) * np.float32(w.b_sigma)
        if w.b_bf16:
            b = (_to_bf16_bits(b).astype(np.uint32) << 16).view(np.float32)
    elif w.kind == "negtie":
        b = np.where(rng.integers(0, 2, size=w.E).astype(bool), np.float32(-0.0), np.float32(0.0))
    else:
        b = np.zeros(w.E, np.float32)
    part_off = partition_offsets(w, rng)

    z = np.empty((w.T, w.E), np.uint16)
    nchunks = -(-w.T // CHUNK_ROWS) if w.T else 0

    def work(c):
        r0 = c * CHUNK_ROWS
        r1 = min(w.T, r0 + CHUNK_ROWS)
        z[r0:r1] = _z_chunk(w, c, r1 - r0, off, batch)

    n = threads or min(16, os.cpu_count() or 1)
    if nchunks <= 1 or n <= 1:
        for c in range(nchunks):
            work(c)
    else:
        with _cf.ThreadPoolExecutor(n) as ex:
            list(ex.map(work, range(nchunks)))
    return z, b.astype(np.float32), part_off
