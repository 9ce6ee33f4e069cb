"""Seeded random layer shapes for the GPU parity tests (inputs only: no
arithmetic of the method, no oracle)."""
import numpy as np

import workloads as W


def random_layer_case(i):
    """Seeded random layer: expert count, fan-out (mostly the common small
    K, sometimes up to E - 1), batch size over five decades, unequal
    partitions with empty ones, a grid cap, and one of the data kinds
    (smooth logits, a tie grid, boosted tokens, non-positive ties)."""
    rng = np.random.default_rng(7000 + i)
    E = int(rng.choice([8, 16, 32, 64, 128, 256]))
    K = int(rng.integers(1, min(E - 1, 16) + 1)) if rng.random() < 0.7 else int(rng.integers(1, E))
    T = int(np.exp(rng.uniform(0.0, np.log(60000.0))))
    P = int(rng.integers(1, 7))
    kind = str(rng.choice(["normal", "tie", "boost", "negtie"]))
    w = W.Workload(f"random{i}", T=T, E=E, K=K, P=P, seed=7000 + i, kind=kind,
                   z_sigma=float(rng.uniform(0.5, 2.0)), z_mean=float(rng.uniform(-3.0, 1.0)),
                   off_sigma=float(rng.uniform(0.0, 1.0)), b_sigma=float(rng.uniform(0.0, 0.3)),
                   b_bf16=bool(rng.random() < 0.3), boost_frac=0.05, boost=3.0)
    z, b, _ = W.generate(w)
    off = np.sort(rng.integers(0, T + 1, P - 1)) if P > 1 else np.zeros(0, np.int64)
    off = np.concatenate([[0], off, [T]]).astype(np.int64)
    cap = int(rng.choice([0, 0, 0, 1, 3, 17, 96]))
    return w, z, b, off, cap
