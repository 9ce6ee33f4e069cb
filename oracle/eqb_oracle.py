"""CPU oracle for one MoE layer's routing and Exact Quantile Balancing statistics.

TEST INFRASTRUCTURE ONLY.  This module exists to check the GPU library.  Only
the test suite, the package smoke check and the benchmark's CPU-baseline leg
may import it.  It shares no code, constant table or helper with the HIP path.

Everything here is the plain definition, written for a reader holding the
paper (arXiv 2609.28053, "Exact Quantile Balancing and Load-Error Injection for
Mixture-of-Experts"):

* Routing (Sec. 2, Eq. 1): I_t = Top-K(z_t + b); the bias only selects, the
  selected experts carry the unbiased scores s_{t,e} = sigmoid(z_{t,e}).
* Loads (Sec. 2): f_e(B) = #{t in B : e in I_t}.
* QB cutoff (Sec. 2, "Quantile Balancing"): tau_t is the (K+1)st largest entry
  of z_t + b.
* QB update (Eq. 2): b_hat_e is the K/E quantile of the margins tau_t - z_{t,e}
  over the global batch, i.e. the r-th smallest with r = TK/E (Sec. 3), and the
  new bias is b_hat minus its mean.
* EQB (Sec. 3, Algorithm 1 in Appendix C): margins are BF16 values, encoded
  order-preservingly as a 16-bit key kappa = (high byte h, low byte l);
  coarse counts H_{p,e,u} over h, fine counts L_{p,e,v} over l inside the
  selected high byte u_e; the all-reduce sums the per-partition counts.

The oracle does NOT run the two-pass radix select.  It computes the quantile
by fully sorting each expert's keys and taking the r-th smallest (the exact
empirical quantile the paper says EQB recovers, Sec. 3 "Distributed radix
selection" and "Communication"), and derives u_e, rho_e, v_e and the counts from
that sorted result and plain counting.

Readings taken where the paper is silent (each is listed in the design notes):
  * z + b is one IEEE binary32 addition (round to nearest even);
  * ties in Top-K go to the lower expert index, and I_t lists the experts in
    rank order (score descending, then index ascending); -0 and +0 compare equal;
  * tau_t keeps the bit pattern of the element at sorted position K;
  * a margin is the binary32 difference tau_t - z_{t,e}, rounded once to BF16
    (nearest, ties to even), with subnormals kept;
  * kappa(bits) = bits XOR (0xFFFF if the sign bit is set else 0x8000), the
    order of IEEE totalOrder (so -0 < +0);
  * r = ceil(T*K/E) over the global T (the paper assumes TK/E is an integer);
  * the mean is a float64 sum in ascending expert order, divided by E, the
    difference taken in float64 and rounded once to binary32;
  * sigmoid is evaluated in float64 and rounded once to binary32.

Inputs are finite (no NaN/Inf), and the logits are given as BF16 bit patterns
(uint16), the bias as float32.
"""
from __future__ import annotations

import concurrent.futures as _cf

import numpy as np

NBINS = 256


# --------------------------------------------------------------------------
# BF16 primitives
# --------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of BF16 bit patterns to float32 (BF16 is the top half)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round float32 values to BF16 bit patterns, nearest with ties to even.

    Written as the definition: the two BF16 neighbours of x are the truncation
    toward zero (keep the top 16 bits) and the next BF16 away from zero; the
    result is the one nearer to x, compared exactly in float64, and the one
    with an even last bit on a tie.  A value at or beyond the midpoint between
    the largest finite BF16 and 2**128 rounds to infinity.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    if np.any((bits & 0x7F800000) == 0x7F800000):
        raise ValueError("oracle inputs must be finite")
    lo = (bits >> 16).astype(np.uint32)              # truncation toward zero
    hi = lo + 1                                      # next BF16 away from zero
    xd = np.abs(x.astype(np.float64))
    lo_val = np.abs(bf16_to_f32(lo.astype(np.uint16)).astype(np.float64))
    # the magnitude of the away-from-zero neighbour; 0x7F80 stands for 2**128
    hi_mag = hi & 0x7FFF
    hi_val = np.where(hi_mag == 0x7F80, 2.0 ** 128,
                      np.abs(bf16_to_f32((hi & 0xFFFF).astype(np.uint16)).astype(np.float64)))
    d_lo = xd - lo_val
    d_hi = hi_val - xd
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ((lo & 1) == 1))
    return np.where(take_hi, hi, lo).astype(np.uint16)


def kappa(bits: np.ndarray) -> np.ndarray:
    """Order-preserving 16-bit key of a BF16 pattern (Algorithm 1 preamble).

    Negative values have all bits flipped, non-negative values only the sign
    bit, so unsigned key order equals IEEE totalOrder of the BF16 values.
    The high byte is h, the low byte l.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return np.where(b & 0x8000, b ^ np.uint16(0xFFFF), b ^ np.uint16(0x8000)).astype(np.uint16)


def kappa_inv(key: np.ndarray) -> np.ndarray:
    """Inverse of kappa: recover the BF16 pattern from its key."""
    k = np.asarray(key, dtype=np.uint16)
    return np.where(k & 0x8000, k ^ np.uint16(0x8000), k ^ np.uint16(0xFFFF)).astype(np.uint16)


# --------------------------------------------------------------------------
# Routing: Top-K of z + b, tau, scores (Sec. 2, Eq. 1; App. B threshold identity)
# --------------------------------------------------------------------------
def biased_scores(z_bits: np.ndarray, b: np.ndarray) -> np.ndarray:
    """s_{t,e} = z_{t,e} + b_e as one binary32 addition."""
    return bf16_to_f32(z_bits) + np.asarray(b, dtype=np.float32)[None, :]


def _row_chunks(T: int, chunk: int, threads: int, fn) -> None:
    """Apply fn(r0, r1) to independent row ranges, optionally on threads."""
    starts = list(range(0, T, chunk))
    if threads <= 1 or len(starts) <= 1:
        for r0 in starts:
            fn(r0, min(T, r0 + chunk))
        return
    with _cf.ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda r0: fn(r0, min(T, r0 + chunk)), starts))


def route_topk(z_bits: np.ndarray, b: np.ndarray, K: int, chunk: int = 1 << 15,
               threads: int = 1):
    """Return (idx int32 [T,K], score float32 [T,K], tau float32 [T]).

    Each row is fully sorted by (s descending, expert index ascending); the
    first K experts are I_t in rank order and tau_t is the element at sorted
    position K, i.e. the (K+1)st largest entry of z_t + b.  Rows are
    independent, so they are processed in chunks to bound memory.
    """
    z_bits = np.asarray(z_bits, dtype=np.uint16)
    T, E = z_bits.shape
    if not 1 <= K < E:
        raise ValueError("need 1 <= K < E")
    idx = np.empty((T, K), np.int32)
    score = np.empty((T, K), np.float32)
    tau = np.empty(T, np.float32)
    cols = np.arange(E)

    def rows_fn(r0, r1):
        s = biased_scores(z_bits[r0:r1], b)
        # lexsort: last key is primary.  -s sorts by s descending; numeric
        # compare treats -0 and +0 as equal, so the index then decides.
        order = np.lexsort((np.broadcast_to(cols, s.shape), -s), axis=-1)
        rows = np.arange(r1 - r0)[:, None]
        idx[r0:r1] = order[:, :K]
        tau[r0:r1] = s[rows[:, 0], order[:, K]]
        zsel = bf16_to_f32(z_bits[r0:r1][rows, order[:, :K]]).astype(np.float64)
        score[r0:r1] = sigmoid64(zsel).astype(np.float32)

    _row_chunks(T, chunk, threads, rows_fn)
    return idx, score, tau


def sigmoid64(x: np.ndarray) -> np.ndarray:
    """The logistic function in float64 (Eq. 1: unbiased, not normalised)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def expert_load(idx: np.ndarray, E: int, part_off) -> np.ndarray:
    """f_{p,e} = #{t in partition p : e in I_t} (Sec. 2), int64 [P,E]."""
    off = np.asarray(part_off, dtype=np.int64)
    P = len(off) - 1
    out = np.zeros((P, E), np.int64)
    for p in range(P):
        sel = idx[off[p]:off[p + 1]].ravel()
        out[p] = np.bincount(sel, minlength=E)[:E]
    return out


# --------------------------------------------------------------------------
# Margins, keys, counts (Eq. 2; Algorithm 1)
# --------------------------------------------------------------------------
def margin_keys(z_bits: np.ndarray, tau: np.ndarray, chunk: int = 1 << 15,
                threads: int = 1) -> np.ndarray:
    """kappa(bf16(tau_t - z_{t,e})) as uint16 [T,E]."""
    z_bits = np.asarray(z_bits, dtype=np.uint16)
    T, E = z_bits.shape
    keys = np.empty((T, E), np.uint16)

    def rows_fn(r0, r1):
        m32 = np.asarray(tau[r0:r1], np.float32)[:, None] - bf16_to_f32(z_bits[r0:r1])
        keys[r0:r1] = kappa(f32_to_bf16_rne(m32))

    _row_chunks(T, chunk, threads, rows_fn)
    return keys


def count_high(keys: np.ndarray, part_off) -> np.ndarray:
    """H_{p,e,u} = #{t in partition p : h_{t,e} = u} (Algorithm 1, step 1)."""
    off = np.asarray(part_off, dtype=np.int64)
    P = len(off) - 1
    E = keys.shape[1]
    H = np.zeros((P, E, NBINS), np.int64)
    for p in range(P):
        hk = keys[off[p]:off[p + 1]] >> 8
        for e in range(E):
            H[p, e] = np.bincount(hk[:, e], minlength=NBINS)
    return H


def count_low(keys: np.ndarray, u: np.ndarray, part_off) -> np.ndarray:
    """L_{p,e,v} = #{t in p : h_{t,e} = u_e and l_{t,e} = v} (Algorithm 1, step 4)."""
    off = np.asarray(part_off, dtype=np.int64)
    P = len(off) - 1
    E = keys.shape[1]
    L = np.zeros((P, E, NBINS), np.int64)
    for p in range(P):
        kp = keys[off[p]:off[p + 1]]
        for e in range(E):
            col = kp[:, e]
            inbin = col[(col >> 8) == u[e]]
            L[p, e] = np.bincount(inbin & 0xFF, minlength=NBINS)
    return L


def quantile_rank(T: int, K: int, E: int) -> int:
    """r = TK/E (Sec. 3), rounded up when TK/E is not an integer."""
    return -(-T * K // E)


def select_by_sort(keys: np.ndarray, r: int) -> np.ndarray:
    """k*_e = the r-th smallest key of expert e, by a full sort of its column."""
    T, E = keys.shape
    if not 1 <= r <= T:
        raise ValueError("need 1 <= r <= T")
    out = np.empty(E, np.uint16)
    for e in range(E):
        out[e] = np.sort(keys[:, e], kind="stable")[r - 1]
    return out


def centred_bias(bhat_bits: np.ndarray) -> np.ndarray:
    """b = b_hat - mean(b_hat) (Eq. 2), float64 arithmetic rounded once to binary32."""
    vals = bf16_to_f32(bhat_bits).astype(np.float64)
    acc = 0.0
    for v in vals:                 # ascending expert order
        acc = acc + float(v)
    mean = acc / len(vals)
    return np.array([np.float32(float(v) - mean) for v in vals], dtype=np.float32)


# --------------------------------------------------------------------------
# The whole layer
# --------------------------------------------------------------------------
def run_layer(z_bits: np.ndarray, b: np.ndarray, K: int, part_off=None,
              threads: int = 1) -> dict:
    """All outputs of one layer's routing + EQB statistics.

    Returns a dict with idx, score, tau, load [P,E], H_p [P,E,256], H [E,256],
    r, u, rho, v, L_p [P,E,256], L [E,256], bhat (BF16 bits [E]) and b_next
    (float32 [E]).  Count arrays are int64.  ``threads`` only spreads the
    independent row ranges over threads; it does not change any result.
    """
    z_bits = np.asarray(z_bits, dtype=np.uint16)
    T, E = z_bits.shape
    if part_off is None:
        part_off = np.array([0, T], np.int64)
    part_off = np.asarray(part_off, np.int64)
    if part_off[0] != 0 or part_off[-1] != T or np.any(np.diff(part_off) < 0):
        raise ValueError("partition offsets must rise from 0 to T")
    _check_finite(z_bits, b)
    idx, score, tau = route_topk(z_bits, b, K, threads=threads)
    load = expert_load(idx, E, part_off)
    keys = margin_keys(z_bits, tau, threads=threads)
    H_p = count_high(keys, part_off)
    H = H_p.sum(axis=0)
    r = quantile_rank(T, K, E)
    kstar = select_by_sort(keys, r)
    u = (kstar >> 8).astype(np.int64)
    v = (kstar & 0xFF).astype(np.int64)
    rho = np.array([r - H[e, :u[e]].sum() for e in range(E)], np.int64)
    L_p = count_low(keys, u, part_off)
    L = L_p.sum(axis=0)
    bhat = kappa_inv(kstar)
    return dict(idx=idx, score=score, tau=tau, load=load, H_p=H_p, H=H, r=r,
                u=u, rho=rho, v=v, L_p=L_p, L=L, bhat=bhat,
                b_next=centred_bias(bhat), keys=keys)


def _check_finite(z_bits, b):
    if np.any((np.asarray(z_bits, np.uint16) & 0x7F80) == 0x7F80):
        raise ValueError("logits must be finite")
    if not np.all(np.isfinite(np.asarray(b, np.float32))):
        raise ValueError("bias must be finite")
