/*
 * eqb.h - C ABI of the MI355X (gfx950) library for one MoE layer's routing
 * and Exact Quantile Balancing (EQB) statistics.
 *
 * Method: arXiv 2609.28053, "Exact Quantile Balancing and Load-Error Injection
 * for Mixture-of-Experts".  Notation follows the paper:
 *   z[T,E]   router logits (BF16), b[E] expert bias (binary32),
 *   I_t      = Top-K(z_t + b)                          (Sec. 2, Eq. 1)
 *   s_{t,e}  = sigmoid(z_{t,e}) for e in I_t, unbiased  (Sec. 2, Eq. 1)
 *   f_e      = #{t : e in I_t}                          (Sec. 2)
 *   tau_t    = (K+1)st largest entry of z_t + b         (Sec. 2, "Quantile Balancing")
 *   margin   = tau_t - z_{t,e} as a BF16 value, key kappa = (h, l) (Appendix C, Algorithm 1)
 *   r        = T*K/E, the rank of the balanced quantile  (Sec. 3)
 *   H_{p,e,u}, L_{p,e,v}  coarse / fine counts of partition p (Algorithm 1, steps 1 and 4)
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.  Every pointer is a DEVICE pointer except `part_off`, which is a
 *   HOST array read during the call.  The caller allocates and owns every
 *   buffer; the library allocates nothing and keeps no pointer after the call
 *   returns.  Calls only enqueue work on `stream` (a hipStream_t, NULL = the
 *   default stream) and never synchronise the host.
 * Layouts.  Row-major.  z is [T,E] BF16 bit patterns (uint16), 16-byte
 *   aligned.  topk_idx/topk_score are [T,K].  Count arrays are int32:
 *   loads [P,E], coarse/fine histograms [P,E,256] (slab p = partition p).
 * Partitions.  Tokens are split into P contiguous ranges
 *   [part_off[p], part_off[p+1]), standing in for P data-parallel ranks.
 *   part_off has P+1 entries, part_off[0] = 0, part_off[P] = T, non-decreasing
 *   (empty partitions are allowed).  part_off = NULL means P = 1.  Summing the
 *   slabs over p is the all-reduce of Algorithm 1, steps 2 and 5.
 * Accumulation.  Histogram and load outputs are ACCUMULATED (+=): zero them
 *   before the first call of a layer.  Every count must stay in [0, 2^31)
 *   before and after a call: the kernels may add to two adjacent int32
 *   counters with one 64-bit atomic, which is exact only while no counter
 *   wraps.  Counts are token counts, so T < 2^31 keeps them in range.
 * Numerics.  z + b and tau - z are single binary32 operations rounded to
 *   nearest even, with subnormals kept; a margin is rounded once to BF16
 *   (nearest, ties to even).  kappa(bits) = bits ^ (sign ? 0xFFFF : 0x8000),
 *   which orders BF16 values as IEEE totalOrder (-0 < +0).  Top-K ties go to
 *   the lower expert index (-0 and +0 are equal there); I_t is written in rank
 *   order (score descending, then index ascending).  Inputs must be finite.
 * Supported shapes.  E in {8, 16, 32, 64, 128, 256}; 1 <= K < E;
 *   0 <= T < 2^31; 1 <= P <= EQB_MAX_PARTITIONS.
 * Errors.  Every argument check runs before anything is enqueued, so a call
 *   that returns an error has left the stream untouched.  T = 0 returns
 *   EQB_OK and enqueues nothing.
 * Concurrency.  The library keeps no state between calls except a per-device
 *   cache of the compute-unit count (filled once, thread-safe) and the
 *   per-thread test cap of eqb_set_max_blocks.  Calls may be made from
 *   several host threads and on several streams at once; calls that write
 *   the same buffers must be ordered by the caller (same stream, or events).
 */
#ifndef EQB_H
#define EQB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t eqb_status;

#define EQB_OK               0
#define EQB_ERR_INVALID_ARG  1   /* null pointer, bad K/T/P, bad partition table */
#define EQB_ERR_UNSUPPORTED  2   /* E outside the supported set, misaligned z */
#define EQB_ERR_RANK         3   /* r < 1 or r > number of counted margins */
#define EQB_ERR_HIP          4   /* the HIP runtime reported a launch error */
#define EQB_ERR_SCRATCH      5   /* eqb_layer_noalloc: the layer needs more than
                                    EQB_NOALLOC_SCRATCH_BYTES of working memory */

#define EQB_NBINS            256
#define EQB_MAX_PARTITIONS   256

/* Device status word written by eqb_select_quantile. */
#define EQB_DEV_OK                 0
#define EQB_DEV_RANK_EXCEEDS_COUNT 1   /* an expert holds fewer than r (or rho) counts */

/*
 * Routing (Sec. 2, Eq. 1 and "Quantile Balancing"), optionally fused with
 * the coarse pass of Algorithm 1 (step 1).
 *   z [T,E] bf16 bits, b [E] binary32                     (in)
 *   topk_idx [T,K] int32, topk_score [T,K] binary32,
 *   tau [T] binary32                                      (out)
 *   load [P,E] int32 (nullable)                           (+= f_{p,e})
 *   hist_hi [P,E,256] int32 (nullable)                    (+= H_{p,e,u}, u = h of the margin key)
 * tau_t carries the bit pattern of the entry at rank K (0-based).
 * Returns EQB_ERR_INVALID_ARG, EQB_ERR_UNSUPPORTED or EQB_ERR_HIP on failure.
 */
eqb_status eqb_route_topk(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                          int32_t* topk_idx, float* topk_score, float* tau,
                          const int64_t* part_off, int32_t P,
                          int32_t* load, int32_t* hist_hi, void* stream);

/*
 * Coarse pass alone (Algorithm 1, step 1): hist_hi[p,e,u] += #{t in p : h_{t,e} = u},
 * where (h, l) = kappa(bf16(tau_t - z_{t,e})).
 *   z [T,E] bf16 bits, tau [T] binary32 (in); hist_hi [P,E,256] int32 (+=).
 */
eqb_status eqb_margin_hist_pass1(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                 const int64_t* part_off, int32_t P, int32_t* hist_hi,
                                 void* stream);

/*
 * Selection (Algorithm 1, steps 2-3 for pass = 1; steps 5-6 for pass = 2).
 * Both passes first sum the P slabs of `hist` (the all-reduce, steps 2 and 5).
 * pass = 1: hist = H_p [P,E,256].  Writes sel_hi[e] = u_e = min{u : sum_{j<=u} H[e,j] >= r}
 *   and rank_in_bin[e] = rho_e = r - sum_{j<u_e} H[e,j].
 * pass = 2: hist = L_p [P,E,256], reads sel_hi and rank_in_bin.  Writes
 *   sel_lo[e] = v_e = min{v : sum_{j<=v} L[e,j] >= rho_e}, q_bf16[e] = kappa^-1(u_e, v_e)
 *   (the exact r-th smallest BF16 margin, b_hat_e) and, if b_next != NULL,
 *   the centred bias b_next[e] = b_hat_e - mean(b_hat) (Eq. 2): a binary64 sum in
 *   ascending e, divided by E, subtracted in binary64 and rounded once to binary32.
 *   r is the rank over the whole batch (all partitions), see eqb_rank.
 *   hist_sum [E,256] int32 (nullable): receives the summed counts.
 *   dev_status (nullable, int32): set to EQB_DEV_RANK_EXCEEDS_COUNT when some
 *   expert holds fewer than r (pass 1) or rho_e (pass 2) counts; it is never
 *   cleared by the library.  The affected sel_hi/sel_lo entries are -1 and
 *   q_bf16 is a NaN pattern.
 * Returns EQB_ERR_RANK if r < 1; other errors as above.
 */
eqb_status eqb_select_quantile(int32_t pass, const int32_t* hist, int32_t P, int32_t E, int64_t r,
                               int32_t* sel_hi, int64_t* rank_in_bin,
                               int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                               int32_t* hist_sum, int32_t* dev_status, void* stream);

/*
 * Fine pass (Algorithm 1, step 4): rescans z and tau and, for margins whose
 * high byte equals sel_hi[e] = u_e, hist_lo[p,e,v] += #{t in p : h_{t,e} = u_e, l_{t,e} = v}.
 *   z [T,E] bf16 bits, tau [T], sel_hi [E] int32 (in); hist_lo [P,E,256] int32 (+=).
 */
eqb_status eqb_margin_hist_pass2(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                 const int32_t* sel_hi, const int64_t* part_off, int32_t P,
                                 int32_t* hist_lo, void* stream);

/*
 * Expert loads (Sec. 2): load[p,e] += #{t in p : e in I_t} from topk_idx [T,K].
 * Entries outside [0, E) are not counted.
 */
eqb_status eqb_expert_load(const int32_t* topk_idx, int64_t T, int32_t K, int32_t E,
                           const int64_t* part_off, int32_t P, int32_t* load, void* stream);

/*
 * The statistics EQB is compared with (Sec. 2, after Eq. 2; Sec. 3).
 *
 * Rank-averaged QB: every shard (partition) takes the K/E quantile of its own
 * margins and the shards average them.  Each shard's quantile is exact, found
 * by the two passes of Algorithm 1 run on that shard's counts alone:
 *   eqb_select_quantile_local(1, hist_hi [P,E,256]) -> sel_hi, rank_in_bin [P,E]
 *     with r_p = ceil(|B_p| K / E) (no summing over partitions);
 *   eqb_margin_hist_pass2_local: like eqb_margin_hist_pass2, but partition p
 *     counts inside its own bin sel_hi[p,e];
 *   eqb_select_quantile_local(2, hist_lo [P,E,256]) -> sel_lo, q_bf16 [P,E]
 *     (q_bf16[p,e] = b_hat_{p,e}, shard p's r_p-th smallest BF16 margin);
 *   eqb_rank_average: b_avg[e] = sum over non-empty p (binary64, ascending p)
 *     of b_hat_{p,e}, divided by their number (nullable output), and b_next =
 *     b_avg - mean(b_avg), centred as in Eq. 2.
 * An empty partition gets sel = -1 and a NaN q_bf16 and is left out of the
 * average.  dev_status as for eqb_select_quantile.  T and part_off describe
 * the whole batch as in every other call; K < E.
 */
eqb_status eqb_select_quantile_local(int32_t pass, const int32_t* hist, int64_t T, int32_t K, int32_t E,
                                     const int64_t* part_off, int32_t P, int32_t* sel_hi,
                                     int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16,
                                     int32_t* dev_status, void* stream);
eqb_status eqb_margin_hist_pass2_local(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                       const int32_t* sel_hi, const int64_t* part_off, int32_t P,
                                       int32_t* hist_lo, void* stream);
eqb_status eqb_rank_average(const uint16_t* q_bf16, int64_t T, int32_t E, const int64_t* part_off,
                            int32_t P, double* b_avg, float* b_next, void* stream);

/*
 * Fixed-resolution histogram QB: margin counts over nbins uniform bins of
 * [lo, hi), summed over the shards, and the quantile read off the sum.
 *   eqb_margin_hist_uniform: hist[p,e,j] += #{t in p : bin(tau_t - z_{t,e}) = j},
 *     the margin being the binary32 difference (no BF16 rounding) and
 *     bin(m) = floor((m - lo) * s) clamped to [0, nbins-1], with
 *     s = nbins / (hi - lo), all in binary32.  hist [P,E,nbins] int32 (+=).
 *   eqb_select_uniform: sums the P slabs, finds the first bin j whose running
 *     count C_j reaches r and writes est[e] = lo + (j + (r - C_{j-1}) / H_j) *
 *     (hi - lo) / nbins in binary64 (linear within the bin), and, if b_next is
 *     not NULL, b_next = est - mean(est) centred as in Eq. 2.
 * 1 <= nbins <= 256 and lo < hi (finite) or EQB_ERR_INVALID_ARG.
 */
eqb_status eqb_margin_hist_uniform(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                   const int64_t* part_off, int32_t P, float lo, float hi, int32_t nbins,
                                   int32_t* hist, void* stream);
eqb_status eqb_select_uniform(const int32_t* hist, int32_t P, int32_t E, int32_t nbins, int64_t r, float lo,
                              float hi, double* est, float* b_next, int32_t* dev_status, void* stream);

/*
 * Balance metric (Sec. 5; Appendix E, "Balance metrics"):
 *   MaxVio(B) = max_e [ f_e(B) / fbar(B) - 1 ],  fbar(B) = K|B|/E  (Sec. 2).
 *   load [P,E] int32 (in): per-partition loads f_{p,e}, e.g. from eqb_route_topk.
 *   maxvio_global [1] binary64 (out): the whole batch, f_e = sum_p f_{p,e}, |B| = T
 *     ("Global MaxVio").
 *   maxvio_local [P] binary64 (out, nullable): partition p alone,
 *     |B| = part_off[p+1] - part_off[p]; NaN for an empty partition.
 *   maxvio_local_mean [1] binary64 (out, nullable): "Local MaxVio" as Appendix E
 *     reports it, the per-partition values averaged over the non-empty
 *     partitions (binary64 sum in ascending p, divided by their number).
 * Each value is (max_e f_e) * E / (K * |B|) - 1 in binary64: an exact integer
 * maximum, then one division and one subtraction, each rounded to nearest even.
 * T = 0 returns EQB_OK and writes nothing.
 */
eqb_status eqb_max_violation(const int32_t* load, int64_t T, int32_t K, int32_t E,
                             const int64_t* part_off, int32_t P, double* maxvio_global,
                             double* maxvio_local, double* maxvio_local_mean, void* stream);

/*
 * Load-Error Injection, the residual (Sec. 4, Eq. lei and the normalisation
 * that bounds it).  For each partition p (a local batch B_l):
 *   rho_{p,e} = f_{p,e} / fbar(B_p) - 1 = f_{p,e} E / (K |B_p|) - 1,
 *   with c > 0: xi_p = max_e |rho_{p,e}| / c and rho~ = rho * tanh(xi_p)/xi_p
 *   (tanh(xi)/xi := 1 at xi = 0); with c <= 0: rho~ = rho (unnormalised LEI);
 *   inj[p,e] = eta * rho~_{p,e}, computed in binary64, rounded once to binary32.
 *   load [P,E] int32 (in); inj [P,E] binary32 (out, 16-byte aligned for
 *   eqb_lei_inject).  An empty partition gets inj = 0.  Unlike the other calls,
 *   T = 0 still writes inj (all zero).  NaN eta or c is EQB_ERR_INVALID_ARG.
 */
eqb_status eqb_lei_residual(const int32_t* load, int64_t T, int32_t K, int32_t E,
                            const int64_t* part_off, int32_t P, double eta, double c, float* inj,
                            void* stream);

/*
 * Load-Error Injection, the gradient correction (Sec. 4, Eq. lei):
 *   grad_s[t,e] += inj[p,e] for every token t of partition p, one binary32
 *   addition each (round to nearest even).  LEI leaves routing and mixture
 *   weights unchanged; only the router-score gradient moves.
 *   grad_s [T,E] binary32 (in/out, 16-byte aligned); inj [P,E] binary32 (in,
 *   16-byte aligned), e.g. from eqb_lei_residual.
 */
eqb_status eqb_lei_inject(float* grad_s, const float* inj, int64_t T, int32_t E,
                          const int64_t* part_off, int32_t P, void* stream);

/*
 * Router backward with Load-Error Injection, fused (Sec. 2 Eq. 1; Sec. 4 Eq. lei):
 *   grad_z[t,e] = (g[t,e] + inj[p,e]) * sigmoid'(z[t,e])    for t in partition p,
 *   where g[t,e] = grad_score[t,k] if e = topk_idx[t,k] (the gradient of the
 *   loss w.r.t. the mixture weight s_{t,e} of a selected expert) and 0 for the
 *   other experts; inj [P,E] from eqb_lei_residual, or NULL for the plain
 *   router backward.  sigmoid'(z) = e/(1+e)^2, e = exp(-|z|), in binary32
 *   (a few ulp); the sum and product are single binary32 operations.
 *   z [T,E] bf16 bits (16-byte aligned), topk_idx [T,K] int32, grad_score
 *   [T,K] binary32 (in); grad_z [T,E] binary32 (out, 16-byte aligned).
 *   Index entries outside [0, E) are ignored.
 */
eqb_status eqb_lei_router_backward(const uint16_t* z, const int32_t* topk_idx, const float* grad_score,
                                   const float* inj, int64_t T, int32_t E, int32_t K, const int64_t* part_off,
                                   int32_t P, float* grad_z, void* stream);

/*
 * One whole layer in one call (Sec. 2, Eq. 1 and "Quantile Balancing";
 * Appendix C, Algorithm 1 steps 1-6; Eq. 2): routing with the fused coarse
 * counts, the coarse selection, the fine counts and the fine selection with
 * the centred bias, enqueued as five kernels on `stream`.  It computes what
 * eqb_route_topk, eqb_select_quantile(1), eqb_margin_hist_pass2 and
 * eqb_select_quantile(2) compute in sequence, with r = eqb_rank(T, K, E).
 *   z [T,E] bf16 bits, b [E] binary32                       (in)
 *   topk_idx [T,K] int32, topk_score [T,K] binary32, tau [T] (out)
 *   load [P,E] int32                                         (out, WRITTEN: f_{p,e})
 *   q_bf16 [E] (out: b_hat_e, BF16 bits), b_next [E] binary32 (out: Eq. 2)
 *   hist_hi_sum, hist_lo_sum [E,256] int32 (nullable out): the summed coarse
 *     counts H[e,u] and the summed fine counts L[e,v] inside u_e.
 *   dev_status [1] int32 (out, WRITTEN): EQB_DEV_OK, or
 *     EQB_DEV_RANK_EXCEEDS_COUNT when some expert's selection failed.
 *   workspace: device memory of at least eqb_layer_workspace_size(E, P)
 *     bytes, 256-byte aligned, owned by the caller.  Its first
 *     eqb_layer_workspace_zero_bytes(E, P) bytes hold the per-partition
 *     counts and the selections while the layer runs: they must be ALL ZERO
 *     when the call's work starts, and the call's work leaves them all zero
 *     again (each selection clears the counts it has summed).  The rest is
 *     scratch for the fine pass's per-block count images, which every call
 *     overwrites before reading; its contents do not matter.  So a caller
 *     zeroes the workspace once after allocating it and may then run layer
 *     after layer with it.  After an error reported by the call or by the
 *     runtime while its work ran, zero it again before the next use.  Two
 *     calls whose work may overlap need two workspaces.
 *   marks (nullable): host array of 5 hipEvent_t handles, each nullable,
 *     recorded on `stream` before the route kernel, after it, after the
 *     coarse selection, after the fine pass and after the last kernel (for
 *     timing the stages of one layer without splitting the call).
 * Returns EQB_ERR_RANK when T = 0 (no quantile), EQB_ERR_INVALID_ARG for a
 * null pointer or a workspace that is too small, EQB_ERR_UNSUPPORTED for a
 * misaligned z or workspace; other errors as for the calls it chains.
 */
size_t eqb_layer_workspace_size(int32_t E, int32_t P);        /* host only; 0 for unsupported E or P */
size_t eqb_layer_workspace_zero_bytes(int32_t E, int32_t P);  /* host only; 0 for unsupported E or P */
eqb_status eqb_layer(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                     const int64_t* part_off, int32_t P, int32_t* topk_idx, float* topk_score, float* tau,
                     int32_t* load, uint16_t* q_bf16, float* b_next, int32_t* hist_hi_sum,
                     int32_t* hist_lo_sum, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                     void* const* marks, void* stream);

/*
 * eqb_layer for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same layer, the same outputs and argument checks, but the working buffers
 * live in a library-owned device array of EQB_NOALLOC_SCRATCH_BYTES per GPU
 * (held until the process ends) instead of a caller workspace.  The call
 * allocates nothing; the caller still passes every input and output.
 *   The array holds the layer's counters only (the fine pass adds its counts
 *   to the partition slabs instead of storing per-block images).
 *   Limit: eqb_layer_workspace_zero_bytes(E, P) <= EQB_NOALLOC_SCRATCH_BYTES,
 *   i.e. P * E <= 4096 (E = 256: up to 16 partitions); larger layers return
 *   EQB_ERR_SCRATCH before anything is enqueued.
 *   Every call on one GPU shares that GPU's array: the call clears the part
 *   it uses (a fill kernel) before the layer runs, and calls whose work may
 *   overlap on one GPU (other streams, other threads) race on it and give
 *   wrong results.  Order them on one stream.
 */
#define EQB_NOALLOC_SCRATCH_BYTES ((size_t)(8u << 20) + (192u << 10))
eqb_status eqb_layer_noalloc(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                             const int64_t* part_off, int32_t P, int32_t* topk_idx, float* topk_score,
                             float* tau, int32_t* load, uint16_t* q_bf16, float* b_next,
                             int32_t* hist_hi_sum, int32_t* hist_lo_sum, int32_t* dev_status, void* stream);

/*
 * Test control (host only, no HIP call): caps the number of blocks of the
 * streaming kernels (routing, the margin passes, the LEI kernels) at
 * max_blocks for the calls that follow FROM THE CALLING HOST THREAD; calls
 * made from other threads keep their own setting (the default 0: a whole
 * number of blocks per compute unit).  Results do not depend on it; tests
 * use it to run one block, or a block count that does not divide the rows,
 * against the same oracle.  Negative values are EQB_ERR_INVALID_ARG.
 * eqb_get_max_blocks returns the calling thread's current cap.
 */
eqb_status eqb_set_max_blocks(int32_t max_blocks);
int32_t eqb_get_max_blocks(void);

/* Host helper: r = ceil(T*K/E) (Sec. 3; the paper assumes T*K/E is an
 * integer), or -1 for invalid arguments.  Host only, no HIP call. */
int64_t eqb_rank(int64_t T_total, int32_t K, int32_t E);

/* Host helper: a static string naming a status code. */
const char* eqb_status_string(eqb_status status);

#ifdef __cplusplus
}
#endif

#endif /* EQB_H */
