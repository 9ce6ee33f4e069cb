// eqb_device.hpp - device helpers shared by the gfx950 kernels of libeqb.
//
// Method: arXiv 2609.28053 (Exact Quantile Balancing), Sec. 2-3 and
// Algorithm 1 of Appendix C.  Nothing in here is exported.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "eqb.h"

namespace eqb {

constexpr int kNBins = 256;
constexpr int kBlock = 1024;            // threads of a streaming block
constexpr int kWaves = kBlock / 64;
constexpr int64_t kSegMax = 65535;      // rows per LDS histogram flush (16-bit counters)
constexpr int kHistStride = kNBins + 1; // LDS words per expert pair (odd stride spreads banks)

// Contiguous token partitions [off[p], off[p+1]), passed by value.  nsub:
// count slabs per partition (1 for the entry points that write a caller's
// [P,E,256] counts; the one-call layer spreads a partition's blocks over
// several slabs of its workspace, summed by the selections).
struct PartTable {
  int64_t off[EQB_MAX_PARTITIONS + 1];
  int32_t P;
  int32_t nsub = 1;
  // Claim counters of the partitions' dynamic tails (one int32 per
  // partition, 256 bytes apart, zero at launch), or null: see block_plan.
  int32_t* pool = nullptr;
  // Coarse count slabs of 16-bit counters (the layer's route sweep, where no
  // slab can receive more than 65,535 rows): slab [E/2][256][2], the counters
  // of experts 2m and 2m+1 for kappa bin k side by side at (m*256 + k)*2,
  // in the first half of the slab's int32 space.
  int32_t slab16 = 0;
};

// The [E,256] count slab that this block adds partition p's counts to: with
// nsub slabs per partition, block b uses slab b % nsub, so that fewer blocks
// add to each counter (the flushes' global atomics on one address
// serialise).
__device__ __forceinline__ int32_t* count_slab(int32_t* hist, const PartTable& pt, int p, int E) {
  const int sub = pt.nsub > 1 ? (int)(blockIdx.x % (unsigned)pt.nsub) : 0;
  return hist + ((int64_t)p * pt.nsub + sub) * E * kNBins;
}

// ------------------------------------------------------------ BF16 ------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Raw high byte of bf16_rne(x) from the binary32 bits of x.  Round-half-up
// and round-half-even only differ on an exact tie with an even last BF16 bit,
// and then the carry cannot reach bit 24, so adding 0x8000 is exact here.
__device__ __forceinline__ uint32_t bf16_raw_hi(uint32_t bits) { return (bits + 0x8000u) >> 24; }

// kappa maps BF16 bits to an order-preserving key: negative patterns flip
// every bit, non-negative ones only the sign.  On the raw high byte hr this
// is hr ^ 0xFF (sign set) or hr ^ 0x80; on the raw low byte lr it is lr ^ 0xFF
// for negative values and lr otherwise.
__device__ __forceinline__ int kappa_hi_of_raw(int hr) { return hr ^ ((hr & 0x80) ? 0xFF : 0x80); }
__device__ __forceinline__ int raw_hi_of_kappa(int u) { return u ^ ((u & 0x80) ? 0x80 : 0xFF); }

__device__ __forceinline__ uint16_t kappa_inv(uint32_t key) {
  return (uint16_t)((key & 0x8000u) ? (key ^ 0x8000u) : (key ^ 0xFFFFu));
}

__device__ __forceinline__ float sigmoid_f32(float x) {
  if (x >= 0.0f) return 1.0f / (1.0f + expf(-x));
  const float ex = expf(x);
  return ex / (1.0f + ex);
}

// sigmoid(x) = 1 / (1 + e) for x >= 0 and e / (1 + e) for x < 0, with
// e = exp(-|x|) = 2^(-|x| log2 e).  The product |x| log2 e is carried as
// p_hi + p_lo (log2 e split into two binary32 parts, the rounding error of
// the leading product recovered with an fma), 2^(-p_hi) comes from the
// hardware exponential and 2^(-p_lo) ~ 1 - p_lo ln 2 corrects it.  Relative
// error stays within a few ulp for |x| <= 64; larger |x| use the libm path.
__device__ __forceinline__ float sigmoid_fast(float x) {
  const float a = fabsf(x);
  if (a > 64.0f) return sigmoid_f32(x);
  const float kLog2eHi = 1.44269502162933349609375f;   // binary32 nearest to log2(e)
  const float kLog2eLo = 1.925963033500011e-08f;       // log2(e) - kLog2eHi
  const float kLn2 = 0.693147180559945309f;
  const float p_hi = a * kLog2eHi;
  const float p_lo = __builtin_fmaf(a, kLog2eLo, __builtin_fmaf(a, kLog2eHi, -p_hi));
  const float e1 = __builtin_amdgcn_exp2f(-p_hi);
  const float e = __builtin_fmaf(-e1, p_lo * kLn2, e1);
  const float r = __builtin_amdgcn_rcpf(1.0f + e);
  return x >= 0.0f ? r : e * r;
}

// sigmoid'(x) = e / (1 + e)^2 with e = exp(-|x|) (the form that keeps its
// relative accuracy for large |x|), e from the same split base-2 exponential
// as sigmoid_fast; a few ulp for |x| <= 64, the libm exponential beyond.
__device__ __forceinline__ float sigmoid_prime_fast(float x) {
  const float a = fabsf(x);
  float e;
  if (a > 64.0f) {
    e = expf(-a);
  } else {
    const float kLog2eHi = 1.44269502162933349609375f;
    const float kLog2eLo = 1.925963033500011e-08f;
    const float kLn2 = 0.693147180559945309f;
    const float p_hi = a * kLog2eHi;
    const float p_lo = __builtin_fmaf(a, kLog2eLo, __builtin_fmaf(a, kLog2eHi, -p_hi));
    const float e1 = __builtin_amdgcn_exp2f(-p_hi);
    e = __builtin_fmaf(-e1, p_lo * kLn2, e1);
  }
  const float r = 1.0f / (1.0f + e);
  return e * r * r;
}

// ------------------------------------------------------- exact 64-bit keys --
// Unsigned key ordered like the binary32 value, with -0 and +0 equal.
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
  u = (u == 0x80000000u) ? 0u : u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint32_t order_key_inv(uint32_t k) {
  return (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
}
// Exact candidate key: high word = order key of s; low word = (255-e) << 24 |
// (s is -0) << 16 | BF16 bits of z.  Unique per row; larger = better rank;
// equal scores favour the lower expert index.
__device__ __forceinline__ uint64_t exact_key(uint32_t sbits, int e, uint32_t zbits) {
  const uint32_t lo = ((uint32_t)(255 - e) << 24) | ((sbits == 0x80000000u) ? (1u << 16) : 0u) | zbits;
  return ((uint64_t)order_key(sbits) << 32) | lo;
}
__device__ __forceinline__ int exact_key_expert(uint64_t k) { return 255 - (int)((uint32_t)k >> 24); }
__device__ __forceinline__ uint32_t exact_key_z(uint64_t k) { return (uint32_t)k & 0xFFFFu; }
__device__ __forceinline__ uint32_t exact_key_sbits(uint64_t k) {
  if ((uint32_t)k & (1u << 16)) return 0x80000000u;
  return order_key_inv((uint32_t)(k >> 32));
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  const uint32_t lo = __shfl_xor((unsigned int)v, mask);
  const uint32_t hi = __shfl_xor((unsigned int)(v >> 32), mask);
  return ((uint64_t)hi << 32) | lo;
}

// ------------------------------------------------ group reductions (DPP) --
// Maximum over aligned groups of G lanes (G = 1, 2, 4, 8 or 16); every lane
// of the group receives it.  quad_perm swaps within quads, the half-row and
// row mirrors pair the two halves of 8- and 16-lane groups.
template <int G>
__device__ __forceinline__ int group_max_i32(int x) {
  if constexpr (G >= 2) x = max(x, __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));
  if constexpr (G >= 4) x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));
  if constexpr (G >= 8) x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false));
  if constexpr (G >= 16) x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false));
  static_assert(G <= 16, "group reductions cover at most 16 lanes");
  return x;
}

template <int G>
__device__ __forceinline__ uint64_t group_max_u64(uint64_t m) {
#pragma unroll
  for (int off = 1; off < G; off <<= 1) {
    const uint64_t o = shfl_xor_u64(m, off);
    m = o > m ? o : m;
  }
  return m;
}

__device__ __forceinline__ int med3_i32(int a, int b, int c) {
  int r;
  asm volatile("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// ------------------------------------------------------- float keys --
// Routing keys are binary32 bit patterns kept in int registers and ordered
// as floats.  A key is finite or the sentinel -inf, never NaN, and the keys
// of one row never include both +0 and -0, so the float order is a strict
// total order on them whatever their signs.  Maximum and median are written
// as the instructions themselves: the compiler's IEEE-mode maximum would
// first quieten both operands with an extra instruction each.  They are
// per-lane functions of their operands, so the asm is not volatile and the
// compiler may schedule loads across it.
constexpr int kKeyNone = (int)0xFF800000u;   // -inf: below every key
constexpr int kKeyTop = (int)0x7F800000u;    // +inf: above every key

__device__ __forceinline__ int key_max(int a, int b) {
  int r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ int key_med3(int a, int b, int c) {
  int r;
  asm("v_med3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ bool key_lt(int a, int b) { return __int_as_float(a) < __int_as_float(b); }

// Float maximum of the keys over aligned groups of G lanes, one DPP maximum
// per level as in group_max_i32.  Built without IEEE mode (the routing
// kernels are), each level compiles to one v_max_f32_dpp, and the compiler
// places the DPP wait states itself, filling them with independent work
// where it can.
template <int G>
__device__ __forceinline__ int group_max_key(int x) {
  float f = __int_as_float(x);
  if constexpr (G >= 2) f = fmaxf(f, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(f), 0xB1, 0xF, 0xF, false)));
  if constexpr (G >= 4) f = fmaxf(f, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(f), 0x4E, 0xF, 0xF, false)));
  if constexpr (G >= 8) f = fmaxf(f, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(f), 0x141, 0xF, 0xF, false)));
  if constexpr (G >= 16) f = fmaxf(f, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(f), 0x140, 0xF, 0xF, false)));
  static_assert(G <= 16, "group reductions cover at most 16 lanes");
  return __float_as_int(f);
}

// Value of lane S of every aligned group of G lanes (G = 1, 2, 4 or 8), by
// DPP: a quad broadcast, and for G = 8 the other quad's copy through the
// half-row mirror.
template <int G, int S>
__device__ __forceinline__ float group_bcast(float x, int g) {
  static_assert(G <= 8 && S >= 0 && S < G, "group broadcast covers at most 8 lanes");
  if constexpr (G == 1) {
    return x;
  } else {
    constexpr int s = S & 3;
    constexpr int sel = G == 2 ? (s | s << 2 | (2 + s) << 4 | (2 + s) << 6) : s * 0x55;
    const int y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), sel, 0xF, 0xF, false);
    if constexpr (G <= 4) {
      return __int_as_float(y);
    } else {
      const int m = __builtin_amdgcn_update_dpp(0, y, 0x141, 0xF, 0xF, false);
      return __int_as_float(((g >> 2) == (S >> 2)) ? y : m);
    }
  }
}

// ------------------------------------------------ per-expert selection --
// Inclusive scan of one count per thread over a 256-thread block: a scan
// inside each wave, then the totals of the lower waves.  Counts and their
// sums stay below 2^31 (T < 2^31).
__device__ __forceinline__ int64_t block_inclusive_scan_256(int64_t x64, int64_t* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = (int)x64;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int lower = 0;
  for (int w = 0; w < wave; ++w) lower += (int)sh[w];
  return (int64_t)(x + lower);
}

// Sum over the P slabs of one counter; the loads are issued eight at a time
// so that their latencies overlap.
__device__ __forceinline__ int64_t slab_sum(const int32_t* __restrict__ hist, int P, int64_t stride) {
  int64_t c = 0;
  int q = 0;
  for (; q + 8 <= P; q += 8) {
    int v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = hist[(q + j) * stride];
#pragma unroll
    for (int j = 0; j < 8; ++j) c += v[j];
  }
  for (; q < P; ++q) c += hist[q * stride];
  return c;
}

// Zeroes the P slabs of one counter (the layer form's consume-and-clear).
__device__ __forceinline__ void slab_clear(int32_t* __restrict__ hist, int P, int64_t stride) {
  for (int q = 0; q < P; ++q) hist[q * stride] = 0;
}

// ------------------------------------------------------- partition walk --
// Calls f(p, s0, s1) for every piece of [r0, r1) lying in one partition and
// holding at most kSegMax rows.  Uniform across the block.
template <class F>
__device__ __forceinline__ void for_each_segment(int64_t r0, int64_t r1, const PartTable& pt, F&& f,
                                                 int64_t seg_max = kSegMax) {
  int p = 0;
  int64_t t = r0;
  while (t < r1) {
    while (p < pt.P - 1 && pt.off[p + 1] <= t) ++p;
    int64_t end = pt.off[p + 1] < r1 ? pt.off[p + 1] : r1;
    if (end - t > seg_max) end = t + seg_max;
    f(p, t, end);
    t = end;
  }
}

// The same pieces in reverse order (last rows first).
template <class F>
__device__ __forceinline__ void for_each_segment_rev(int64_t r0, int64_t r1, const PartTable& pt, F&& f,
                                                     int64_t seg_max = kSegMax) {
  int p = pt.P - 1;
  int64_t t = r1;
  while (t > r0) {
    while (p > 0 && pt.off[p] >= t) --p;
    int64_t start = pt.off[p] > r0 ? pt.off[p] : r0;
    if (t - start > seg_max) start = t - seg_max;
    f(p, start, t);
    t = start;
  }
}

// ------------------------------------------- packed LDS histograms -------
// Counters of experts 2m (low half) and 2m+1 (high half) share one 32-bit
// word at m * kHistStride + bin.  Bins are RAW BF16 bytes; the flush maps them
// to kappa bins.
template <int E>
constexpr int hist_words() { return (E / 2) * kHistStride; }

// Flush order: the i-th word a block visits when it adds its LDS counts to
// global memory.  Blocks start at different words (a stride per block that
// is not a multiple of the bank count), so that blocks flushing at the same
// time add to different global counters instead of queueing on one address.
__device__ __forceinline__ int flush_word(int i, int nwords) {
  int w = i + (int)((blockIdx.x * 1031u) % (uint32_t)nwords);
  return w >= nwords ? w - nwords : w;
}

// Adds n_lo to counter c[0] and n_hi to c[1] (two adjacent int32 counters):
// one 64-bit atomic when c is 8-byte aligned, else two 32-bit ones.  The
// 64-bit add is exact because no count reaches 2^31, so the low word never
// carries into the high one.
__device__ __forceinline__ void add_count_pair(int32_t* c, uint32_t n_lo, uint32_t n_hi) {
  if ((reinterpret_cast<uintptr_t>(c) & 7u) == 0) {
    atomicAdd(reinterpret_cast<unsigned long long*>(c),
              (unsigned long long)n_lo | ((unsigned long long)n_hi << 32));
  } else {
    if (n_lo) atomicAdd(c, (int32_t)n_lo);
    if (n_hi) atomicAdd(c + 1, (int32_t)n_hi);
  }
}

// Adds the counts of raw bins 2j (n_even) and 2j+1 (n_odd) of expert e to
// its row of kappa bins.  Both raw bins of a pair map to two adjacent kappa
// bins: in order when the map keeps the low bit (XOR 0x80, or no change for
// a fine bin of a non-negative selection), swapped when it flips every bit
// (XOR 0xFF).
__device__ __forceinline__ void add_raw_pair(int32_t* row, bool flips, uint32_t n_even, uint32_t n_odd,
                                             int kappa_even) {
  if (!flips) add_count_pair(row + kappa_even, n_even, n_odd);
  else add_count_pair(row + (kappa_even - 1), n_odd, n_even);
}

// Adds a block's packed LDS counts to global slab [E][256] (kappa bins) and
// clears them, one pair of adjacent raw bins per thread and step.
// kFine = false: raw high byte -> kappa high byte (same map for every expert).
// kFine = true : raw low byte  -> kappa low byte, flipped for experts whose
//                selected coarse bin holds negative values (u_e < 0x80);
//                experts without a valid selection are skipped.
template <int E, bool kFine>
__device__ __forceinline__ void flush_hist(uint32_t* sh, int32_t* __restrict__ slab,
                                           const int32_t* __restrict__ sel_hi) {
  constexpr int kItems = (E / 2) * (kNBins / 2);
  for (int i = threadIdx.x; i < kItems; i += blockDim.x) {
    const int it = flush_word(i, kItems);
    const int pair = it / (kNBins / 2), j = it % (kNBins / 2);
    const int w0 = pair * kHistStride + 2 * j;
    const uint32_t c0 = sh[w0], c1 = sh[w0 + 1];
    if (c0 | c1) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint32_t n0 = h ? (c0 >> 16) : (c0 & 0xFFFFu);
        const uint32_t n1 = h ? (c1 >> 16) : (c1 & 0xFFFFu);
        const int e = 2 * pair + h;
        if (n0 | n1) {
          if (kFine) {
            const int u = sel_hi[e];
            if (u >= 0 && u < kNBins) {
              const bool neg = u < 0x80;
              add_raw_pair(slab + e * kNBins, neg, n0, n1, neg ? (2 * j) ^ 0xFF : 2 * j);
            }
          } else {
            const bool neg = (2 * j) & 0x80;
            add_raw_pair(slab + e * kNBins, neg, n0, n1, kappa_hi_of_raw(2 * j));
          }
        }
      }
      sh[w0] = 0;
      sh[w0 + 1] = 0;
    }
  }
}

// Word offset of expert e's row in a packed histogram and its increment.
__device__ __forceinline__ uint32_t hist_row(int e) { return (uint32_t)(e >> 1) * kHistStride; }
__device__ __forceinline__ uint32_t hist_inc(int e) { return 1u << ((e & 1) * 16); }

// Rows handled by block blockIdx.x.
// A 64-bit value every lane of the wave holds, moved to scalar registers.
// Offsets of segment bases pass through it, so that the compiler knows the
// bases are wave-uniform: loads and stores then take a 64-bit scalar base
// next to a 32-bit vector offset instead of a 64-bit address per lane.
__device__ __forceinline__ int64_t wave_uniform(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void block_rows(int64_t T, int64_t rows_per_block, int64_t* r0, int64_t* r1) {
  *r0 = (int64_t)blockIdx.x * rows_per_block;
  *r1 = (*r0 + rows_per_block < T) ? *r0 + rows_per_block : T;
}

// Dynamic tails (the one-call layer's route sweep).  Compute units do not
// sweep at one speed (the blocks of a launch finish up to ~5% apart), so a
// static split waits for the slowest.  With pt.pool set, the blocks of a
// launch are dealt out to the partitions in proportion to their rows (block
// b serves partition p when floor(nb off[p] / T) <= b < floor(nb off[p+1] /
// T); the host checks that every non-empty partition gets a block), and a
// partition's blocks form groups of at most kGroupBlocks, each taking a share
// of the partition's rows in proportion to its blocks.  A group keeps the
// last 1/kPoolDiv of its rows (at most kPoolMax) as a pool and splits the rest
// into contiguous static ranges, one per block; once a wave has finished its
// block's range it claims pool chunks from the group's counter until none is
// left.  Groups keep the claims on one counter few.  Static ranges are
// flushed every kSegPool rows, so a block's last static segment plus any pool
// rows it takes stay below the 16-bit LDS counters' limit.  Groups of 8 with
// half their rows pooled (at most 49,152: a large workload's group of 8 keeps
// 37.5% back and its blocks' 10,240-row static ranges stay one segment)
// measured 2-3.5% faster per step than groups of 16 pooling an eighth
// (4,194,304 tokens), and 1-2% at 1.5-2 M tokens; groups of 4, and pools of
// a quarter or a third, fell in between.
constexpr int64_t kPoolMax = 49152;
constexpr int64_t kPoolDiv = 2;
constexpr int kGroupBlocks = 8;
constexpr int64_t kSegPool = kSegMax - kPoolMax;
// A group's claim counter is indexed by the group's first block and sits on
// its own 128-byte line; pool mode is used for grids of at most
// kPoolCounters blocks.
constexpr int kPoolStride = 32;
constexpr int kPoolCounters = 1024;

struct BlockPlan {
  int64_t r0, r1;     // the block's static rows
  int64_t q0, q1;     // its group's pool (pool mode)
  int p;              // the partition served (pool mode), else -1
  int ctr;            // its group's counter (pool mode)
  bool pool;
};

inline __host__ __device__ int64_t pool_block_start(const PartTable& pt, int64_t T, int64_t nb, int p) {
  return nb * pt.off[p] / T;
}

__device__ __forceinline__ BlockPlan block_plan(const PartTable& pt, int64_t T, int64_t rows_per_block) {
  BlockPlan w;
  w.p = -1;
  w.ctr = 0;
  w.q0 = w.q1 = 0;
  w.pool = pt.pool != nullptr;
  if (!w.pool) {
    block_rows(T, rows_per_block, &w.r0, &w.r1);
    return w;
  }
  const int64_t nb = gridDim.x, b = blockIdx.x;
  // block b serves p when nb off[p] < (b + 1) T <= nb off[p+1]
  int p = 0;
  while (p < pt.P - 1 && nb * pt.off[p + 1] < (b + 1) * T) ++p;
  const int64_t b0 = pool_block_start(pt, T, nb, p), m = pool_block_start(pt, T, nb, p + 1) - b0;
  const int64_t n = pt.off[p + 1] - pt.off[p], i = b - b0;
  const int64_t gb0 = (i / kGroupBlocks) * kGroupBlocks;
  const int64_t gb1 = gb0 + kGroupBlocks < m ? gb0 + kGroupBlocks : m;
  const int64_t g0 = pt.off[p] + n * gb0 / m, g1 = pt.off[p] + n * gb1 / m;   // the group's rows
  const int64_t gn = g1 - g0, q = gn / kPoolDiv < kPoolMax ? gn / kPoolDiv : kPoolMax;
  const int64_t s = gn - q, j = i - gb0, mg = gb1 - gb0;
  w.p = p;
  w.ctr = (int)(b0 + gb0);
  w.r0 = g0 + s * j / mg;
  w.r1 = g0 + s * (j + 1) / mg;
  w.q0 = g0 + s;
  w.q1 = g1;
  return w;
}

}  // namespace eqb

namespace eqb {
// Orders this wave's LDS writes before its later LDS reads by other lanes.
__device__ __forceinline__ void lds_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}
}  // namespace eqb

namespace eqb {
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));
// Both values rounded to BF16 (nearest, ties to even) in one conversion; the
// first lands in bits 0..15, the second in bits 16..31.
__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  const float2_t f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
}  // namespace eqb
