// eqb.hip - gfx950 kernels and C ABI for one MoE layer's routing and Exact
// Quantile Balancing statistics (arXiv 2609.28053, Sec. 2-3, Appendix C).
//
// Data path (one layer, one stream):
//   route_hist1  : z, b -> Top-K indices, sigmoid scores, tau, loads, and the
//                  coarse counts H_p (Algorithm 1 step 1) in the same sweep.
//   select (1)   : sum of the P slabs (all-reduce stand-in), u_e, rho_e.
//   margin_hist  : z, tau, u -> fine counts L_p (Algorithm 1 step 4).
//   select (2)   : v_e, b_hat_e = kappa^-1(u_e, v_e), centred bias (Eq. 2).
//
// Streaming kernels use 1024-thread blocks, each owning a contiguous range of
// rows.  A row of E BF16 logits is spread over G = E/8 lanes, 8 experts (one
// 16-byte load) per lane.  Per-block histograms live in LDS as two 16-bit
// counters per 32-bit word (bins 2i and 2i+1 of one expert), so E*256 bins
// take E*512 bytes; a block flushes them with global atomics at every
// partition boundary and at least every 65535 rows, so no 16-bit counter
// can overflow.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "eqb.h"

namespace {

constexpr int kNBins = 256;
constexpr int kBlock = 1024;
constexpr int kWaves = kBlock / 64;
constexpr int64_t kSegMax = 65535;

struct PartTable {
  int64_t off[EQB_MAX_PARTITIONS + 1];
  int32_t P;
};

// ---------------------------------------------------------------- helpers --
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Unsigned key ordered like the binary32 value, with -0 and +0 equal.
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
  u = (u == 0x80000000u) ? 0u : u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint32_t order_key_inv(uint32_t k) {
  return (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
}

// kappa(bf16_rne(tau - zf)): the binary32 difference rounded to the nearest
// BF16 (ties to even) by integer arithmetic on the bit pattern (exact for
// finite values, subnormals included), then the order-preserving 16-bit key.
__device__ __forceinline__ uint32_t margin_key(float tau, float zf) {
  const uint32_t m = __float_as_uint(tau - zf);
  const uint32_t r = (m + 0x7FFFu + ((m >> 16) & 1u)) >> 16;
  return r ^ ((r & 0x8000u) ? 0xFFFFu : 0x8000u);
}

__device__ __forceinline__ uint16_t kappa_inv(uint32_t key) {
  return (uint16_t)((key & 0x8000u) ? (key ^ 0x8000u) : (key ^ 0xFFFFu));
}

__device__ __forceinline__ float sigmoid_f32(float x) {
  if (x >= 0.0f) return 1.0f / (1.0f + expf(-x));
  const float ex = expf(x);
  return ex / (1.0f + ex);
}

// Top-K candidate key: high word = order key of s, low word = (255 - e) << 24
// | (s is -0) << 16 | BF16 bits of z.  Keys are unique per row (distinct e);
// a larger key is a better rank, and equal scores favour the lower index.
__device__ __forceinline__ uint64_t cand_key(float s, int e, uint32_t zbits) {
  const uint32_t sb = __float_as_uint(s);
  const uint32_t lo = ((uint32_t)(255 - e) << 24) | ((sb == 0x80000000u) ? (1u << 16) : 0u) | zbits;
  return ((uint64_t)order_key(sb) << 32) | lo;
}

__device__ __forceinline__ int cand_expert(uint64_t k) { return 255 - (int)((uint32_t)k >> 24); }
__device__ __forceinline__ float cand_z(uint64_t k) { return __uint_as_float(((uint32_t)k & 0xFFFFu) << 16); }
__device__ __forceinline__ float cand_s(uint64_t k) {
  if ((uint32_t)k & (1u << 16)) return __uint_as_float(0x80000000u);
  return __uint_as_float(order_key_inv((uint32_t)(k >> 32)));
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  const uint32_t lo = __shfl_xor((unsigned int)v, mask);
  const uint32_t hi = __shfl_xor((unsigned int)(v >> 32), mask);
  return ((uint64_t)hi << 32) | lo;
}

// Calls f(p, s0, s1) for every piece of [r0, r1) that lies in one partition
// and holds at most kSegMax rows.  Uniform across the block.
template <class F>
__device__ __forceinline__ void for_each_segment(int64_t r0, int64_t r1, const PartTable& pt, F&& f) {
  int p = 0;
  int64_t t = r0;
  while (t < r1) {
    while (p < pt.P - 1 && pt.off[p + 1] <= t) ++p;
    int64_t end = pt.off[p + 1] < r1 ? pt.off[p + 1] : r1;
    if (end - t > kSegMax) end = t + kSegMax;
    f(p, t, end);
    t = end;
  }
}

// Adds the packed LDS histogram (word = (bin >> 1) * E + e) into the global
// slab [E][256] and clears it.  Caller synchronises before and after.
template <int E>
__device__ __forceinline__ void flush_hist(uint32_t* sh, int32_t* __restrict__ slab) {
  for (int w = threadIdx.x; w < (kNBins / 2) * E; w += blockDim.x) {
    const uint32_t c = sh[w];
    if (c) {
      const int pair = w / E, e = w % E;
      int32_t* dst = slab + e * kNBins + 2 * pair;
      if (c & 0xFFFFu) atomicAdd(dst, (int32_t)(c & 0xFFFFu));
      if (c >> 16) atomicAdd(dst + 1, (int32_t)(c >> 16));
      sh[w] = 0;
    }
  }
}

__device__ __forceinline__ void lds_count(uint32_t* sh, int E, int bin, int e) {
  atomicAdd(&sh[(bin >> 1) * E + e], 1u << ((bin & 1) * 16));
}

// ------------------------------------------------------ route + coarse pass --
template <int E>
__global__ __launch_bounds__(kBlock) void route_hist1_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ b, int64_t T, int K,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_score, float* __restrict__ tau,
    int32_t* __restrict__ load, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 8;           // lanes per row
  constexpr int R = 64 / G;          // rows per wave
  constexpr int ROWS = kWaves * R;   // rows per block step
  __shared__ uint32_t sh_hist[(kNBins / 2) * E];
  __shared__ uint32_t sh_load[E];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  float bb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) bb[j] = b[e0 + j];
  for (int w = threadIdx.x; w < (kNBins / 2) * E; w += kBlock) sh_hist[w] = 0;
  for (int w = threadIdx.x; w < E; w += kBlock) sh_load[w] = 0;
  __syncthreads();

  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = (r0 + rows_per_block < T) ? r0 + rows_per_block : T;

  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t base = s0; base < s1; base += ROWS) {
      const int64_t t = base + wave * R + rr;
      const bool valid = t < s1;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (valid) v = *reinterpret_cast<const uint4*>(z + t * E + e0);
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
      float zf[8];
      uint64_t key[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t zb = (j & 1) ? (w4[j >> 1] >> 16) : (w4[j >> 1] & 0xFFFFu);
        zf[j] = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
        key[j] = cand_key(zf[j] + bb[j], e0 + j, zb);
      }
      // K+1 rounds: each round takes the largest key below the previous one.
      uint64_t prev = ~0ull;
      for (int k = 0; k <= K; ++k) {
        uint64_t m = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) m = (key[j] < prev && key[j] > m) ? key[j] : m;
#pragma unroll
        for (int off = 1; off < G; off <<= 1) {
          const uint64_t o = shfl_xor_u64(m, off);
          m = o > m ? o : m;
        }
        prev = m;
        if (k < K && valid && g == k % G) {
          const int e = cand_expert(m);   // in [0, E) because the row holds E > K distinct keys
          topk_idx[t * K + k] = e;
          topk_score[t * K + k] = sigmoid_f32(cand_z(m));
          if (load && e >= 0 && e < E) atomicAdd(&sh_load[e], 1u);
        }
      }
      const float tv = cand_s(prev);
      if (valid && g == 0) tau[t] = tv;
      if (hist && valid) {
#pragma unroll
        for (int j = 0; j < 8; ++j) lds_count(sh_hist, E, (int)(margin_key(tv, zf[j]) >> 8), e0 + j);
      }
    }
    __syncthreads();
    if (hist) flush_hist<E>(sh_hist, hist + (int64_t)p * E * kNBins);
    if (load) {
      for (int e = threadIdx.x; e < E; e += kBlock) {
        const uint32_t c = sh_load[e];
        if (c) atomicAdd(&load[(int64_t)p * E + e], (int32_t)c);
        sh_load[e] = 0;
      }
    }
    __syncthreads();
  });
}

// ------------------------------------------------- coarse or fine pass alone --
template <int E, bool kFine>
__global__ __launch_bounds__(kBlock) void margin_hist_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ tau, int64_t T,
    const int32_t* __restrict__ sel_hi, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R;
  __shared__ uint32_t sh_hist[(kNBins / 2) * E];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  int uu[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) uu[j] = kFine ? sel_hi[e0 + j] : 0;
  for (int w = threadIdx.x; w < (kNBins / 2) * E; w += kBlock) sh_hist[w] = 0;
  __syncthreads();

  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = (r0 + rows_per_block < T) ? r0 + rows_per_block : T;

  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t base = s0; base < s1; base += ROWS) {
      const int64_t t = base + wave * R + rr;
      if (t < s1) {
        const uint4 v = *reinterpret_cast<const uint4*>(z + t * E + e0);
        const float tv = tau[t];
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float zf = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
          const uint32_t key = margin_key(tv, zf);
          if (!kFine) {
            lds_count(sh_hist, E, (int)(key >> 8), e0 + j);
          } else if ((int)(key >> 8) == uu[j]) {
            lds_count(sh_hist, E, (int)(key & 0xFFu), e0 + j);
          }
        }
      }
    }
    __syncthreads();
    flush_hist<E>(sh_hist, hist + (int64_t)p * E * kNBins);
    __syncthreads();
  });
}

// ------------------------------------------------------------- expert load --
__global__ __launch_bounds__(kBlock) void expert_load_kernel(
    const int32_t* __restrict__ topk_idx, int64_t T, int K, int E, int32_t* __restrict__ load,
    const PartTable pt, int64_t rows_per_block) {
  __shared__ uint32_t sh[256];
  for (int e = threadIdx.x; e < 256; e += kBlock) sh[e] = 0;
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = (r0 + rows_per_block < T) ? r0 + rows_per_block : T;
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t i = s0 * K + threadIdx.x; i < s1 * K; i += kBlock) {
      const int e = topk_idx[i];
      if (e >= 0 && e < E) atomicAdd(&sh[e], 1u);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kBlock) {
      const uint32_t c = sh[e];
      if (c) atomicAdd(&load[(int64_t)p * E + e], (int32_t)c);
      sh[e] = 0;
    }
    __syncthreads();
  });
}

// ---------------------------------------------------------------- select --
// One block per expert, one thread per bin: sum the P slabs, inclusive scan,
// and pick the first bin whose cumulative count reaches the target rank.
__device__ __forceinline__ int64_t block_inclusive_scan_256(int64_t x, int64_t* sh) {
  const int i = threadIdx.x;
  sh[i] = x;
  __syncthreads();
  for (int d = 1; d < kNBins; d <<= 1) {
    const int64_t add = (i >= d) ? sh[i - d] : 0;
    __syncthreads();
    sh[i] += add;
    __syncthreads();
  }
  return sh[i];
}

__global__ __launch_bounds__(kNBins) void select_coarse_kernel(
    const int32_t* __restrict__ hist, int P, int E, int64_t r, int32_t* __restrict__ sel_hi,
    int64_t* __restrict__ rank_in_bin, int32_t* __restrict__ hist_sum, int32_t* __restrict__ status) {
  __shared__ int64_t sh[kNBins];
  const int e = blockIdx.x, u = threadIdx.x;
  int64_t c = 0;
  for (int p = 0; p < P; ++p) c += hist[((int64_t)p * E + e) * kNBins + u];
  if (hist_sum) hist_sum[(int64_t)e * kNBins + u] = (int32_t)c;
  const int64_t cum = block_inclusive_scan_256(c, sh);
  if (cum >= r && cum - c < r) {
    sel_hi[e] = u;
    rank_in_bin[e] = r - (cum - c);
  }
  if (u == kNBins - 1 && cum < r) {
    sel_hi[e] = -1;
    rank_in_bin[e] = 0;
    if (status) *status = EQB_DEV_RANK_EXCEEDS_COUNT;
  }
}

__global__ __launch_bounds__(kNBins) void select_fine_kernel(
    const int32_t* __restrict__ hist, int P, int E, const int32_t* __restrict__ sel_hi,
    const int64_t* __restrict__ rank_in_bin, int32_t* __restrict__ sel_lo,
    uint16_t* __restrict__ q_bf16, int32_t* __restrict__ hist_sum, int32_t* __restrict__ status) {
  __shared__ int64_t sh[kNBins];
  const int e = blockIdx.x, v = threadIdx.x;
  int64_t c = 0;
  for (int p = 0; p < P; ++p) c += hist[((int64_t)p * E + e) * kNBins + v];
  if (hist_sum) hist_sum[(int64_t)e * kNBins + v] = (int32_t)c;
  const int64_t cum = block_inclusive_scan_256(c, sh);
  const int u = sel_hi[e];
  const int64_t rho = rank_in_bin[e];
  const bool ok = u >= 0 && u < kNBins && rho >= 1;
  if (ok && cum >= rho && cum - c < rho) {
    sel_lo[e] = v;
    q_bf16[e] = kappa_inv(((uint32_t)u << 8) | (uint32_t)v);
  }
  if (v == kNBins - 1 && (!ok || cum < rho)) {
    sel_lo[e] = -1;
    q_bf16[e] = 0x7FC0;
    if (status) *status = EQB_DEV_RANK_EXCEEDS_COUNT;
  }
}

// b = b_hat - mean(b_hat): binary64 sum in ascending expert order, one rounding.
__global__ __launch_bounds__(256) void center_kernel(const uint16_t* __restrict__ q, int E,
                                                     float* __restrict__ b_next) {
  __shared__ double mean;
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int e = 0; e < E; ++e) acc += (double)__uint_as_float((uint32_t)q[e] << 16);
    mean = acc / (double)E;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x)
    b_next[e] = (float)((double)__uint_as_float((uint32_t)q[e] << 16) - mean);
}

// ------------------------------------------------------------- host side --
bool supported_E(int32_t E) {
  return E == 8 || E == 16 || E == 32 || E == 64 || E == 128 || E == 256;
}

eqb_status make_table(const int64_t* part_off, int32_t P, int64_t T, PartTable* pt) {
  if (part_off == nullptr) {
    if (P != 1) return EQB_ERR_INVALID_ARG;
    pt->P = 1;
    pt->off[0] = 0;
    pt->off[1] = T;
    return EQB_OK;
  }
  if (P < 1 || P > EQB_MAX_PARTITIONS) return EQB_ERR_INVALID_ARG;
  if (part_off[0] != 0 || part_off[P] != T) return EQB_ERR_INVALID_ARG;
  for (int p = 0; p < P; ++p)
    if (part_off[p + 1] < part_off[p]) return EQB_ERR_INVALID_ARG;
  pt->P = P;
  for (int p = 0; p <= P; ++p) pt->off[p] = part_off[p];
  return EQB_OK;
}

int num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Blocks and rows per block for a streaming kernel over T rows.
void grid_for(int64_t T, int rows_per_step, int blocks_per_cu, int* blocks, int64_t* rows_per_block) {
  const int64_t max_blocks = (int64_t)num_cus() * blocks_per_cu;
  int64_t steps = (T + rows_per_step - 1) / rows_per_step;
  int64_t nb = steps < max_blocks ? steps : max_blocks;
  if (nb < 1) nb = 1;
  const int64_t steps_per_block = (steps + nb - 1) / nb;
  *rows_per_block = steps_per_block * rows_per_step;
  *blocks = (int)((T + *rows_per_block - 1) / *rows_per_block);
}

template <int E>
constexpr int rows_per_step() { return kWaves * (64 / (E / 8)); }

template <int E>
constexpr int hist_blocks_per_cu() { return (E * 512 + 1024) * 2 <= 160 * 1024 ? 2 : 1; }

eqb_status launch_status() { return hipGetLastError() == hipSuccess ? EQB_OK : EQB_ERR_HIP; }

template <int E>
eqb_status launch_route(const uint16_t* z, const float* b, int64_t T, int K, int32_t* idx, float* score,
                        float* tau, int32_t* load, int32_t* hist, const PartTable& pt, hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, rows_per_step<E>(), hist_blocks_per_cu<E>(), &blocks, &rpb);
  route_hist1_kernel<E><<<blocks, kBlock, 0, s>>>(z, b, T, K, idx, score, tau, load, hist, pt, rpb);
  return launch_status();
}

template <int E>
eqb_status launch_margin(bool fine, const uint16_t* z, const float* tau, int64_t T, const int32_t* sel_hi,
                         int32_t* hist, const PartTable& pt, hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, rows_per_step<E>(), hist_blocks_per_cu<E>(), &blocks, &rpb);
  if (fine)
    margin_hist_kernel<E, true><<<blocks, kBlock, 0, s>>>(z, tau, T, sel_hi, hist, pt, rpb);
  else
    margin_hist_kernel<E, false><<<blocks, kBlock, 0, s>>>(z, tau, T, sel_hi, hist, pt, rpb);
  return launch_status();
}

}  // namespace

extern "C" {

eqb_status eqb_route_topk(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                          int32_t* topk_idx, float* topk_score, float* tau,
                          const int64_t* part_off, int32_t P,
                          int32_t* load, int32_t* hist_hi, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !b || !topk_idx || !topk_score || !tau) return EQB_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(z) % 16 != 0) return EQB_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
#define ROUTE_CALL(EE) launch_route<EE>(z, b, T, K, topk_idx, topk_score, tau, load, hist_hi, pt, s)
  switch (E) {
    case 8: return ROUTE_CALL(8);
    case 16: return ROUTE_CALL(16);
    case 32: return ROUTE_CALL(32);
    case 64: return ROUTE_CALL(64);
    case 128: return ROUTE_CALL(128);
    case 256: return ROUTE_CALL(256);
    default: return EQB_ERR_UNSUPPORTED;
  }
#undef ROUTE_CALL
}

static eqb_status margin_pass(bool fine, const uint16_t* z, const float* tau, int64_t T, int32_t E,
                              const int32_t* sel_hi, const int64_t* part_off, int32_t P, int32_t* hist,
                              void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !tau || !hist || (fine && !sel_hi)) return EQB_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(z) % 16 != 0) return EQB_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
#define MARGIN_CALL(EE) launch_margin<EE>(fine, z, tau, T, sel_hi, hist, pt, s)
  switch (E) {
    case 8: return MARGIN_CALL(8);
    case 16: return MARGIN_CALL(16);
    case 32: return MARGIN_CALL(32);
    case 64: return MARGIN_CALL(64);
    case 128: return MARGIN_CALL(128);
    case 256: return MARGIN_CALL(256);
    default: return EQB_ERR_UNSUPPORTED;
  }
#undef MARGIN_CALL
}

eqb_status eqb_margin_hist_pass1(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                 const int64_t* part_off, int32_t P, int32_t* hist_hi, void* stream) {
  return margin_pass(false, z, tau, T, E, nullptr, part_off, P, hist_hi, stream);
}

eqb_status eqb_margin_hist_pass2(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                 const int32_t* sel_hi, const int64_t* part_off, int32_t P,
                                 int32_t* hist_lo, void* stream) {
  return margin_pass(true, z, tau, T, E, sel_hi, part_off, P, hist_lo, stream);
}

eqb_status eqb_select_quantile(int32_t pass, const int32_t* hist, int32_t P, int32_t E, int64_t r,
                               int32_t* sel_hi, int64_t* rank_in_bin,
                               int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                               int32_t* hist_sum, int32_t* dev_status, void* stream) {
  if (pass != 1 && pass != 2) return EQB_ERR_INVALID_ARG;
  if (P < 1 || P > EQB_MAX_PARTITIONS) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  if (r < 1 || r > INT32_MAX) return EQB_ERR_RANK;
  if (!hist || !sel_hi || !rank_in_bin) return EQB_ERR_INVALID_ARG;
  if (pass == 2 && (!sel_lo || !q_bf16)) return EQB_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (pass == 1) {
    select_coarse_kernel<<<E, kNBins, 0, s>>>(hist, P, E, r, sel_hi, rank_in_bin, hist_sum, dev_status);
    return launch_status();
  }
  select_fine_kernel<<<E, kNBins, 0, s>>>(hist, P, E, sel_hi, rank_in_bin, sel_lo, q_bf16, hist_sum,
                                          dev_status);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  if (b_next) {
    center_kernel<<<1, 256, 0, s>>>(q_bf16, E, b_next);
    return launch_status();
  }
  return EQB_OK;
}

eqb_status eqb_expert_load(const int32_t* topk_idx, int64_t T, int32_t K, int32_t E,
                           const int64_t* part_off, int32_t P, int32_t* load, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!topk_idx || !load) return EQB_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int blocks;
  int64_t rpb;
  grid_for(T, kBlock / 4, 2, &blocks, &rpb);
  expert_load_kernel<<<blocks, kBlock, 0, s>>>(topk_idx, T, K, E, load, pt, rpb);
  return launch_status();
}

int64_t eqb_rank(int64_t T_total, int32_t K, int32_t E) {
  if (T_total < 0 || E < 1 || K < 1 || K >= E) return -1;
  if (T_total > (int64_t)1 << 40) return -1;
  return (T_total * (int64_t)K + E - 1) / E;
}

const char* eqb_status_string(eqb_status status) {
  switch (status) {
    case EQB_OK: return "EQB_OK";
    case EQB_ERR_INVALID_ARG: return "EQB_ERR_INVALID_ARG";
    case EQB_ERR_UNSUPPORTED: return "EQB_ERR_UNSUPPORTED";
    case EQB_ERR_RANK: return "EQB_ERR_RANK";
    case EQB_ERR_HIP: return "EQB_ERR_HIP";
    default: return "EQB_ERR_UNKNOWN";
  }
}

}  // extern "C"
