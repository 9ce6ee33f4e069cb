// variants.hip - the two distributed QB statistics that EQB is compared with
// (arXiv 2609.28053, Sec. 2 after Eq. 2, and Sec. 3):
//  * rank-averaged QB: every shard's own K/E quantile (exact, by the same two
//    passes run per partition), averaged over the shards;
//  * fixed-resolution histogram QB: margin counts over fixed uniform bins,
//    summed over the shards, and the quantile read off the summed histogram.
#include "eqb_internal.hpp"

namespace eqb {

// Binary64 mean of the values, ascending order, then v - mean rounded once to
// binary32 (the centring of Eq. 2).  One block; E <= 256.
__device__ __forceinline__ void centre_block(double* val, int E, float* b_next) {
  __shared__ double mean;
  __syncthreads();
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int e = 0; e < E; ++e) acc += val[e];
    mean = acc / (double)E;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) b_next[e] = (float)(val[e] - mean);
}

// Average of the shards' quantiles over the non-empty shards (binary64 sum in
// ascending p, divided by their number), then centred.
__global__ __launch_bounds__(256) void rank_average_kernel(const uint16_t* __restrict__ q, int E,
                                                           const PartTable pt, double* __restrict__ b_avg,
                                                           float* __restrict__ b_next) {
  __shared__ double val[256];
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    double acc = 0.0;
    int n = 0;
    for (int p = 0; p < pt.P; ++p) {
      if (pt.off[p + 1] == pt.off[p]) continue;
      acc += (double)__uint_as_float((uint32_t)q[(int64_t)p * E + e] << 16);
      ++n;
    }
    val[e] = n > 0 ? acc / (double)n : __builtin_nan("");
    if (b_avg) b_avg[e] = val[e];
  }
  centre_block(val, E, b_next);
}

eqb_status launch_rank_average(const uint16_t* q_bf16, int E, const PartTable& pt, double* b_avg,
                               float* b_next, hipStream_t s) {
  rank_average_kernel<<<1, 256, 0, s>>>(q_bf16, E, pt, b_avg, b_next);
  return launch_status();
}

// Counts of the binary32 margins tau - z over nbins uniform bins:
// bin = floor((m - lo) * scale) clamped to [0, nbins - 1], computed in
// binary32.  Layout and flush as in the coarse pass (bins < 256), without the
// kappa map.
template <int E>
__global__ __launch_bounds__(kBlock) void uniform_hist_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ tau, int64_t T, float lo, float scale,
    int nbins, int32_t* __restrict__ hist, const PartTable pt, int64_t rows_per_block) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int U = 4;
  constexpr int ROWS = kWaves * R * U;
  __shared__ uint32_t sh_hist[hist_words<E>()];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  const uint32_t row0 = hist_row(e0);
  const float top = (float)(nbins - 1);
  for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) sh_hist[w] = 0;
  __syncthreads();
  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t base = s0; base < s1; base += ROWS) {
      uint4 v[U];
      float tv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t t = base + (int64_t)(u * kWaves + wave) * R + rr;
        v[u] = make_uint4(0, 0, 0, 0);
        tv[u] = 0.0f;
        if (t < s1) {
          v[u] = *reinterpret_cast<const uint4*>(z + t * E + e0);
          tv[u] = tau[t];
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t t = base + (int64_t)(u * kWaves + wave) * R + rr;
        if (t >= s1) continue;
        const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float zf = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
          float x = ((tv[u] - zf) - lo) * scale;
          x = fminf(fmaxf(x, 0.0f), top);        // in [0, nbins-1]: truncation is the floor
          atomicAdd(&sh_hist[row0 + (j >> 1) * kHistStride + (uint32_t)(int)x], hist_inc(j));
        }
      }
    }
    __syncthreads();
    int32_t* slab = hist + (int64_t)p * E * nbins;
    for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) {
      const uint32_t c = sh_hist[w];
      if (c) {
        const int pair = w / kHistStride;
        const int bin = w - pair * kHistStride;
        if (c & 0xFFFFu) atomicAdd(slab + (2 * pair) * nbins + bin, (int32_t)(c & 0xFFFFu));
        if (c >> 16) atomicAdd(slab + (2 * pair + 1) * nbins + bin, (int32_t)(c >> 16));
        sh_hist[w] = 0;
      }
    }
    __syncthreads();
  });
}

template <int E>
static void launch_uniform_e(const uint16_t* z, const float* tau, int64_t T, const PartTable& pt, float lo,
                             float scale, int nbins, int32_t* hist, hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, kWaves * (64 / (E / 8)) * 4, hist_words<E>() * 4 * 2 <= 160 * 1024 ? 2 : 1, &blocks, &rpb);
  uniform_hist_kernel<E><<<blocks, kBlock, 0, s>>>(z, tau, T, lo, scale, nbins, hist, pt, rpb);
}

eqb_status launch_uniform_hist(const uint16_t* z, const float* tau, int64_t T, int E, const PartTable& pt,
                               float lo, float scale, int nbins, int32_t* hist, hipStream_t s) {
  switch (E) {
    case 8: launch_uniform_e<8>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    case 16: launch_uniform_e<16>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    case 32: launch_uniform_e<32>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    case 64: launch_uniform_e<64>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    case 128: launch_uniform_e<128>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    case 256: launch_uniform_e<256>(z, tau, T, pt, lo, scale, nbins, hist, s); break;
    default: return EQB_ERR_UNSUPPORTED;
  }
  return launch_status();
}

// One block per expert, one thread per bin: sum the slabs, scan, and read the
// r-th smallest as lo + (j + (r - C_{j-1}) / H_j) * width in binary64, j the
// first bin whose running count reaches r.
__global__ __launch_bounds__(kNBins) void select_uniform_kernel(
    const int32_t* __restrict__ hist, int P, int E, int nbins, int64_t r, double lo, double width,
    double* __restrict__ est, int32_t* __restrict__ status) {
  __shared__ int64_t sh[kNBins];
  const int e = blockIdx.x, j = threadIdx.x;
  const int64_t c = (j < nbins) ? slab_sum(hist + (int64_t)e * nbins + j, P, (int64_t)E * nbins) : 0;
  const int64_t cum = block_inclusive_scan_256(c, sh);
  if (c > 0 && cum >= r && cum - c < r)
    est[e] = lo + ((double)j + (double)(r - (cum - c)) / (double)c) * width;
  if (j == kNBins - 1 && cum < r) {
    est[e] = __builtin_nan("");
    if (status) *status = EQB_DEV_RANK_EXCEEDS_COUNT;
  }
}

__global__ __launch_bounds__(256) void centre64_kernel(const double* __restrict__ est, int E,
                                                       float* __restrict__ b_next) {
  __shared__ double val[256];
  for (int e = threadIdx.x; e < E; e += blockDim.x) val[e] = est[e];
  centre_block(val, E, b_next);
}

eqb_status launch_select_uniform(const int32_t* hist, int P, int E, int nbins, int64_t r, double lo,
                                 double width, double* est, float* b_next, int32_t* status, hipStream_t s) {
  select_uniform_kernel<<<E, kNBins, 0, s>>>(hist, P, E, nbins, r, lo, width, est, status);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  if (b_next) {
    centre64_kernel<<<1, 256, 0, s>>>(est, E, b_next);
    return launch_status();
  }
  return EQB_OK;
}

}  // namespace eqb
