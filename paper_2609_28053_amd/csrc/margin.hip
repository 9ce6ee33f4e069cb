// margin.hip - coarse and fine counts of the BF16 margins tau_t - z_{t,e}
// (Algorithm 1, steps 1 and 4 of arXiv 2609.28053, Appendix C) and the
// expert loads f_e (Sec. 2) from stored Top-K indices.
//
// Each lane holds 8 experts of a row (one 16-byte load); G = E/8 lanes cover a
// row and every lane works on U rows per step, so U loads are in flight
// before any arithmetic.  Counts go to packed LDS histograms indexed by the
// raw BF16 byte; the flush maps them to kappa bins.
#include "eqb_internal.hpp"

namespace eqb {

constexpr int kMarginU = 4;   // rows per lane per block step

template <int E, bool kFine>
__global__ __launch_bounds__(kBlock) void margin_hist_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ tau, int64_t T,
    const int32_t* __restrict__ sel_hi, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R * kMarginU;
  __shared__ uint32_t sh_hist[hist_words<E>()];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  // Fine pass: a margin is counted when the high byte of its rounded BF16
  // pattern equals the raw form U of u_e.  With y = bits + lsb + (0x7FFF - (U << 24)),
  // that holds exactly when y < 2^24 (unsigned), and bits 16..23 of y are then
  // the raw low byte of the rounded pattern.
  uint32_t cfine[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    int u = kFine ? sel_hi[e0 + j] : 0;
    u = (u >= 0 && u < kNBins) ? u : 0;   // invalid selections are skipped at the flush
    cfine[j] = 0x7FFFu - ((uint32_t)raw_hi_of_kappa(u) << 24);
  }
  for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) sh_hist[w] = 0;
  __syncthreads();

  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t base = s0; base < s1; base += ROWS) {
      uint4 v[kMarginU];
      float tv[kMarginU];
      bool ok[kMarginU];
#pragma unroll
      for (int u = 0; u < kMarginU; ++u) {
        const int64_t t = base + (int64_t)(u * kWaves + wave) * R + rr;
        ok[u] = t < s1;
        v[u] = make_uint4(0, 0, 0, 0);
        tv[u] = 0.0f;
        if (ok[u]) {
          v[u] = *reinterpret_cast<const uint4*>(z + t * E + e0);
          tv[u] = tau[t];
        }
      }
#pragma unroll
      for (int u = 0; u < kMarginU; ++u) {
        if (!ok[u]) continue;
        const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float zf = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
          const uint32_t bits = __float_as_uint(tv[u] - zf);
          const uint32_t row = hist_row(e0 + j);
          if (!kFine) {
            atomicAdd(&sh_hist[row + bf16_raw_hi(bits)], hist_inc(j));
          } else {
            const uint32_t y = bits + ((bits >> 16) & 1u) + cfine[j];
            if (y < (1u << 24)) atomicAdd(&sh_hist[row + ((y >> 16) & 0xFFu)], hist_inc(j));
          }
        }
      }
    }
    __syncthreads();
    int32_t* slab = hist + (int64_t)p * E * kNBins;
    if (!kFine) {
      flush_hist<E, false>(sh_hist, slab, nullptr);
    } else {
      // skip experts whose selection is invalid
      for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) {
        const uint32_t c = sh_hist[w];
        if (c) {
          const int pair = w / kHistStride;
          const int lr = w - pair * kHistStride;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t n = h ? (c >> 16) : (c & 0xFFFFu);
            const int e = 2 * pair + h;
            const int u = sel_hi[e];
            if (n && u >= 0 && u < kNBins)
              atomicAdd(slab + e * kNBins + ((u < 0x80) ? (lr ^ 0xFF) : lr), (int32_t)n);
          }
          sh_hist[w] = 0;
        }
      }
    }
    __syncthreads();
  });
}

template <int E>
eqb_status launch_margin_e(bool fine, const MarginArgs& a, hipStream_t s) {
  int blocks;
  int64_t rpb;
  const int rows_per_step = kWaves * (64 / (E / 8)) * kMarginU;
  grid_for(a.T, rows_per_step, hist_words<E>() * 4 * 2 <= 160 * 1024 ? 2 : 1, &blocks, &rpb);
  if (fine)
    margin_hist_kernel<E, true><<<blocks, kBlock, 0, s>>>(a.z, a.tau, a.T, a.sel_hi, a.hist, a.pt, rpb);
  else
    margin_hist_kernel<E, false><<<blocks, kBlock, 0, s>>>(a.z, a.tau, a.T, a.sel_hi, a.hist, a.pt, rpb);
  return launch_status();
}

eqb_status launch_margin(bool fine, const MarginArgs& a, hipStream_t s) {
  switch (a.E) {
    case 8: return launch_margin_e<8>(fine, a, s);
    case 16: return launch_margin_e<16>(fine, a, s);
    case 32: return launch_margin_e<32>(fine, a, s);
    case 64: return launch_margin_e<64>(fine, a, s);
    case 128: return launch_margin_e<128>(fine, a, s);
    case 256: return launch_margin_e<256>(fine, a, s);
    default: return EQB_ERR_UNSUPPORTED;
  }
}

// ------------------------------------------------------------ expert load --
__global__ __launch_bounds__(kBlock) void expert_load_kernel(
    const int32_t* __restrict__ topk_idx, int64_t T, int K, int E, int32_t* __restrict__ load,
    const PartTable pt, int64_t rows_per_block) {
  __shared__ uint32_t sh[kNBins];
  for (int e = threadIdx.x; e < kNBins; e += kBlock) sh[e] = 0;
  __syncthreads();
  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
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

eqb_status launch_load(const int32_t* idx, int64_t T, int K, int E, int32_t* load, const PartTable& pt,
                       hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, kBlock / 4, 2, &blocks, &rpb);
  expert_load_kernel<<<blocks, kBlock, 0, s>>>(idx, T, K, E, load, pt, rpb);
  return launch_status();
}

}  // namespace eqb
