// balance.hip - load-balance quantities computed from the expert loads:
// MaxVio (arXiv 2609.28053, Sec. 5 and Appendix E, "Balance metrics") and
// Load-Error Injection (Sec. 4, Eq. lei and its normalisation).
#include "eqb_internal.hpp"

namespace eqb {

// Maximum of f over the block (every thread receives it): within each wave,
// then over the waves.
__device__ __forceinline__ int64_t block_max_i64(int64_t f, int64_t* sh) {
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t o = (int64_t)__shfl_xor((unsigned long long)f, off);
    f = o > f ? o : f;
  }
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = f;
  __syncthreads();
  int64_t m = sh[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) m = sh[w] > m ? sh[w] : m;
  __syncthreads();
  return m;
}

// MaxVio = (max_e f_e) * E / (K * |B|) - 1 in binary64: the integer maximum
// is exact, the division and the subtraction round once each; NaN for an
// empty batch.
__device__ __forceinline__ double maxvio_of(int64_t m, int E, int K, int64_t n) {
  return n > 0 ? (double)(m * E) / ((double)K * (double)n) - 1.0 : __builtin_nan("");
}

// Block p < P: partition p alone; block P: the whole batch (loads summed over
// the partitions) and, with out_local_mean, the mean of the partitions'
// values over the non-empty partitions (Appendix E: Local MaxVio is computed
// per local batch and then averaged), a binary64 sum in ascending partition
// order divided by their number.
__global__ __launch_bounds__(kNBins) void max_violation_kernel(
    const int32_t* __restrict__ load, int E, int K, const PartTable pt,
    double* __restrict__ out_global, double* __restrict__ out_local, double* __restrict__ out_local_mean) {
  __shared__ int64_t sh_max[kNBins / 64];
  const int p = blockIdx.x;
  const int e = threadIdx.x;
  int64_t f = 0;
  if (e < E) {
    if (p < pt.P) {
      f = load[(int64_t)p * E + e];
    } else {
      for (int q = 0; q < pt.P; ++q) f += load[(int64_t)q * E + e];
    }
  }
  const int64_t m = block_max_i64(f, sh_max);
  const int64_t n = (p < pt.P) ? pt.off[p + 1] - pt.off[p] : pt.off[pt.P];
  if (p < pt.P) {
    if (e == 0 && out_local) out_local[p] = maxvio_of(m, E, K, n);
    return;
  }
  if (e == 0) *out_global = maxvio_of(m, E, K, n);
  if (out_local_mean == nullptr) return;
  double acc = 0.0;
  int count = 0;
  for (int q = 0; q < pt.P; ++q) {
    const int64_t nq = pt.off[q + 1] - pt.off[q];
    if (nq == 0) continue;            // block-uniform
    const int64_t mq = block_max_i64(e < E ? (int64_t)load[(int64_t)q * E + e] : 0, sh_max);
    acc += maxvio_of(mq, E, K, nq);
    ++count;
  }
  if (e == 0) *out_local_mean = count > 0 ? acc / (double)count : __builtin_nan("");
}

eqb_status launch_max_violation(const int32_t* load, int E, int K, const PartTable& pt,
                                double* out_global, double* out_local, double* out_local_mean, hipStream_t s) {
  max_violation_kernel<<<pt.P + 1, kNBins, 0, s>>>(load, E, K, pt, out_global, out_local, out_local_mean);
  return launch_status();
}

// ------------------------------------------------- Load-Error Injection --
// Block p: rho_e = f_{p,e} E / (K |B_p|) - 1 in binary64; with c > 0 the
// shared scale tanh(xi)/xi, xi = max_e |rho_e| / c (1 at xi = 0); the value
// injected into every score gradient of partition p is eta * (rho_e * scale),
// rounded once to binary32.  An empty partition injects 0.
__global__ __launch_bounds__(kNBins) void lei_residual_kernel(
    const int32_t* __restrict__ load, int E, int K, const PartTable pt, double eta, double c,
    float* __restrict__ inj) {
  __shared__ double sh_max[kNBins / 64];
  const int p = blockIdx.x;
  const int e = threadIdx.x;
  const int64_t n = pt.off[p + 1] - pt.off[p];
  double rho = 0.0;
  if (e < E && n > 0) rho = (double)((int64_t)load[(int64_t)p * E + e] * E) / ((double)K * (double)n) - 1.0;
  double a = fabs(rho);
  for (int off = 32; off > 0; off >>= 1) a = fmax(a, __shfl_xor(a, off));
  if ((e & 63) == 0) sh_max[e >> 6] = a;
  __syncthreads();
  double m = sh_max[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) m = fmax(m, sh_max[w]);
  double scale = 1.0;
  if (c > 0.0) {
    const double xi = m / c;
    if (xi > 0.0) scale = tanh(xi) / xi;
  }
  if (e < E) inj[(int64_t)p * E + e] = n > 0 ? (float)(eta * (rho * scale)) : 0.0f;
}

// grad_s[t,e] += inj[p(t),e], one binary32 addition per score.  G = E/4
// lanes cover a row with one 16-byte access each; every lane handles kLeiU
// rows per step, so that many loads are in flight before the first store.
constexpr int kLeiU = 4;

template <int E>
__global__ __launch_bounds__(kBlock) void lei_inject_kernel(
    float* __restrict__ grad, const float* __restrict__ inj, int64_t T, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 4;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R * kLeiU;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    const float4 d = *reinterpret_cast<const float4*>(inj + (int64_t)p * E + g * 4);
    for (int64_t base = s0; base < s1; base += ROWS) {
      float4 v[kLeiU];
#pragma unroll
      for (int u = 0; u < kLeiU; ++u) {
        const int64_t t = base + (int64_t)(u * kWaves + wave) * R + rr;
        if (t < s1) v[u] = *reinterpret_cast<const float4*>(grad + t * E + g * 4);
      }
#pragma unroll
      for (int u = 0; u < kLeiU; ++u) {
        const int64_t t = base + (int64_t)(u * kWaves + wave) * R + rr;
        if (t < s1) {
          const float4 o = make_float4(v[u].x + d.x, v[u].y + d.y, v[u].z + d.z, v[u].w + d.w);
          *reinterpret_cast<float4*>(grad + t * E + g * 4) = o;
        }
      }
    }
  });
}

// ------------------------------------- router backward with LEI ---------
// grad_z[t,e] = (g[t,e] + inj[p(t),e]) * sigmoid'(z[t,e]), where g[t,e] is
// grad_score[t,k] for e = topk_idx[t,k] and 0 for the other experts.  G = E/8
// lanes hold a row, 8 experts each (one 16-byte load of z, two of grad_z),
// and every lane works on kBwdU rows per step.  The K mixture gradients of a
// row are scattered into a per-wave LDS row (zeroed first) and read back 8 at
// a time.  With K <= G lane g of a row owns pair k = g, and the next step's
// logits and pairs are loaded while a step is processed; a larger K reads its
// pairs inside the step.
constexpr int kBwdU = 2;

template <int E>
__global__ __launch_bounds__(kBlock) void lei_router_backward_kernel(
    const uint16_t* __restrict__ z, const int32_t* __restrict__ topk_idx, const float* __restrict__ grad_score,
    const float* __restrict__ inj, int64_t T, int K, float* __restrict__ grad_z, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R * kBwdU;
  __shared__ __align__(16) float sh_g[kWaves][kBwdU][R][E];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  const bool one_pair = K <= G;
  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    float d[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] = inj ? inj[(int64_t)p * E + e0 + j] : 0.0f;
    auto row_of = [&](int64_t base, int u) -> int64_t { return base + (int64_t)(u * kWaves + wave) * R + rr; };
    // logits and this lane's pair of its rows at step base
    auto load = [&](int64_t base, uint4 (&zw)[kBwdU], int (&e)[kBwdU], float (&gv)[kBwdU]) {
#pragma unroll
      for (int u = 0; u < kBwdU; ++u) {
        const int64_t t = row_of(base, u);
        zw[u] = make_uint4(0, 0, 0, 0);
        e[u] = -1;
        gv[u] = 0.0f;
        if (t < s1) {
          zw[u] = *reinterpret_cast<const uint4*>(z + t * E + e0);
          if (one_pair && g < K) {
            e[u] = topk_idx[t * K + g];
            gv[u] = grad_score[t * K + g];
          }
        }
      }
    };
    uint4 zn[kBwdU];
    int en[kBwdU];
    float gn[kBwdU];
    load(s0, zn, en, gn);
    for (int64_t base = s0; base < s1; base += ROWS) {
      uint4 zw[kBwdU];
      int ec[kBwdU];
      float gc[kBwdU];
#pragma unroll
      for (int u = 0; u < kBwdU; ++u) {
        zw[u] = zn[u];
        ec[u] = en[u];
        gc[u] = gn[u];
      }
      if (base + ROWS < s1) load(base + ROWS, zn, en, gn);
      // scatter the rows' mixture gradients
#pragma unroll
      for (int u = 0; u < kBwdU; ++u) {
        float* myrow = sh_g[wave][u][rr];
        *reinterpret_cast<float4*>(myrow + e0) = make_float4(0.f, 0.f, 0.f, 0.f);
        *reinterpret_cast<float4*>(myrow + e0 + 4) = make_float4(0.f, 0.f, 0.f, 0.f);
      }
      lds_wave_sync();
#pragma unroll
      for (int u = 0; u < kBwdU; ++u) {
        const int64_t t = row_of(base, u);
        float* myrow = sh_g[wave][u][rr];
        if (t < s1) {
          if (one_pair) {
            if (ec[u] >= 0 && ec[u] < E) myrow[ec[u]] = gc[u];
          } else {
            for (int k = g; k < K; k += G) {
              const int e = topk_idx[t * K + k];
              if (e >= 0 && e < E) myrow[e] = grad_score[t * K + k];
            }
          }
        }
      }
      lds_wave_sync();
#pragma unroll
      for (int u = 0; u < kBwdU; ++u) {
        const int64_t t = row_of(base, u);
        const float* myrow = sh_g[wave][u][rr];
        const float4 ga = *reinterpret_cast<const float4*>(myrow + e0);
        const float4 gb = *reinterpret_cast<const float4*>(myrow + e0 + 4);
        const float gm[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
        const uint32_t w4[4] = {zw[u].x, zw[u].y, zw[u].z, zw[u].w};
        float o[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float zf = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
          o[j] = (gm[j] + d[j]) * sigmoid_prime_fast(zf);
        }
        if (t < s1) {
          *reinterpret_cast<float4*>(grad_z + t * E + e0) = make_float4(o[0], o[1], o[2], o[3]);
          *reinterpret_cast<float4*>(grad_z + t * E + e0 + 4) = make_float4(o[4], o[5], o[6], o[7]);
        }
      }
      lds_wave_sync();          // the row buffers are rewritten by the next step
    }
  });
}

template <int E>
static void launch_backward_e(const uint16_t* z, const int32_t* idx, const float* gs, const float* inj, int64_t T,
                              int K, float* gz, const PartTable& pt, hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, kWaves * (64 / (E / 8)) * kBwdU, 2, &blocks, &rpb);
  lei_router_backward_kernel<E><<<blocks, kBlock, 0, s>>>(z, idx, gs, inj, T, K, gz, pt, rpb);
}

eqb_status launch_lei_router_backward(const uint16_t* z, const int32_t* idx, const float* gs, const float* inj,
                                      int64_t T, int E, int K, float* gz, const PartTable& pt, hipStream_t s) {
  switch (E) {
    case 8: launch_backward_e<8>(z, idx, gs, inj, T, K, gz, pt, s); break;
    case 16: launch_backward_e<16>(z, idx, gs, inj, T, K, gz, pt, s); break;
    case 32: launch_backward_e<32>(z, idx, gs, inj, T, K, gz, pt, s); break;
    case 64: launch_backward_e<64>(z, idx, gs, inj, T, K, gz, pt, s); break;
    case 128: launch_backward_e<128>(z, idx, gs, inj, T, K, gz, pt, s); break;
    case 256: launch_backward_e<256>(z, idx, gs, inj, T, K, gz, pt, s); break;
    default: return EQB_ERR_UNSUPPORTED;
  }
  return launch_status();
}

eqb_status launch_lei_residual(const int32_t* load, int E, int K, const PartTable& pt, double eta,
                               double c, float* inj, hipStream_t s) {
  lei_residual_kernel<<<pt.P, kNBins, 0, s>>>(load, E, K, pt, eta, c, inj);
  return launch_status();
}

template <int E>
static void launch_inject_e(float* grad, const float* inj, int64_t T, const PartTable& pt, hipStream_t s) {
  int blocks;
  int64_t rpb;
  grid_for(T, kWaves * (64 / (E / 4)) * kLeiU, 2, &blocks, &rpb);
  lei_inject_kernel<E><<<blocks, kBlock, 0, s>>>(grad, inj, T, pt, rpb);
}

eqb_status launch_lei_inject(float* grad, const float* inj, int64_t T, int E, const PartTable& pt,
                             hipStream_t s) {
  switch (E) {
    case 8: launch_inject_e<8>(grad, inj, T, pt, s); break;
    case 16: launch_inject_e<16>(grad, inj, T, pt, s); break;
    case 32: launch_inject_e<32>(grad, inj, T, pt, s); break;
    case 64: launch_inject_e<64>(grad, inj, T, pt, s); break;
    case 128: launch_inject_e<128>(grad, inj, T, pt, s); break;
    case 256: launch_inject_e<256>(grad, inj, T, pt, s); break;
    default: return EQB_ERR_UNSUPPORTED;
  }
  return launch_status();
}

}  // namespace eqb
