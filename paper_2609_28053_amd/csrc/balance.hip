// balance.hip - load-balance quantities computed from the expert loads:
// MaxVio (arXiv 2609.28053, Sec. 5 and Appendix E, "Balance metrics").
#include "eqb_internal.hpp"

namespace eqb {

// Block p < P: partition p alone; block P: the whole batch (loads summed over
// the partitions).  MaxVio = (max_e f_e) * E / (K * |B|) - 1 in binary64: the
// integer maximum is exact, the division and the subtraction round once each.
__global__ __launch_bounds__(kNBins) void max_violation_kernel(
    const int32_t* __restrict__ load, int E, int K, const PartTable pt,
    double* __restrict__ out_global, double* __restrict__ out_local) {
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
  // maximum over the block: within each wave, then over the waves
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t o = (int64_t)__shfl_xor((unsigned long long)f, off);
    f = o > f ? o : f;
  }
  if ((e & 63) == 0) sh_max[e >> 6] = f;
  __syncthreads();
  if (e == 0) {
    int64_t m = sh_max[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) m = sh_max[w] > m ? sh_max[w] : m;
    const int64_t n = (p < pt.P) ? pt.off[p + 1] - pt.off[p] : pt.off[pt.P];
    const double v = n > 0 ? (double)(m * E) / ((double)K * (double)n) - 1.0 : __builtin_nan("");
    if (p < pt.P) {
      if (out_local) out_local[p] = v;
    } else {
      *out_global = v;
    }
  }
}

eqb_status launch_max_violation(const int32_t* load, int E, int K, const PartTable& pt,
                                double* out_global, double* out_local, hipStream_t s) {
  max_violation_kernel<<<pt.P + 1, kNBins, 0, s>>>(load, E, K, pt, out_global, out_local);
  return launch_status();
}

}  // namespace eqb
