// select.hip - selection steps of Algorithm 1 (arXiv 2609.28053, Appendix C):
// the all-reduce stand-in (sum of the P partition slabs), the coarse choice
// u_e, rho_e (step 3), the fine choice v_e and b_hat_e = kappa^-1(u_e, v_e)
// (steps 5-6), and the centred bias of Eq. 2.
#include "eqb_internal.hpp"

namespace eqb {

// Inclusive scan of one value per thread over a 256-thread block.
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

// One block per expert, one thread per bin.
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

// b = b_hat - mean(b_hat): binary64 sum in ascending expert order, divided by
// E, difference in binary64, one rounding to binary32.
__global__ __launch_bounds__(256) void center_kernel(const uint16_t* __restrict__ q, int E,
                                                     float* __restrict__ b_next) {
  __shared__ double val[256];
  __shared__ double mean;
  for (int e = threadIdx.x; e < E; e += blockDim.x) val[e] = (double)__uint_as_float((uint32_t)q[e] << 16);
  __syncthreads();
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int e = 0; e < E; ++e) acc += val[e];
    mean = acc / (double)E;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) b_next[e] = (float)(val[e] - mean);
}

eqb_status launch_select(int pass, const int32_t* hist, int P, int E, int64_t r, int32_t* sel_hi,
                         int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                         int32_t* hist_sum, int32_t* status, hipStream_t s) {
  if (pass == 1) {
    select_coarse_kernel<<<E, kNBins, 0, s>>>(hist, P, E, r, sel_hi, rank_in_bin, hist_sum, status);
    return launch_status();
  }
  select_fine_kernel<<<E, kNBins, 0, s>>>(hist, P, E, sel_hi, rank_in_bin, sel_lo, q_bf16, hist_sum, status);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  if (b_next) {
    center_kernel<<<1, 256, 0, s>>>(q_bf16, E, b_next);
    return launch_status();
  }
  return EQB_OK;
}

}  // namespace eqb
