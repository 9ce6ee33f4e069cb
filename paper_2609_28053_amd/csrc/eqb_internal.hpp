// eqb_internal.hpp - launch interfaces between the C ABI shim and the kernels.
#pragma once

#include "eqb_device.hpp"

namespace eqb {

struct RouteArgs {
  const uint16_t* z;
  const float* b;
  int64_t T;
  int E, K;
  int32_t* idx;
  float* score;
  float* tau;
  int32_t* load;
  int32_t* hist;
  PartTable pt;
};

struct MarginArgs {
  const uint16_t* z;
  const float* tau;
  int64_t T;
  int E;
  const int32_t* sel_hi;   // fine pass only
  int sel_stride = 0;      // 0: one selection for all partitions; E: one per partition
  int32_t* hist;
  PartTable pt;
};

eqb_status launch_route(const RouteArgs& a, hipStream_t s);
eqb_status launch_margin(bool fine, const MarginArgs& a, hipStream_t s);
eqb_status launch_load(const int32_t* idx, int64_t T, int K, int E, int32_t* load, const PartTable& pt,
                       hipStream_t s);
eqb_status launch_select(int pass, const int32_t* hist, int P, int E, int64_t r, int32_t* sel_hi,
                         int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                         int32_t* hist_sum, int32_t* status, hipStream_t s);

eqb_status launch_select_local(int pass, const int32_t* hist, int E, int K, const PartTable& pt,
                               int32_t* sel_hi, int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16,
                               int32_t* status, hipStream_t s);
eqb_status launch_rank_average(const uint16_t* q_bf16, int E, const PartTable& pt, double* b_avg,
                               float* b_next, hipStream_t s);
eqb_status launch_uniform_hist(const uint16_t* z, const float* tau, int64_t T, int E, const PartTable& pt,
                               float lo, float scale, int nbins, int32_t* hist, hipStream_t s);
eqb_status launch_select_uniform(const int32_t* hist, int P, int E, int nbins, int64_t r, double lo,
                                 double width, double* est, float* b_next, int32_t* status, hipStream_t s);
eqb_status launch_max_violation(const int32_t* load, int E, int K, const PartTable& pt,
                                double* out_global, double* out_local, hipStream_t s);

eqb_status launch_lei_residual(const int32_t* load, int E, int K, const PartTable& pt, double eta,
                               double c, float* inj, hipStream_t s);
eqb_status launch_lei_router_backward(const uint16_t* z, const int32_t* idx, const float* gs, const float* inj,
                                      int64_t T, int E, int K, float* gz, const PartTable& pt, hipStream_t s);
eqb_status launch_lei_inject(float* grad, const float* inj, int64_t T, int E, const PartTable& pt,
                             hipStream_t s);

// Number of compute units of the current device (cached per device).
int num_cus();

// Upper bound on the grid of the streaming kernels set by eqb_set_max_blocks
// (0: none).
int max_blocks_cap();

// Blocks and rows per block for a streaming kernel over T rows that advances
// rows_per_step rows per block step: at most blocks_per_cu blocks per CU,
// each owning a contiguous range of ceil(T / blocks) rows (the last may be
// shorter), and at least min_steps steps per block where T allows (a
// block's fixed costs, zeroing and flushing its LDS counts, then pay for
// more rows).  The ranges are not rounded to whole steps: with P equal
// partitions and a block count that P divides, every partition boundary
// then falls on a block boundary, and no block pays for a second segment
// (a second flush and a cold restart of its prefetch).
inline void grid_for(int64_t T, int rows_per_step, int blocks_per_cu, int* blocks, int64_t* rows_per_block,
                     int min_steps = 1) {
  int64_t max_blocks = (int64_t)num_cus() * blocks_per_cu;
  const int cap = max_blocks_cap();
  if (cap > 0 && cap < max_blocks) max_blocks = cap;
  const int64_t steps = (T + rows_per_step - 1) / rows_per_step;
  const int64_t want = (steps + min_steps - 1) / min_steps;
  int64_t nb = want < max_blocks ? want : max_blocks;
  if (nb < 1) nb = 1;
  *rows_per_block = T > 0 ? (T + nb - 1) / nb : 1;
  *blocks = (int)((T + *rows_per_block - 1) / *rows_per_block);
  if (*blocks < 1) *blocks = 1;
}

inline eqb_status launch_status() { return hipGetLastError() == hipSuccess ? EQB_OK : EQB_ERR_HIP; }

}  // namespace eqb
