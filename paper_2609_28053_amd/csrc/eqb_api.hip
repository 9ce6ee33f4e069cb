// eqb_api.hip - the C ABI declared in include/eqb.h.  Every argument check
// runs before anything is enqueued; the calls never synchronise the host.
#include <atomic>

#include "eqb_internal.hpp"

namespace eqb {

// Compute units per device, queried once per device.  Concurrent first
// calls may both query; they store the same value.
int num_cus() {
  static std::atomic<int> cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

namespace {
// Grid cap of eqb_set_max_blocks: per host thread, so a cap one caller sets
// never changes the grids of calls made from other threads.
thread_local int t_max_blocks = 0;
}  // namespace

int max_blocks_cap() { return t_max_blocks; }

namespace {

bool supported_E(int32_t E) { return E == 8 || E == 16 || E == 32 || E == 64 || E == 128 || E == 256; }

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

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

}  // namespace
}  // namespace eqb

using namespace eqb;

extern "C" {

eqb_status eqb_route_topk(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                          int32_t* topk_idx, float* topk_score, float* tau,
                          const int64_t* part_off, int32_t P,
                          int32_t* load, int32_t* hist_hi, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  RouteArgs a;
  const eqb_status st = make_table(part_off, P, T, &a.pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !b || !topk_idx || !topk_score || !tau) return EQB_ERR_INVALID_ARG;
  if (!aligned16(z)) return EQB_ERR_UNSUPPORTED;
  a.z = z;
  a.b = b;
  a.T = T;
  a.E = E;
  a.K = K;
  a.idx = topk_idx;
  a.score = topk_score;
  a.tau = tau;
  a.load = load;
  a.hist = hist_hi;
  return launch_route(a, static_cast<hipStream_t>(stream));
}

static eqb_status margin_pass(bool fine, const uint16_t* z, const float* tau, int64_t T, int32_t E,
                              const int32_t* sel_hi, const int64_t* part_off, int32_t P, int32_t* hist,
                              void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  MarginArgs a;
  const eqb_status st = make_table(part_off, P, T, &a.pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !tau || !hist || (fine && !sel_hi)) return EQB_ERR_INVALID_ARG;
  if (!aligned16(z)) return EQB_ERR_UNSUPPORTED;
  a.z = z;
  a.tau = tau;
  a.T = T;
  a.E = E;
  a.sel_hi = sel_hi;
  a.hist = hist;
  return launch_margin(fine, a, static_cast<hipStream_t>(stream));
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
  return launch_select(pass, hist, P, E, r, sel_hi, rank_in_bin, sel_lo, q_bf16, b_next, hist_sum,
                       dev_status, static_cast<hipStream_t>(stream));
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
  return launch_load(topk_idx, T, K, E, load, pt, static_cast<hipStream_t>(stream));
}

eqb_status eqb_select_quantile_local(int32_t pass, const int32_t* hist, int64_t T, int32_t K, int32_t E,
                                     const int64_t* part_off, int32_t P, int32_t* sel_hi,
                                     int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16,
                                     int32_t* dev_status, void* stream) {
  if (pass != 1 && pass != 2) return EQB_ERR_INVALID_ARG;
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (!hist || !sel_hi || !rank_in_bin) return EQB_ERR_INVALID_ARG;
  if (pass == 2 && (!sel_lo || !q_bf16)) return EQB_ERR_INVALID_ARG;
  return launch_select_local(pass, hist, E, K, pt, sel_hi, rank_in_bin, sel_lo, q_bf16, dev_status,
                             static_cast<hipStream_t>(stream));
}

eqb_status eqb_margin_hist_pass2_local(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                       const int32_t* sel_hi, const int64_t* part_off, int32_t P,
                                       int32_t* hist_lo, void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  MarginArgs a;
  const eqb_status st = make_table(part_off, P, T, &a.pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !tau || !hist_lo || !sel_hi) return EQB_ERR_INVALID_ARG;
  if (!aligned16(z)) return EQB_ERR_UNSUPPORTED;
  a.z = z;
  a.tau = tau;
  a.T = T;
  a.E = E;
  a.sel_hi = sel_hi;
  a.sel_stride = E;
  a.hist = hist_lo;
  return launch_margin(true, a, static_cast<hipStream_t>(stream));
}

eqb_status eqb_rank_average(const uint16_t* q_bf16, int64_t T, int32_t E, const int64_t* part_off,
                            int32_t P, double* b_avg, float* b_next, void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (!q_bf16 || !b_next) return EQB_ERR_INVALID_ARG;
  return launch_rank_average(q_bf16, E, pt, b_avg, b_next, static_cast<hipStream_t>(stream));
}

eqb_status eqb_margin_hist_uniform(const uint16_t* z, const float* tau, int64_t T, int32_t E,
                                   const int64_t* part_off, int32_t P, float lo, float hi, int32_t nbins,
                                   int32_t* hist, void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  if (nbins < 1 || nbins > EQB_NBINS) return EQB_ERR_INVALID_ARG;
  const float width = hi - lo;
  if (!(width > 0.0f) || width > 3.4e38f || !(lo == lo)) return EQB_ERR_INVALID_ARG;
  const float scale = (float)nbins / width;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !tau || !hist) return EQB_ERR_INVALID_ARG;
  if (!aligned16(z)) return EQB_ERR_UNSUPPORTED;
  return launch_uniform_hist(z, tau, T, E, pt, lo, scale, nbins, hist, static_cast<hipStream_t>(stream));
}

eqb_status eqb_select_uniform(const int32_t* hist, int32_t P, int32_t E, int32_t nbins, int64_t r, float lo,
                              float hi, double* est, float* b_next, int32_t* dev_status, void* stream) {
  if (P < 1 || P > EQB_MAX_PARTITIONS) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  if (nbins < 1 || nbins > EQB_NBINS) return EQB_ERR_INVALID_ARG;
  if (!(hi - lo > 0.0f) || !(lo == lo)) return EQB_ERR_INVALID_ARG;
  if (r < 1 || r > INT32_MAX) return EQB_ERR_RANK;
  if (!hist || !est) return EQB_ERR_INVALID_ARG;
  const double lo64 = (double)lo;
  const double width = ((double)hi - lo64) / (double)nbins;
  return launch_select_uniform(hist, P, E, nbins, r, lo64, width, est, b_next, dev_status,
                               static_cast<hipStream_t>(stream));
}

eqb_status eqb_max_violation(const int32_t* load, int64_t T, int32_t K, int32_t E,
                             const int64_t* part_off, int32_t P, double* maxvio_global,
                             double* maxvio_local, double* maxvio_local_mean, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!load || !maxvio_global) return EQB_ERR_INVALID_ARG;
  return launch_max_violation(load, E, K, pt, maxvio_global, maxvio_local, maxvio_local_mean,
                              static_cast<hipStream_t>(stream));
}

eqb_status eqb_lei_residual(const int32_t* load, int64_t T, int32_t K, int32_t E,
                            const int64_t* part_off, int32_t P, double eta, double c, float* inj,
                            void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  if (!(eta == eta) || !(c == c)) return EQB_ERR_INVALID_ARG;     // NaN coefficients
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (!load || !inj) return EQB_ERR_INVALID_ARG;
  return launch_lei_residual(load, E, K, pt, eta, c, inj, static_cast<hipStream_t>(stream));
}

eqb_status eqb_lei_inject(float* grad_s, const float* inj, int64_t T, int32_t E,
                          const int64_t* part_off, int32_t P, void* stream) {
  if (T < 0 || T > INT32_MAX) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!grad_s || !inj) return EQB_ERR_INVALID_ARG;
  if (!aligned16(grad_s) || !aligned16(inj)) return EQB_ERR_UNSUPPORTED;
  return launch_lei_inject(grad_s, inj, T, E, pt, static_cast<hipStream_t>(stream));
}

eqb_status eqb_lei_router_backward(const uint16_t* z, const int32_t* topk_idx, const float* grad_score,
                                   const float* inj, int64_t T, int32_t E, int32_t K, const int64_t* part_off,
                                   int32_t P, float* grad_z, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  PartTable pt;
  const eqb_status st = make_table(part_off, P, T, &pt);
  if (st != EQB_OK) return st;
  if (T == 0) return EQB_OK;
  if (!z || !topk_idx || !grad_score || !grad_z) return EQB_ERR_INVALID_ARG;
  if (!aligned16(z) || !aligned16(grad_z)) return EQB_ERR_UNSUPPORTED;
  return launch_lei_router_backward(z, topk_idx, grad_score, inj, T, E, K, grad_z, pt,
                                    static_cast<hipStream_t>(stream));
}

size_t eqb_layer_workspace_size(int32_t E, int32_t P) {
  if (!supported_E(E) || P < 1 || P > EQB_MAX_PARTITIONS) return 0;
  return layer_workspace(nullptr, E, P, nullptr);
}

size_t eqb_layer_workspace_zero_bytes(int32_t E, int32_t P) {
  if (!supported_E(E) || P < 1 || P > EQB_MAX_PARTITIONS) return 0;
  size_t zero = 0;
  layer_workspace(nullptr, E, P, nullptr, true, &zero);
  return zero;
}

eqb_status eqb_layer(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                     const int64_t* part_off, int32_t P, int32_t* topk_idx, float* topk_score, float* tau,
                     int32_t* load, uint16_t* q_bf16, float* b_next, int32_t* hist_hi_sum,
                     int32_t* hist_lo_sum, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                     void* const* marks, void* stream) {
  return layer_call(z, b, T, E, K, part_off, P, topk_idx, topk_score, tau, load, q_bf16, b_next, hist_hi_sum,
                    hist_lo_sum, dev_status, workspace, workspace_bytes, true, marks, stream);
}

}  // extern "C"

namespace eqb {

eqb_status layer_call(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                      const int64_t* part_off, int32_t P, int32_t* topk_idx, float* topk_score, float* tau,
                      int32_t* load, uint16_t* q_bf16, float* b_next, int32_t* hist_hi_sum,
                      int32_t* hist_lo_sum, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                      bool with_part, void* const* marks, void* stream) {
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (!supported_E(E)) return EQB_ERR_UNSUPPORTED;
  RouteArgs a;
  const eqb_status st = make_table(part_off, P, T, &a.pt);
  if (st != EQB_OK) return st;
  const int64_t r = eqb_rank(T, K, E);
  if (r < 1) return EQB_ERR_RANK;
  if (!z || !b || !topk_idx || !topk_score || !tau || !load || !q_bf16 || !b_next || !dev_status || !workspace)
    return EQB_ERR_INVALID_ARG;
  if (!aligned16(z)) return EQB_ERR_UNSUPPORTED;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return EQB_ERR_UNSUPPORTED;
  LayerWorkspace w;
  if (workspace_bytes < layer_workspace(workspace, E, a.pt.P, &w, with_part)) return EQB_ERR_INVALID_ARG;
  a.z = z;
  a.b = b;
  a.T = T;
  a.E = E;
  a.K = K;
  a.idx = topk_idx;
  a.score = topk_score;
  a.tau = tau;
  return launch_layer(a, r, w, q_bf16, b_next, load, hist_hi_sum, hist_lo_sum, dev_status, marks,
                      static_cast<hipStream_t>(stream));
}

}  // namespace eqb

extern "C" {

eqb_status eqb_set_max_blocks(int32_t max_blocks) {
  if (max_blocks < 0) return EQB_ERR_INVALID_ARG;
  t_max_blocks = max_blocks;
  return EQB_OK;
}

int32_t eqb_get_max_blocks(void) { return t_max_blocks; }

int64_t eqb_rank(int64_t T_total, int32_t K, int32_t E) {
  if (T_total < 0 || E < 1 || K < 1 || K >= E) return -1;
  if (T_total > ((int64_t)1 << 40)) return -1;
  return (T_total * (int64_t)K + E - 1) / E;
}

const char* eqb_status_string(eqb_status status) {
  switch (status) {
    case EQB_OK: return "EQB_OK";
    case EQB_ERR_INVALID_ARG: return "EQB_ERR_INVALID_ARG";
    case EQB_ERR_UNSUPPORTED: return "EQB_ERR_UNSUPPORTED";
    case EQB_ERR_RANK: return "EQB_ERR_RANK";
    case EQB_ERR_HIP: return "EQB_ERR_HIP";
    case EQB_ERR_SCRATCH: return "EQB_ERR_SCRATCH";
    default: return "EQB_ERR_UNKNOWN";
  }
}

}  // extern "C"
