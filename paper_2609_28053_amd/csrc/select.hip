// select.hip - selection steps of Algorithm 1 (arXiv 2609.28053, Appendix C):
// the all-reduce stand-in (sum of the P partition slabs), the coarse choice
// u_e, rho_e (step 3), the fine choice v_e and b_hat_e = kappa^-1(u_e, v_e)
// (steps 5-6), and the centred bias of Eq. 2.
#include "eqb_internal.hpp"

namespace eqb {

// One block per expert (and, with kLocal, per partition), one thread per bin.
// Global: the P slabs are summed first (the all-reduce) and r is the rank over
// the whole batch.  kLocal: slab p alone, with its own rank
// r_p = ceil(|B_p| K / E), written to entry [p, e]; an empty partition has no
// quantile and gets -1 without raising the status.
// Layer form (eqb_layer): `clear` zeroes the summed counters once read, and
// the loads accumulated by the route kernel (load_acc [P,E]) are copied to
// load_out and zeroed, so the workspace is left as it was found: all zero.
// Each counter is read and cleared by the same thread.
// kSlab16 (the layer, global form): the P slabs hold 16-bit counters in the
// layout of PartTable::slab16; each is read, summed and cleared as a uint16.
template <bool kLocal, bool kSlab16 = false>
__global__ __launch_bounds__(kNBins) void select_coarse_kernel(
    int32_t* __restrict__ hist, int P, int E, int K, int64_t r, const PartTable pt,
    int32_t* __restrict__ sel_hi, int64_t* __restrict__ rank_in_bin, int32_t* __restrict__ hist_sum,
    int32_t* __restrict__ status, bool clear = false, int32_t* __restrict__ load_acc = nullptr,
    int32_t* __restrict__ load_out = nullptr, int32_t* __restrict__ pool_reset = nullptr) {
  __shared__ int64_t sh[kNBins];
  const int e = blockIdx.x, u = threadIdx.x, p = kLocal ? (int)blockIdx.y : 0;
  // the layer's claim counters of the sweep that ran before (one per partition)
  if (pool_reset && e == 0)
    for (int q = u; q < kPoolCounters; q += kNBins) pool_reset[(int64_t)q * kPoolStride] = 0;
  const int64_t out = kLocal ? (int64_t)p * E + e : e;
  if (kLocal) {
    const int64_t n = pt.off[p + 1] - pt.off[p];
    if (n == 0) {
      if (u == 0) {
        sel_hi[out] = -1;
        rank_in_bin[out] = 0;
      }
      return;
    }
    r = (n * K + E - 1) / E;
  }
  int64_t c = 0;
  if (kLocal) {
    c = hist[((int64_t)p * E + e) * kNBins + u];
  } else {
    if (kSlab16) {
      uint16_t* h16 = reinterpret_cast<uint16_t*>(hist) + ((int64_t)(e >> 1) * kNBins + u) * 2 + (e & 1);
      const int64_t stride = (int64_t)E * kNBins * 2;  // one int32 slab, in 16-bit units
      int q = 0;
      for (; q + 8 <= P; q += 8) {
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = h16[(q + j) * stride];
#pragma unroll
        for (int j = 0; j < 8; ++j) c += v[j];
      }
      for (; q < P; ++q) c += h16[q * stride];
      if (clear)
        for (int q2 = 0; q2 < P; ++q2) h16[q2 * stride] = 0;
    } else {
      c = slab_sum(hist + (int64_t)e * kNBins + u, P, (int64_t)E * kNBins);
      if (clear) slab_clear(hist + (int64_t)e * kNBins + u, P, (int64_t)E * kNBins);
    }
    if (hist_sum) hist_sum[(int64_t)e * kNBins + u] = (int32_t)c;
    if (load_acc) {
      for (int q = u; q < pt.P; q += kNBins) {
        load_out[(int64_t)q * E + e] = load_acc[(int64_t)q * E + e];
        load_acc[(int64_t)q * E + e] = 0;
      }
    }
  }
  const int64_t cum = block_inclusive_scan_256(c, sh);
  if (cum >= r && cum - c < r) {
    sel_hi[out] = u;
    rank_in_bin[out] = r - (cum - c);
  }
  if (u == kNBins - 1 && cum < r) {
    sel_hi[out] = -1;
    rank_in_bin[out] = 0;
    if (status) *status = EQB_DEV_RANK_EXCEEDS_COUNT;
  }
}

template <bool kLocal>
__global__ __launch_bounds__(kNBins) void select_fine_kernel(
    int32_t* __restrict__ hist, int P, int E, const PartTable pt, const int32_t* __restrict__ sel_hi,
    const int64_t* __restrict__ rank_in_bin, int32_t* __restrict__ sel_lo,
    uint16_t* __restrict__ q_bf16, int32_t* __restrict__ hist_sum, int32_t* __restrict__ status,
    bool clear = false, int32_t* __restrict__ pool_reset = nullptr) {
  __shared__ int64_t sh[kNBins];
  const int e = blockIdx.x, v = threadIdx.x, p = kLocal ? (int)blockIdx.y : 0;
  if (pool_reset && e == 0)
    for (int q = v; q < kPoolCounters; q += kNBins) pool_reset[(int64_t)q * kPoolStride] = 0;
  const int64_t out = kLocal ? (int64_t)p * E + e : e;
  if (kLocal && pt.off[p + 1] == pt.off[p]) {
    if (v == 0) {
      sel_lo[out] = -1;
      q_bf16[out] = 0x7FC0;
    }
    return;
  }
  // the coarse choice is read first: its load overlaps those of the counts
  const int u = sel_hi[out];
  const int64_t rho = rank_in_bin[out];
  int64_t c = 0;
  if (kLocal) {
    c = hist[((int64_t)p * E + e) * kNBins + v];
  } else {
    c = slab_sum(hist + (int64_t)e * kNBins + v, P, (int64_t)E * kNBins);
    if (hist_sum) hist_sum[(int64_t)e * kNBins + v] = (int32_t)c;
    if (clear) slab_clear(hist + (int64_t)e * kNBins + v, P, (int64_t)E * kNBins);
  }
  const int64_t cum = block_inclusive_scan_256(c, sh);
  const bool ok = u >= 0 && u < kNBins && rho >= 1;
  if (ok && cum >= rho && cum - c < rho) {
    sel_lo[out] = v;
    q_bf16[out] = kappa_inv(((uint32_t)u << 8) | (uint32_t)v);
  }
  if (v == kNBins - 1 && (!ok || cum < rho)) {
    sel_lo[out] = -1;
    q_bf16[out] = 0x7FC0;
    if (status) *status = EQB_DEV_RANK_EXCEEDS_COUNT;
  }
}

// The fine selection of a layer from the fine pass's per-block count images
// (steps 5-6 of Algorithm 1 with the all-reduce stand-in summing the images
// instead of partition slabs).  One block per expert pair (2m, 2m+1), 512
// threads: each wave sums every eighth image's row for the pair (one
// 16-byte load per lane: raw low bytes 4l..4l+3 of both experts), the waves'
// sums meet in LDS, and threads 256x + v then hold kappa bin v of expert
// 2m + x: raw low byte v, or v ^ 0xFF when the expert's selected coarse bin
// holds negative margins (kappa flips every bit of a negative value).  The
// scan and the choice are those of select_fine_kernel.  Image counts are
// below 2^16 and the sums below 2^31 (T < 2^31).
constexpr int kPartThreads = 512;
__global__ __launch_bounds__(kPartThreads) void select_fine_parts_kernel(
    const uint32_t* __restrict__ part, int nparts, int E, const int32_t* __restrict__ sel_hi,
    const int64_t* __restrict__ rank_in_bin, int32_t* __restrict__ sel_lo, uint16_t* __restrict__ q_bf16,
    int32_t* __restrict__ hist_sum) {
  constexpr int kW = kPartThreads / 64;
  __shared__ uint32_t sh[kW][2 * kNBins];   // per wave: raw bins of expert 2m, then of 2m+1
  __shared__ int sh_tot[kW];
  const int m = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t words = part_words(E);
  const uint4* src = reinterpret_cast<const uint4*>(part + (int64_t)m * kNBins) + lane;
  uint32_t lo[4] = {0, 0, 0, 0}, hi[4] = {0, 0, 0, 0};
  int b = wave;
  for (; b + 3 * kW < nparts; b += 4 * kW) {
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = src[(b + j * kW) * words / 4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lo[i] += w[i] & 0xFFFFu;
        hi[i] += w[i] >> 16;
      }
    }
  }
  for (; b < nparts; b += kW) {
    const uint4 v = src[b * words / 4];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lo[i] += w[i] & 0xFFFFu;
      hi[i] += w[i] >> 16;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sh[wave][4 * lane + i] = lo[i];
    sh[wave][kNBins + 4 * lane + i] = hi[i];
  }
  __syncthreads();
  const int x = threadIdx.x >> 8, v = threadIdx.x & (kNBins - 1);
  const int e = 2 * m + x;
  const int u = sel_hi[e];
  const int64_t rho = rank_in_bin[e];
  const bool ok = u >= 0 && u < kNBins && rho >= 1;
  const bool valid_u = u >= 0 && u < kNBins;
  const int raw = (valid_u && u < 0x80) ? (v ^ 0xFF) : v;
  int c = 0;
#pragma unroll
  for (int w = 0; w < kW; ++w) c += (int)sh[w][x * kNBins + raw];
  // the fine pass counted an expert without a valid coarse choice in bin 0;
  // like the slab flush, the selection drops those counts
  if (!valid_u) c = 0;
  if (hist_sum) hist_sum[(int64_t)e * kNBins + v] = c;
  // inclusive scan over the 256 threads of expert x (waves 4x .. 4x+3)
  int y = c;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(y, d);
    if (lane >= d) y += t;
  }
  if (lane == 63) sh_tot[wave] = y;
  __syncthreads();
  for (int w = 4 * x; w < wave; ++w) y += sh_tot[w];
  const int64_t cum = y;
  if (ok && cum >= rho && cum - c < rho) {
    sel_lo[e] = v;
    q_bf16[e] = kappa_inv(((uint32_t)u << 8) | (uint32_t)v);
  }
  if (v == kNBins - 1 && (!ok || cum < rho)) {
    sel_lo[e] = -1;
    q_bf16[e] = 0x7FC0;
  }
}

// b = b_hat - mean(b_hat): binary64 sum in ascending expert order, divided by
// E, difference in binary64, one rounding to binary32.  With status_out (the
// layer form) the kernel also writes the layer's status (an expert whose fine
// selection failed, sel_lo = -1, holds fewer counts than its rank) and, as the
// layer's last kernel, zeroes the selections it leaves behind in the
// workspace (sel_hi, rank_in_bin, sel_lo), each by the thread that read it.
__global__ __launch_bounds__(256) void center_kernel(const uint16_t* __restrict__ q, int E,
                                                     float* __restrict__ b_next,
                                                     int32_t* __restrict__ sel_lo = nullptr,
                                                     int32_t* __restrict__ status_out = nullptr,
                                                     int32_t* __restrict__ sel_hi = nullptr,
                                                     int64_t* __restrict__ rank_in_bin = nullptr) {
  __shared__ double val[256];
  __shared__ double mean;
  for (int e = threadIdx.x; e < E; e += blockDim.x) val[e] = (double)__uint_as_float((uint32_t)q[e] << 16);
  int bad = 0;
  if (status_out) {
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
      bad |= (int)(sel_lo[e] < 0);
      sel_lo[e] = 0;
      sel_hi[e] = 0;
      rank_in_bin[e] = 0;
    }
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int e = 0; e < E; ++e) acc += val[e];
    mean = acc / (double)E;
    if (status_out) *status_out = bad ? EQB_DEV_RANK_EXCEEDS_COUNT : EQB_DEV_OK;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) b_next[e] = (float)(val[e] - mean);
}

// The layer's selections: the counts sit in P * nsub slabs, all summed; the
// loads in P rows.
eqb_status launch_layer_selects(int pass, int32_t* hist, int P, int nsub, int E, int64_t r, int32_t* sel_hi,
                                int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                                int32_t* hist_sum, int32_t* load_acc, int32_t* load_out, int32_t* status,
                                int32_t* pool_reset, hipStream_t s, bool slab16) {
  PartTable none{};
  none.P = P;
  const int nslabs = P * nsub;
  if (pass == 1) {
    if (slab16)
      select_coarse_kernel<false, true><<<E, kNBins, 0, s>>>(hist, nslabs, E, 0, r, none, sel_hi, rank_in_bin,
                                                             hist_sum, nullptr, true, load_acc, load_out, pool_reset);
    else
      select_coarse_kernel<false><<<E, kNBins, 0, s>>>(hist, nslabs, E, 0, r, none, sel_hi, rank_in_bin, hist_sum,
                                                       nullptr, true, load_acc, load_out, pool_reset);
    return launch_status();
  }
  select_fine_kernel<false><<<E, kNBins, 0, s>>>(hist, nslabs, E, none, sel_hi, rank_in_bin, sel_lo, q_bf16,
                                                 hist_sum, nullptr, true, pool_reset);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  center_kernel<<<1, 256, 0, s>>>(q_bf16, E, b_next, sel_lo, status, sel_hi, rank_in_bin);
  return launch_status();
}

eqb_status launch_layer_select_parts(const uint32_t* part, int nparts, int E, int32_t* sel_hi,
                                     int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                                     int32_t* hist_sum, int32_t* status, hipStream_t s) {
  select_fine_parts_kernel<<<E / 2, kPartThreads, 0, s>>>(part, nparts, E, sel_hi, rank_in_bin, sel_lo, q_bf16,
                                                          hist_sum);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  center_kernel<<<1, 256, 0, s>>>(q_bf16, E, b_next, sel_lo, status, sel_hi, rank_in_bin);
  return launch_status();
}

static eqb_status mark(void* const* marks, int i, hipStream_t s) {
  if (marks == nullptr || marks[i] == nullptr) return EQB_OK;
  return hipEventRecord(static_cast<hipEvent_t>(marks[i]), s) == hipSuccess ? EQB_OK : EQB_ERR_HIP;
}

eqb_status launch_layer(const RouteArgs& route, int64_t r, const LayerWorkspace& w, uint16_t* q_bf16,
                        float* b_next, int32_t* load_out, int32_t* hist_hi_sum, int32_t* hist_lo_sum,
                        int32_t* dev_status, void* const* marks, hipStream_t s) {
  RouteArgs a = route;
  a.load = w.load_acc;
  a.hist = w.hist_hi;
  a.pt.nsub = w.nsub;
  a.pt.pool = w.pool;
  a.slab16_ok = true;
  eqb_status st = mark(marks, 0, s);
  if (st != EQB_OK) return st;
  bool slab16 = false;
  st = launch_route(a, s, &slab16);
  if (st != EQB_OK) return st;
  if ((st = mark(marks, 1, s)) != EQB_OK) return st;
  const int P = a.pt.P, E = a.E;
  st = launch_layer_selects(1, w.hist_hi, P, w.nsub, E, r, w.sel_hi, w.rank_in_bin, nullptr, nullptr, nullptr,
                            hist_hi_sum, w.load_acc, load_out, nullptr, w.pool, s, slab16);
  if (st != EQB_OK) return st;
  if ((st = mark(marks, 2, s)) != EQB_OK) return st;
  MarginArgs m;
  m.z = a.z;
  m.tau = a.tau;
  m.T = a.T;
  m.E = E;
  m.sel_hi = w.sel_hi;
  m.hist = w.hist_lo;
  m.pt = a.pt;
  m.pt.pool = nullptr;   // the fine pass keeps static ranges
  m.part = w.part;
  m.part_blocks = w.part_blocks;
  int nparts = 0;
  st = launch_margin(true, m, s, &nparts);
  if (st != EQB_OK) return st;
  if ((st = mark(marks, 3, s)) != EQB_OK) return st;
  if (nparts > 0)
    st = launch_layer_select_parts(w.part, nparts, E, w.sel_hi, w.rank_in_bin, w.sel_lo, q_bf16, b_next,
                                   hist_lo_sum, dev_status, s);
  else
    st = launch_layer_selects(2, w.hist_lo, P, w.nsub, E, r, w.sel_hi, w.rank_in_bin, w.sel_lo, q_bf16, b_next,
                              hist_lo_sum, nullptr, nullptr, dev_status, nullptr, s);
  if (st != EQB_OK) return st;
  return mark(marks, 4, s);
}

eqb_status launch_select(int pass, const int32_t* hist, int P, int E, int64_t r, int32_t* sel_hi,
                         int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                         int32_t* hist_sum, int32_t* status, hipStream_t s) {
  PartTable none{};
  none.P = P;
  if (pass == 1) {
    select_coarse_kernel<false><<<E, kNBins, 0, s>>>(const_cast<int32_t*>(hist), P, E, 0, r, none, sel_hi,
                                                     rank_in_bin, hist_sum, status);
    return launch_status();
  }
  select_fine_kernel<false><<<E, kNBins, 0, s>>>(const_cast<int32_t*>(hist), P, E, none, sel_hi, rank_in_bin,
                                                 sel_lo, q_bf16, hist_sum, status);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  if (b_next) {
    center_kernel<<<1, 256, 0, s>>>(q_bf16, E, b_next);
    return launch_status();
  }
  return EQB_OK;
}

eqb_status launch_select_local(int pass, const int32_t* hist, int E, int K, const PartTable& pt,
                               int32_t* sel_hi, int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16,
                               int32_t* status, hipStream_t s) {
  const dim3 grid(E, pt.P);
  if (pass == 1)
    select_coarse_kernel<true><<<grid, kNBins, 0, s>>>(const_cast<int32_t*>(hist), pt.P, E, K, 0, pt, sel_hi,
                                                       rank_in_bin, nullptr, status);
  else
    select_fine_kernel<true><<<grid, kNBins, 0, s>>>(const_cast<int32_t*>(hist), pt.P, E, pt, sel_hi,
                                                     rank_in_bin, sel_lo, q_bf16, nullptr, status);
  return launch_status();
}

}  // namespace eqb
