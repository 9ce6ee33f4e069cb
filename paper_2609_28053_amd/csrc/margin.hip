// margin.hip - coarse and fine counts of the BF16 margins tau_t - z_{t,e}
// (Algorithm 1, steps 1 and 4 of arXiv 2609.28053, Appendix C) and the
// expert loads f_e (Sec. 2) from stored Top-K indices.
//
// Each lane holds 8 experts of a row (one 16-byte load); G = E/8 lanes cover a
// row and every lane works on U rows per step; the next step's U loads are
// issued before a step is counted.  Margins are rounded to BF16 two at a time
// by the hardware conversion (round to nearest even, subnormals kept).  Counts
// go to packed LDS histograms indexed by the raw BF16 byte; the flush maps
// them to kappa bins.  In the one-call layer the fine pass instead stores
// each block's LDS counts, raw bytes and all, as one image that the fine
// selection sums (select.hip).
#include "eqb_internal.hpp"

namespace eqb {

constexpr int kMarginU = 3;   // rows per lane per block step
constexpr int kPartMinRows = 512;    // least rows per block when the blocks store count images
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Counts the margins of one row piece: eight experts e0 .. e0+7 (four packed
// BF16 pairs in w) against tau.  Two margins are rounded by one conversion;
// p holds bf16(tau - z_j) in bits 0..15 and bf16(tau - z_{j+1}) in bits 16..31.
//  coarse: the raw high bytes are bits 8..15 and 24..31 of p;
//  fine  : x = p ^ C with C = U_{j+1} << 24 | U_j << 8 (U = raw form of the
//          selected bin u_e) has zero high bytes exactly for the margins in the
//          selected bins, and its bits 0..7 / 16..23 are their raw low bytes.
template <bool kFine>
__device__ __forceinline__ void count_piece(uint32_t* sh, const uint4& w, float tv, uint32_t row0,
                                            const uint32_t (&csel)[4]) {
  const uint32_t w4[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t p = bf16x2_bits(tv - bf16_lo(w4[i]), tv - bf16_hi(w4[i]));
    uint32_t* rowp = sh + row0 + i * kHistStride;
    if (!kFine) {
      atomicAdd(rowp + ((p >> 8) & 0xFFu), 1u);
      atomicAdd(rowp + (p >> 24), 1u << 16);
    } else {
      const uint32_t x = p ^ csel[i];
      if ((x & 0xFF00u) == 0u) atomicAdd(rowp + (x & 0xFFu), 1u);
      if (x < (1u << 24)) atomicAdd(rowp + ((x >> 16) & 0xFFu), 1u << 16);
    }
  }
}

// sel_stride = 0: every partition uses the selection sel_hi[e] (EQB: the
// bins chosen from the summed counts).  sel_stride = E: partition p uses its
// own selection sel_hi[p*E + e] (each shard's own quantile).
// part (fine pass with sel_stride 0, at most kSegMax rows per block): the
// block's counts, summed over the partitions it covers, are stored as one
// image of part_words(E) words at part + blockIdx.x * part_words(E) (plain
// stores; the fine selection sums the images) instead of being added to the
// partition slabs, whose atomics queue in the memory system when every block
// flushes at once.
template <int E, bool kFine>
__global__ __launch_bounds__(kBlock) void margin_hist_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ tau, int64_t T,
    const int32_t* __restrict__ sel_hi, int sel_stride, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block, uint32_t* __restrict__ part) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R * kMarginU;
  __shared__ __align__(16) uint32_t sh_hist[hist_words<E>()];
  __shared__ int32_t sh_sel[kFine ? E : 1];   // the segment's selections, for the flush

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  const uint32_t row0 = hist_row(e0);
  for (int w = threadIdx.x; w < hist_words<E>() / 4; w += kBlock)
    reinterpret_cast<uint4*>(sh_hist)[w] = make_uint4(0, 0, 0, 0);
  for (int w = (hist_words<E>() / 4) * 4 + threadIdx.x; w < hist_words<E>(); w += kBlock) sh_hist[w] = 0;
  __syncthreads();

  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  // Rows are visited last to first: the route sweep that precedes this one
  // reads every block range first to last, so the rows it read last may still
  // be held by the memory-side cache.
  for_each_segment_rev(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    const int32_t* sel = kFine ? sel_hi + (int64_t)p * sel_stride : nullptr;
    if (kFine) {
      // read once here: the flush looks a selection up per populated bin,
      // and a global load there would sit on its critical path
      for (int e = threadIdx.x; e < E; e += kBlock) sh_sel[e] = sel[e];
    }
    uint32_t csel[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t c = 0;
      if (kFine) {
        int u0 = sel[e0 + 2 * i], u1 = sel[e0 + 2 * i + 1];
        u0 = (u0 >= 0 && u0 < kNBins) ? u0 : 0;   // invalid selections are skipped at the flush
        u1 = (u1 >= 0 && u1 < kNBins) ? u1 : 0;
        c = ((uint32_t)raw_hi_of_kappa(u1) << 24) | ((uint32_t)raw_hi_of_kappa(u0) << 8);
      }
      csel[i] = c;
    }
    // Rows are addressed by 32-bit byte offsets from the segment's first row
    // (a segment holds at most kSegMax rows).  The next step's rows are in
    // flight while a step is counted; each step starts by taking the rows
    // prefetched one step earlier.  A row past the segment reads the
    // segment's last row instead and is not counted.
    uint4 va[kMarginU], vb[kMarginU];
    float ta[kMarginU], tb[kMarginU];
    const char* seg_z = reinterpret_cast<const char*>(z + s0 * E);
    const char* seg_tau = reinterpret_cast<const char*>(tau + s0);
    const uint32_t n = (uint32_t)(s1 - s0);
    auto load_step = [&](uint4 (&v)[kMarginU], float (&tv)[kMarginU], uint32_t base) {
#pragma unroll
      for (int u = 0; u < kMarginU; ++u) {
        uint32_t t = base + (uint32_t)((u * kWaves + wave) * R + rr);
        t = t < n ? t : n - 1;
        // z is read once per sweep and not again in this layer: a
        // non-temporal load streams it without allocating it in the caches
        const u32x4 x = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(seg_z + (t * (uint32_t)E + (uint32_t)e0) * 2u));
        v[u] = make_uint4(x.x, x.y, x.z, x.w);
        tv[u] = *reinterpret_cast<const float*>(seg_tau + t * 4u);
      }
    };
    const uint32_t last = ((n - 1) / ROWS) * ROWS;
    load_step(vb, tb, last);
    for (uint32_t step = 0; step <= last / ROWS; ++step) {
      const uint32_t base = last - step * ROWS;
#pragma unroll
      for (int u = 0; u < kMarginU; ++u) { va[u] = vb[u]; ta[u] = tb[u]; }
      if (base >= ROWS) load_step(vb, tb, base - ROWS);
#pragma unroll
      for (int u = 0; u < kMarginU; ++u) {
        const uint32_t t = base + (uint32_t)((u * kWaves + wave) * R + rr);
        if (t < n) count_piece<kFine>(sh_hist, va[u], ta[u], row0, csel);
      }
    }
    if (kFine && part) return;   // the counts stay in LDS until the block's image is stored
    __syncthreads();
    int32_t* slab = count_slab(hist, pt, p, E);
    if (!kFine) {
      flush_hist<E, false>(sh_hist, slab, nullptr);
    } else {
      flush_hist<E, true>(sh_hist, slab, sh_sel);
    }
    __syncthreads();
  });
  if (kFine && part) {
    __syncthreads();
    // four words of one pair's row per thread: word m*257 + 4k.. in LDS,
    // 16 bytes at m*256 + 4k in the image
    uint4* dst = reinterpret_cast<uint4*>(part + (int64_t)blockIdx.x * part_words(E));
    for (int it = threadIdx.x; it < (E / 2) * (kNBins / 4); it += kBlock) {
      const uint32_t* src = sh_hist + (it / (kNBins / 4)) * kHistStride + 4 * (it % (kNBins / 4));
      dst[it] = make_uint4(src[0], src[1], src[2], src[3]);
    }
  }
}

template <int E>
eqb_status launch_margin_e(bool fine, const MarginArgs& a, hipStream_t s, int* part_used) {
  static_assert(hist_words<E>() == (E / 2) * kHistStride, "LDS counts as margin_blocks_per_cu assumes");
  int blocks;
  int64_t rpb;
  const int rows_per_step = kWaves * (64 / (E / 8)) * kMarginU;
  // At least 1,024 rows per block when the counts are flushed with atomics:
  // at one rank's share of the paper's batch (147,456 tokens, E = 256) that
  // roughly halves the blocks whose LDS counts are zeroed and flushed; large
  // batches still fill every CU.  Per-block images cost a block far less, so
  // their blocks may be shorter; they run one block per CU (half the images
  // for the selection to sum where two would fit, and a faster pass: E = 64
  // and 128 layers took 7-13% less time per step).
  const bool want_part = fine && a.part != nullptr && a.sel_stride == 0;
  const int min_rows = want_part ? kPartMinRows : 1024;
  grid_for(a.T, rows_per_step, want_part ? 1 : margin_blocks_per_cu(E), &blocks, &rpb,
           (min_rows + rows_per_step - 1) / rows_per_step);
  const bool use_part = want_part && blocks <= a.part_blocks && rpb <= kSegMax;
  if (part_used) *part_used = use_part ? blocks : 0;
  if (fine)
    margin_hist_kernel<E, true><<<blocks, kBlock, 0, s>>>(a.z, a.tau, a.T, a.sel_hi, a.sel_stride, a.hist,
                                                         a.pt, rpb, use_part ? a.part : nullptr);
  else
    margin_hist_kernel<E, false><<<blocks, kBlock, 0, s>>>(a.z, a.tau, a.T, a.sel_hi, 0, a.hist, a.pt, rpb,
                                                          nullptr);
  return launch_status();
}

eqb_status launch_margin(bool fine, const MarginArgs& a, hipStream_t s, int* part_used) {
  switch (a.E) {
    case 8: return launch_margin_e<8>(fine, a, s, part_used);
    case 16: return launch_margin_e<16>(fine, a, s, part_used);
    case 32: return launch_margin_e<32>(fine, a, s, part_used);
    case 64: return launch_margin_e<64>(fine, a, s, part_used);
    case 128: return launch_margin_e<128>(fine, a, s, part_used);
    case 256: return launch_margin_e<256>(fine, a, s, part_used);
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
