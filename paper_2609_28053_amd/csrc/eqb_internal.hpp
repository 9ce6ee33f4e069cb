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
  // The layer: `hist` is workspace slabs that only its own coarse selection
  // reads, so the route kernel may use 16-bit counters (PartTable::slab16).
  bool slab16_ok = false;
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
  // Fine pass of a layer (sel_stride 0, counts summed over partitions): room
  // for part_blocks per-block images of the LDS counts (part_words(E) words
  // each).  When the pass's grid fits (at most part_blocks blocks, at most
  // kSegMax rows per block) every block stores its counts there with plain
  // stores instead of adding them to `hist`.
  uint32_t* part = nullptr;
  int part_blocks = 0;
};

// Words of one block's image of the fine counts: for each expert pair
// (2m, 2m+1), 256 words holding the two experts' 16-bit counts of raw low
// byte j in their low and high halves.
__host__ __device__ inline int64_t part_words(int E) { return (int64_t)(E / 2) * kNBins; }
// Blocks of the fine pass per compute unit (its LDS counts take (E/2) * 257
// words per block) when it adds its counts to slabs, and the per-block images
// a layer workspace holds: the image-storing pass runs one block per compute
// unit, and the workspace has room for one full grid on a device of up to
// 256 compute units (a larger device runs the pass with fewer, longer blocks).
inline int margin_blocks_per_cu(int E) { return (E / 2) * kHistStride * 4 * 2 <= 160 * 1024 ? 2 : 1; }
constexpr int kPartCUs = 256;
inline int layer_part_blocks(int) { return kPartCUs; }

// *slab16_used: the coarse counts went to 16-bit slabs (see PartTable).
eqb_status launch_route(const RouteArgs& a, hipStream_t s, bool* slab16_used = nullptr);
// *part_used: the number of per-block images the fine pass wrote (0 when it
// added its counts to a.hist).
eqb_status launch_margin(bool fine, const MarginArgs& a, hipStream_t s, int* part_used = nullptr);
eqb_status launch_load(const int32_t* idx, int64_t T, int K, int E, int32_t* load, const PartTable& pt,
                       hipStream_t s);
eqb_status launch_select(int pass, const int32_t* hist, int P, int E, int64_t r, int32_t* sel_hi,
                         int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                         int32_t* hist_sum, int32_t* status, hipStream_t s);

// slab16: the pass-1 slabs hold 16-bit counters (PartTable::slab16).
eqb_status launch_layer_selects(int pass, int32_t* hist, int P, int nsub, int E, int64_t r, int32_t* sel_hi,
                                int64_t* rank_in_bin, int32_t* sel_lo, uint16_t* q_bf16, float* b_next,
                                int32_t* hist_sum, int32_t* load_acc, int32_t* load_out, int32_t* status,
                                int32_t* pool_reset, hipStream_t s, bool slab16 = false);
// The fine selection of a layer from the fine pass's per-block images
// (nparts of them), then the centring and status as launch_layer_selects(2).
eqb_status launch_layer_select_parts(const uint32_t* part, int nparts, int E, int32_t* sel_hi,
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
                                double* out_global, double* out_local, double* out_local_mean, hipStream_t s);

eqb_status launch_lei_residual(const int32_t* load, int E, int K, const PartTable& pt, double eta,
                               double c, float* inj, hipStream_t s);
eqb_status launch_lei_router_backward(const uint16_t* z, const int32_t* idx, const float* gs, const float* inj,
                                      int64_t T, int E, int K, float* gz, const PartTable& pt, hipStream_t s);
eqb_status launch_lei_inject(float* grad, const float* inj, int64_t T, int E, const PartTable& pt,
                             hipStream_t s);

// Count slabs per partition in a layer's workspace: enough that about 8
// slabs share the blocks of a launch, so no counter receives the flush
// atomics of every block.  Only the route sweep's coarse counts use them
// when the fine pass stores per-block images, and the coarse selection reads
// and clears every slab: 8 measured faster than 16, 4, 2 or 1 at one
// partition of 147,456 tokens (1.2% against 16), and no slower on the other
// workloads.
inline int layer_replicas(int P) { return P >= 8 ? 1 : 8 / P; }

// Working buffers of one layer (eqb_layer): the per-partition coarse and
// fine counts (layer_replicas(P) slabs per partition), the loads as the
// route kernel accumulates them, the selections, and (optionally) room for
// the fine pass's per-block count images.  Each piece starts on a 256-byte
// boundary.  The counters (everything before the images) are zero when a
// layer starts and zero again when it ends: the selection that reads a
// counter clears it.  The images are scratch: the fine pass overwrites the
// ones the fine selection reads.
struct LayerWorkspace {
  int nsub;               // count slabs per partition
  int32_t* hist_hi;       // [P,nsub,E,256]
  int32_t* hist_lo;       // [P,nsub,E,256]
  int32_t* load_acc;      // [P,E]
  int32_t* sel_hi;        // [E]
  int32_t* sel_lo;        // [E]
  int64_t* rank_in_bin;   // [E]
  int32_t* pool;          // claim counters of the route sweep's dynamic tails (kPoolCounters, kPoolStride apart)
  uint32_t* part;         // [part_blocks, part_words(E)] or null
  int part_blocks;
};

inline size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Bytes of a layer workspace, and its pieces carved from base (null base:
// only the size is computed).  with_part = false leaves out the fine pass's
// images (the layer then adds the fine counts to the slabs); *zero_bytes
// (nullable) receives the size of the leading part that holds the counters.
inline size_t layer_workspace(void* base, int E, int P, LayerWorkspace* w, bool with_part = true,
                              size_t* zero_bytes = nullptr) {
  const int nsub = layer_replicas(P);
  const size_t hist = align256((size_t)P * nsub * E * kNBins * sizeof(int32_t));
  const size_t load = align256((size_t)P * E * sizeof(int32_t));
  const size_t sel = align256((size_t)E * sizeof(int32_t));
  const size_t rib = align256((size_t)E * sizeof(int64_t));
  const size_t pool = (size_t)kPoolCounters * kPoolStride * sizeof(int32_t);
  const size_t zero = 2 * hist + load + 2 * sel + rib + pool;
  const size_t part = with_part ? align256((size_t)layer_part_blocks(E) * part_words(E) * sizeof(uint32_t)) : 0;
  if (base && w) {
    char* p = static_cast<char*>(base);
    w->nsub = nsub;
    w->hist_hi = reinterpret_cast<int32_t*>(p);
    w->hist_lo = reinterpret_cast<int32_t*>(p + hist);
    w->load_acc = reinterpret_cast<int32_t*>(p + 2 * hist);
    w->sel_hi = reinterpret_cast<int32_t*>(p + 2 * hist + load);
    w->sel_lo = reinterpret_cast<int32_t*>(p + 2 * hist + load + sel);
    w->rank_in_bin = reinterpret_cast<int64_t*>(p + 2 * hist + load + 2 * sel);
    w->pool = reinterpret_cast<int32_t*>(p + 2 * hist + load + 2 * sel + rib);
    w->part = with_part ? reinterpret_cast<uint32_t*>(p + zero) : nullptr;
    w->part_blocks = with_part ? layer_part_blocks(E) : 0;
  }
  if (zero_bytes) *zero_bytes = zero;
  return zero + part;
}

// eqb_layer with the workspace layout chosen by with_part (the fine pass's
// per-block images present or not; see layer_workspace).
eqb_status layer_call(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                      const int64_t* part_off, int32_t P, int32_t* topk_idx, float* topk_score, float* tau,
                      int32_t* load, uint16_t* q_bf16, float* b_next, int32_t* hist_hi_sum,
                      int32_t* hist_lo_sum, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                      bool with_part, void* const* marks, void* stream);

// The whole layer on one stream: route + loads + coarse counts, coarse
// selection (clearing the coarse counts, handing the loads out), fine
// counts, fine selection (clearing the fine counts), centring and status.
// marks (nullable, 5 entries, each nullable): events recorded before the
// route kernel, after it, after the coarse selection, after the fine pass
// and at the end.
eqb_status launch_layer(const RouteArgs& route, int64_t r, const LayerWorkspace& w, uint16_t* q_bf16,
                        float* b_next, int32_t* load_out, int32_t* hist_hi_sum, int32_t* hist_lo_sum,
                        int32_t* dev_status, void* const* marks, hipStream_t s);

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

// The partition table for a launch of `blocks` blocks: pool mode (pt.pool)
// is kept only when every non-empty partition gets a block of its own under
// block_plan's proportional deal and a block's share is at least min_rows
// (small batches gain nothing from it), else the table falls back to static
// ranges.
inline PartTable pool_table(const PartTable& pt, int64_t T, int blocks, int64_t min_rows) {
  PartTable out = pt;
  if (out.pool == nullptr) return out;
  if (blocks > kPoolCounters || T < min_rows * blocks) {
    out.pool = nullptr;
    return out;
  }
  for (int p = 0; p < pt.P; ++p) {
    if (pt.off[p + 1] > pt.off[p] &&
        pool_block_start(pt, T, blocks, p + 1) <= pool_block_start(pt, T, blocks, p)) {
      out.pool = nullptr;
      break;
    }
  }
  return out;
}

// Most rows any count slab of a route launch with static ranges receives:
// block b covers rows [b * rows_per_block, (b + 1) * rows_per_block) and adds
// partition p's rows to slab p * nsub + b % nsub, so a slab of partition p
// takes at most ceil(c_p / nsub) blocks' rows, c_p the blocks overlapping p.
inline int64_t slab_rows_bound(const PartTable& pt, int64_t rows_per_block) {
  int64_t worst = 0;
  for (int p = 0; p < pt.P; ++p) {
    if (pt.off[p + 1] <= pt.off[p]) continue;
    const int64_t b0 = pt.off[p] / rows_per_block, b1 = (pt.off[p + 1] - 1) / rows_per_block;
    const int64_t c = b1 - b0 + 1;
    const int64_t per = (c + pt.nsub - 1) / pt.nsub;
    const int64_t n = pt.off[p + 1] - pt.off[p];
    const int64_t rows = per * rows_per_block < n ? per * rows_per_block : n;
    worst = rows > worst ? rows : worst;
  }
  return worst;
}

}  // namespace eqb
