// route.hip - Top-K routing of z + b, cutoff tau, sigmoid scores, expert
// loads, fused with the coarse counts of Algorithm 1 step 1 (arXiv
// 2609.28053, Sec. 2 Eq. 1, "Quantile Balancing", Appendix C).
//
// Fast kernel (K <= kFastKmax).  A row of E logits is spread over G lanes,
// each holding N = E/G experts as N/4 8-byte pieces.  Per element it forms a
// 32-bit key: the binary32 bits of s = z + b with the low byte replaced by
// 255 - e, and keeps a sorted top-4 list of keys (one v_max + three v_med3).
// K+2 extraction rounds then take the group maximum of the list heads with
// DPP and pop the winner, refilling a lane whose list runs dry.  For a
// positive tau, signed key order is score order except between scores that
// agree in their top 24 bits; extraction continues until the last key leaves
// the top-24-bit run of rank K, the winners' exact scores are recomputed from
// z and b, and a row whose extracted scores are not in exact order is sorted
// exactly.  Rows with tau <= 0 take the exact 64-bit path.
//
// Generic kernel (any K < E): K+1 rounds over exact 64-bit keys.
#include "eqb_internal.hpp"

namespace eqb {

constexpr int kRmax = 16;              // extracted ranks kept per row
constexpr int kFastKmax = kRmax - 2;

template <int E> struct FastCfg { static constexpr int G = E >= 64 ? 8 : E / 8; };

template <int E>
__global__ __launch_bounds__(kBlock) void route_fast_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ b, int64_t T, int K,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_score, float* __restrict__ tau,
    int32_t* __restrict__ load, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = FastCfg<E>::G;      // lanes per row
  constexpr int N = E / G;              // experts per lane
  constexpr int NQ = N / 4;             // 8-byte pieces per lane and row
  constexpr int R = 64 / G;             // rows per wave
  constexpr int ROWS = kWaves * R;      // rows per block step
  constexpr int RSLOT = (kRmax + G - 1) / G;
  static_assert(N % 4 == 0 && N >= 8, "layout");

  __shared__ uint32_t sh_hist[hist_words<E>()];
  __shared__ uint32_t sh_load[E];
  __shared__ float sh_b[E];
  __shared__ uint2 sh_rank[kWaves][R][kRmax];   // (score bits, zbits << 16 | e) in rank order

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, r = lane / G;

  // Piece q of this lane covers experts ex(q) .. ex(q)+3, so the G lanes of a
  // row read 8*G contiguous bytes per piece.  b is read from LDS, four experts
  // at a time.
  auto ex = [&](int q) -> int { return q * 4 * G + g * 4; };
  // bytes 255 - e for the four experts of a piece (ex is a multiple of 4, no borrow)
  auto idxpk = [&](int q) -> uint32_t { return 0xFCFDFEFFu - (uint32_t)ex(q) * 0x01010101u; };
  for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) sh_hist[w] = 0;
  for (int e = threadIdx.x; e < E; e += kBlock) {
    sh_load[e] = 0;
    sh_b[e] = b[e];
  }
  __syncthreads();

  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  uint2* myrank = sh_rank[wave][r];

  auto bias4 = [&](int q) -> float4 { return *reinterpret_cast<const float4*>(&sh_b[ex(q)]); };
  auto key_of = [&](const uint2* raw, int q, int i, const float4& bq, uint32_t ipk) -> int {
    const uint32_t w = (i < 2) ? raw[q].x : raw[q].y;
    const float zf = (i & 1) ? bf16_hi(w) : bf16_lo(w);
    const float bv = i == 0 ? bq.x : i == 1 ? bq.y : i == 2 ? bq.z : bq.w;
    const uint32_t sb = __float_as_uint(zf + bv);
    return (int)__builtin_amdgcn_perm(sb, ipk, 0x07060500u | (uint32_t)i);
  };

  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    uint2 raw[NQ], nxt[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) nxt[q] = make_uint2(0, 0);
    auto load_rows = [&](uint2* dst, int64_t base) {
      const int64_t t = base + wave * R + r;
#pragma unroll
      for (int q = 0; q < NQ; ++q) dst[q] = make_uint2(0, 0);
      if (t < s1) {
        const uint2* row = reinterpret_cast<const uint2*>(z + t * E);
#pragma unroll
        for (int q = 0; q < NQ; ++q) dst[q] = row[ex(q) >> 2];
      }
    };
    load_rows(raw, s0);
    for (int64_t base = s0; base < s1; base += ROWS) {
      if (base + ROWS < s1) load_rows(nxt, base + ROWS);
      const int64_t t = base + wave * R + r;
      const bool valid = t < s1;

      // ---- per-lane sorted top-4 of keys
      int la = INT_MIN, lb = INT_MIN, lc = INT_MIN, ld = INT_MIN;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const float4 bq = bias4(q);
        const uint32_t ipk = idxpk(q);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = key_of(raw, q, i, bq, ipk);
          ld = med3_i32(lc, ld, x);
          lc = med3_i32(lb, lc, x);
          lb = med3_i32(la, lb, x);
          la = max(la, x);
        }
      }

      // ---- extraction rounds (group-uniform M); lane 0 of the group stages
      // the key of rank k in myrank[k].x
      bool done = !valid;
      int nrank = 0, tauhi = 0;
#pragma unroll 1
      for (int k = 0; k < kRmax; ++k) {
        if (!__any(!done)) break;
        const int M = group_max_i32<G>(la);
        const bool win = (la == M) && (M != INT_MIN);
        if (win) {
          la = lb;
          lb = lc;
          lc = ld;
          ld = INT_MIN;
        }
        if (!done) {
          if (M == INT_MIN) {           // no keys left in the row
            done = true;
          } else {
            if (g == 0) myrank[k].x = (uint32_t)M;
            nrank = k + 1;
            if (k == K) tauhi = M >> 8;
            if (k > K && (M >> 8) != tauhi) done = true;   // one key past the run of rank K
          }
        }
        const bool need = win && la == INT_MIN && !done;
        if (__any(need)) {
          if (need) {   // rebuild this lane's list from its keys below M
            lb = lc = ld = INT_MIN;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
              const float4 bq = bias4(q);
              const uint32_t ipk = idxpk(q);
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                int x = key_of(raw, q, i, bq, ipk);
                x = (x < M) ? x : INT_MIN;
                ld = med3_i32(lc, ld, x);
                lc = med3_i32(lb, lc, x);
                lb = med3_i32(la, lb, x);
                la = max(la, x);
              }
            }
          }
        }
      }
      // exact path when tau is not a positive score or the run did not end
      const bool slow = valid && (!done || tauhi <= 0);
      lds_wave_sync();

      // ---- owners replace the staged keys of their ranks by exact scores
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (valid && !slow && k < nrank) {
          const int e = 255 - (int)(myrank[k].x & 0xFF);
          const uint32_t zb = z[t * E + e];
          const uint32_t sb = __float_as_uint(__uint_as_float(zb << 16) + sh_b[e]);
          myrank[k] = make_uint2(sb, (zb << 16) | (uint32_t)e);
        }
      }
      lds_wave_sync();

      // ---- equal top-24-bit keys whose exact scores differ: sort the row exactly
      bool coll = false;
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (valid && !slow && k + 1 < nrank) {
          const uint2 a = myrank[k], c = myrank[k + 1];
          coll |= ((a.x >> 8) == (c.x >> 8)) && (a.x != c.x);
        }
      }
      const bool coll_row = group_max_i32<G>((int)coll) != 0;
      if (__any(coll_row)) {
        if (coll_row && g == 0) {
          for (int i = 1; i < nrank; ++i) {
            const uint2 v = myrank[i];
            int j = i - 1;
            while (j >= 0) {
              const uint2 u = myrank[j];
              const bool worse = ((int)u.x < (int)v.x) || (u.x == v.x && (u.y & 0xFF) > (v.y & 0xFF));
              if (!worse) break;
              myrank[j + 1] = u;
              --j;
            }
            myrank[j + 1] = v;
          }
        }
        lds_wave_sync();
      }

      // ---- exact 64-bit extraction for rows flagged slow
      if (__any(slow)) {
        if (slow) {
          uint64_t prev = ~0ull;
          for (int k = 0; k <= K; ++k) {
            uint64_t m = 0;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
              const float4 bq = bias4(q);
              // keys are rebuilt every round instead of being held in 2*N registers
              uint2 rq = raw[q];
              asm volatile("" : "+v"(rq.x), "+v"(rq.y));
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const uint32_t w = (i < 2) ? rq.x : rq.y;
                const uint32_t zb = (i & 1) ? (w >> 16) : (w & 0xFFFFu);
                const float bv = i == 0 ? bq.x : i == 1 ? bq.y : i == 2 ? bq.z : bq.w;
                const uint32_t sb = __float_as_uint(__uint_as_float(zb << 16) + bv);
                const uint64_t key = exact_key(sb, ex(q) + i, zb);
                m = (key < prev && key > m) ? key : m;
              }
            }
            m = group_max_u64<G>(m);
            prev = m;
            if (g == 0)
              myrank[k] = make_uint2(exact_key_sbits(m), (exact_key_z(m) << 16) | (uint32_t)exact_key_expert(m));
          }
        }
        lds_wave_sync();
      }

      // ---- outputs: ranks 0..K-1, loads, tau
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (valid && k < K) {
          const uint2 v = myrank[k];
          const int e = (int)(v.y & 0xFF);
          topk_idx[t * K + k] = e;
          topk_score[t * K + k] = sigmoid_f32(__uint_as_float((v.y >> 16) << 16));
          if (load) atomicAdd(&sh_load[e], 1u);
        }
      }
      const float tv = __uint_as_float(myrank[K].x);
      if (valid && g == 0) tau[t] = tv;

      // ---- coarse counts: raw high byte of bf16(tau - z) per expert
      if (hist && valid) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const uint32_t row = hist_row(ex(q));
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t w = (i < 2) ? raw[q].x : raw[q].y;
            const float zf = (i & 1) ? bf16_hi(w) : bf16_lo(w);
            const uint32_t hr = bf16_raw_hi(__float_as_uint(tv - zf));
            atomicAdd(&sh_hist[row + (i >> 1) * kHistStride + hr], 1u << ((i & 1) * 16));
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int q = 0; q < NQ; ++q) raw[q] = nxt[q];
    }
    __syncthreads();
    if (hist) flush_hist<E, false>(sh_hist, hist + (int64_t)p * E * kNBins, nullptr);
    if (load) {
      for (int e = threadIdx.x; e < E; e += kBlock) {
        const uint32_t c = sh_load[e];
        if (c) atomicAdd(&load[(int64_t)p * E + e], (int32_t)c);
        sh_load[e] = 0;
      }
    }
    __syncthreads();
  });
}

// ----------------------------------------------------------- generic ----
template <int E>
__global__ __launch_bounds__(kBlock) void route_generic_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ b, int64_t T, int K,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_score, float* __restrict__ tau,
    int32_t* __restrict__ load, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = E / 8;
  constexpr int R = 64 / G;
  constexpr int ROWS = kWaves * R;
  __shared__ uint32_t sh_hist[hist_words<E>()];
  __shared__ uint32_t sh_load[E];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, rr = lane / G;
  const int e0 = g * 8;
  float bb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) bb[j] = b[e0 + j];
  for (int w = threadIdx.x; w < hist_words<E>(); w += kBlock) sh_hist[w] = 0;
  for (int w = threadIdx.x; w < E; w += kBlock) sh_load[w] = 0;
  __syncthreads();

  int64_t r0, r1;
  block_rows(T, rows_per_block, &r0, &r1);
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    for (int64_t base = s0; base < s1; base += ROWS) {
      const int64_t t = base + wave * R + rr;
      const bool valid = t < s1;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (valid) v = *reinterpret_cast<const uint4*>(z + t * E + e0);
      const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
      float zf[8];
      uint64_t key[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t zb = (j & 1) ? (w4[j >> 1] >> 16) : (w4[j >> 1] & 0xFFFFu);
        zf[j] = (j & 1) ? bf16_hi(w4[j >> 1]) : bf16_lo(w4[j >> 1]);
        key[j] = exact_key(__float_as_uint(zf[j] + bb[j]), e0 + j, zb);
      }
      uint64_t prev = ~0ull;
      for (int k = 0; k <= K; ++k) {
        uint64_t m = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) m = (key[j] < prev && key[j] > m) ? key[j] : m;
        m = group_max_u64<G>(m);
        prev = m;
        if (k < K && valid && g == k % G) {
          const int e = exact_key_expert(m);   // in [0, E): the row holds E > K distinct keys
          topk_idx[t * K + k] = e;
          topk_score[t * K + k] = sigmoid_f32(__uint_as_float(exact_key_z(m) << 16));
          if (load && e >= 0 && e < E) atomicAdd(&sh_load[e], 1u);
        }
      }
      const float tv = __uint_as_float(exact_key_sbits(prev));
      if (valid && g == 0) tau[t] = tv;
      if (hist && valid) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int e = e0 + j;
          const uint32_t hr = bf16_raw_hi(__float_as_uint(tv - zf[j]));
          atomicAdd(&sh_hist[hist_row(e) + hr], hist_inc(e));
        }
      }
    }
    __syncthreads();
    if (hist) flush_hist<E, false>(sh_hist, hist + (int64_t)p * E * kNBins, nullptr);
    if (load) {
      for (int e = threadIdx.x; e < E; e += kBlock) {
        const uint32_t c = sh_load[e];
        if (c) atomicAdd(&load[(int64_t)p * E + e], (int32_t)c);
        sh_load[e] = 0;
      }
    }
    __syncthreads();
  });
}

// ------------------------------------------------------------- launch ---
template <int E>
eqb_status launch_route_e(const RouteArgs& a, hipStream_t s) {
  int blocks;
  int64_t rpb;
  if (a.K <= kFastKmax) {
    grid_for(a.T, kWaves * (64 / FastCfg<E>::G), 1, &blocks, &rpb);
    route_fast_kernel<E><<<blocks, kBlock, 0, s>>>(a.z, a.b, a.T, a.K, a.idx, a.score, a.tau, a.load,
                                                   a.hist, a.pt, rpb);
  } else {
    grid_for(a.T, kWaves * (64 / (E / 8)), 1, &blocks, &rpb);
    route_generic_kernel<E><<<blocks, kBlock, 0, s>>>(a.z, a.b, a.T, a.K, a.idx, a.score, a.tau, a.load,
                                                      a.hist, a.pt, rpb);
  }
  return launch_status();
}

eqb_status launch_route(const RouteArgs& a, hipStream_t s) {
  switch (a.E) {
    case 8: return launch_route_e<8>(a, s);
    case 16: return launch_route_e<16>(a, s);
    case 32: return launch_route_e<32>(a, s);
    case 64: return launch_route_e<64>(a, s);
    case 128: return launch_route_e<128>(a, s);
    case 256: return launch_route_e<256>(a, s);
    default: return EQB_ERR_UNSUPPORTED;
  }
}

}  // namespace eqb
