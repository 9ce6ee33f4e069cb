// route.hip - Top-K routing of z + b, cutoff tau, sigmoid scores, expert
// loads, fused with the coarse counts of Algorithm 1 step 1 (arXiv
// 2609.28053, Sec. 2 Eq. 1, "Quantile Balancing", Appendix C).
//
// Fast kernel (K <= kFastKmax).  A row of E logits is spread over G lanes,
// each holding N = E/G experts as N/4 8-byte pieces; row r of a wave visits
// its pieces in the order q XOR r, so that at any step the rows of a wave
// work on different experts (and count into different LDS words).  The
// coarse counts, two margins per BF16 conversion, go to a slot-major LDS
// histogram addressed by one byte permute.  Per element the kernel forms a
// 32-bit key: the binary32 bits of s = z + b with the low byte replaced by
// 255 - e, and keeps a sorted list of its kList largest keys (one maximum and
// kList-1 medians per element).  Keys are compared as floats, so negative
// scores order correctly; the key's sum takes -0 in b as +0, so a score of
// -0 keys as +0 and the two zeros share one run of keys.
// K+1 extraction rounds then take the group maximum of the list heads with
// DPP and pop the winner; the largest head left is rank K+1.  A lane whose
// list runs dry is refilled below its last key (generic-K variant) or, in
// the unrolled variants, scanned once for its next key, and a row whose
// rounds missed a key is extracted again with refilled lists.  Key order is
// score order except between scores that agree in their top 24 bits;
// extraction continues until the last key leaves the top-24-bit run of rank
// K, the winners' exact scores are recomputed from z and b, and a row whose
// extracted scores are not in exact order is sorted exactly.  A block whose
// bias has |b| >= 2^119 (where z + b could overflow) takes the exact 64-bit
// path for every row.
//
// Generic kernel (any K < E): K+1 rounds over exact 64-bit keys.
#include "eqb_internal.hpp"

namespace eqb {

constexpr int kRmax = 16;              // extracted ranks kept per row
// Sorted keys kept per lane.  With eight lanes per row (E >= 64) a lane
// holds five or more of a row's top K+1 keys in about one wave in fourteen
// of the large E = 256, K = 8 workload; such lanes are settled by one scan
// for their next key (below), which costs less than a sixth list level in
// every row.  Narrower rows (fewer lanes each holding a larger share of
// the top keys) keep six.
template <int E> constexpr int kListOf = E >= 64 ? 5 : 6;
constexpr int kFastKmax = kRmax - 2;
// Block of the fast kernel: 12 waves, three per SIMD, so that a wave may hold
// up to 168 VGPRs (with 16 waves the cap of 128 forces spills).
constexpr int kRouteBlock = 768;
constexpr int kRouteWaves = kRouteBlock / 64;

template <int E> struct FastCfg { static constexpr int G = E >= 64 ? 8 : E / 8; };
constexpr int kBiasPad = 32;           // words between the rotated bias copies beyond E

// The BF16 logit z of an extracted key.  The key holds the top 24 bits H of
// s = fl32(z + b) (low byte = expert index).  The candidate is
// zc = bf16(s_mid - b), with s_mid the middle of the 256-ulp interval of H;
// it is accepted when fl32(zc + b) reproduces H and |zc| * 64 >= |s_mid|.
// The second test gives exponent(zc) >= exponent(s) - 6, so the BF16
// neighbours of zc lie at least half a BF16 ulp of zc = 2^(exponent(s)-141)
// away, about 512 binary32 ulps of s: no other BF16 value maps to H, and zc
// is z.  s_mid is never zero, so the test also rejects both zeros (+0 and -0
// give the same sum, and which one z is decides the sign of a zero tau), and
// an infinite or NaN zc cannot reproduce the finite H.  *ok reports the
// tests; otherwise z must be read from memory.
__device__ __forceinline__ uint32_t z_from_key(int key, float b, bool* ok) {
  const uint32_t kb = (uint32_t)key;
  const float s_mid = __uint_as_float((kb & 0xFFFFFF00u) | 0x80u);
  const uint32_t zc = bf16x2_bits(s_mid - b, 0.0f);   // bits 16..31: bf16(+0) = 0
  const float zf = __uint_as_float(zc << 16);
  const uint32_t sc = __float_as_uint(zf + b);
  // bitwise, not short-circuit: a branch per test would cost more than it does
  *ok = ((sc ^ kb) < 256u) & (fabsf(zf) * 64.0f >= fabsf(s_mid));
  return zc;
}

// Element at a 32-bit byte offset from a (wave-uniform) base pointer: the
// form the loads and stores take as a 64-bit scalar base plus a 32-bit
// vector offset.
template <class V, class B>
__device__ __forceinline__ V& at(B* base, uint32_t byte_off) {
  return *reinterpret_cast<V*>(reinterpret_cast<char*>(const_cast<std::remove_const_t<B>*>(base)) + byte_off);
}

// Coarse counts of the fast kernel for E >= 64: a slot-major packed
// histogram.  Experts e, e+1 (e = 4j + 2h, a piece of four experts starting
// at 4j and its half h) share a word, counted in its low and high 16 bits.
// Half h lives in array h (64 KiB each); inside an array, slot 63 - j of bin
// u is word u*64 + 63 - j.  The counter's byte offset h << 16 | u << 8 |
// (252 - 4j) is assembled by one byte permute: u is the raw high byte of the
// BF16 margin, 252 - 4j is byte 3 of the piece's index bytes (255 - e for
// its four experts).  With the piece order rotated per row (below), the 64
// lanes of a wave hit 64 different slots at E = 256, so 64 different LDS
// banks.  Smaller E keep the expert-major layout of hist_row, which needs
// less LDS.
template <int E> constexpr bool kSlotHist = E >= 64;
template <int E>
constexpr int fast_hist_words() { return kSlotHist<E> ? 2 * 64 * kNBins : hist_words<E>(); }

// Adds the coarse counts of a slot-major histogram to slab [E][256] (kappa
// bins) and clears it, one pair of adjacent raw bins (words 64 apart) per
// thread and step.
template <int E>
__device__ __forceinline__ void flush_hist_slots(uint32_t* sh, int32_t* __restrict__ slab) {
  constexpr int kItems = fast_hist_words<E>() / 2;
  for (int i = threadIdx.x; i < kItems; i += blockDim.x) {
    const int it = flush_word(i, kItems);
    const int arr = it >> 13, j = (it >> 6) & 127, slot = it & 63;
    const int w0 = arr * 16384 + 2 * j * 64 + slot;
    const uint32_t c0 = sh[w0], c1 = sh[w0 + 64];
    if (c0 | c1) {
      const int e = 4 * (63 - slot) + 2 * arr;   // < E: no other slot is counted
      const bool neg = (2 * j) & 0x80;
      const int k0 = kappa_hi_of_raw(2 * j);
      if ((c0 | c1) & 0xFFFFu) add_raw_pair(slab + e * kNBins, neg, c0 & 0xFFFFu, c1 & 0xFFFFu, k0);
      if ((c0 | c1) >> 16) add_raw_pair(slab + (e + 1) * kNBins, neg, c0 >> 16, c1 >> 16, k0);
      sh[w0] = 0;
      sh[w0 + 64] = 0;
    }
  }
}

// flush_hist_slots into a slab of 16-bit counters (PartTable::slab16): an LDS
// word already holds the counts of experts e and e+1 (e = 4j + 2h) for one raw
// bin, so the item's two words (raw bins 2b, 2b+1, kappa bins k, k+1 or k, k-1)
// are four adjacent 16-bit counters of the slab, added with one 64-bit atomic.
// The host uses it only where no counter can pass 65,535 (no carry between
// the fields).
template <int E>
__device__ __forceinline__ void flush_hist_slots16(uint32_t* sh, int32_t* __restrict__ slab32) {
  constexpr int kItems = fast_hist_words<E>() / 2;
  uint16_t* slab = reinterpret_cast<uint16_t*>(slab32);
  for (int i = threadIdx.x; i < kItems; i += blockDim.x) {
    const int it = flush_word(i, kItems);
    const int arr = it >> 13, j = (it >> 6) & 127, slot = it & 63;
    const int w0 = arr * 16384 + 2 * j * 64 + slot;
    const uint32_t c0 = sh[w0], c1 = sh[w0 + 64];
    if (c0 | c1) {
      const int m = 2 * (63 - slot) + arr;   // the pair of experts 2m, 2m+1
      const bool neg = (2 * j) & 0x80;
      const int k0 = kappa_hi_of_raw(2 * j);  // even, or odd (flipped) for negative bins
      const int k = neg ? k0 - 1 : k0;
      const uint64_t v = neg ? ((uint64_t)c1 | ((uint64_t)c0 << 32)) : ((uint64_t)c0 | ((uint64_t)c1 << 32));
      atomicAdd(reinterpret_cast<unsigned long long*>(slab + ((int64_t)m * kNBins + k) * 2),
                (unsigned long long)v);
      sh[w0] = 0;
      sh[w0 + 64] = 0;
    }
  }
}

// The histogram byte offset of half 1 of a piece: byte 3 of its index bytes
// to byte 0, 1 to byte 2.  Volatile so that it is formed where it is used
// rather than kept in a register per piece.
__device__ __forceinline__ uint32_t half1_base(uint32_t ipk, uint32_t one16) {
  uint32_t r;
  asm volatile("v_perm_b32 %0, %1, %2, %3" : "=v"(r) : "v"(one16), "v"(ipk), "s"(0x0C060C03u));
  return r;
}

// Insert key x into the sorted list L[0] >= ... >= L[n-1] (one max, n-1 med3).
template <int n>
__device__ __forceinline__ void list_insert(int (&L)[n], int x) {
#pragma unroll
  for (int j = n - 1; j > 0; --j) L[j] = key_med3(L[j - 1], L[j], x);
  L[0] = key_max(L[0], x);
}

template <int E, int KT>
__global__ __launch_bounds__(kRouteBlock) void route_fast_kernel(
    const uint16_t* __restrict__ z, const float* __restrict__ b, int64_t T, int Kdyn,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_score, float* __restrict__ tau,
    int32_t* __restrict__ load, int32_t* __restrict__ hist, const PartTable pt,
    int64_t rows_per_block) {
  constexpr int G = FastCfg<E>::G;      // lanes per row
  constexpr int N = E / G;              // experts per lane
  constexpr int NQ = N / 4;             // 8-byte pieces per lane and row
  constexpr int R = 64 / G;             // rows per wave
  constexpr int ROWS = kRouteWaves * R;      // rows per block step
  constexpr int RSLOT = (kRmax + G - 1) / G;
  static_assert(N % 4 == 0 && N >= 8, "layout");
  static_assert(KT == 0 || KT + 2 <= E, "K+2 keys must exist");
  constexpr int kList = kListOf<E>;
  const int K = KT > 0 ? KT : Kdyn;

  __shared__ __align__(16) uint32_t sh_hist[fast_hist_words<E>()];
  __shared__ uint32_t sh_load[E];
  __shared__ float sh_b[E];             // b as given: exact scores and tau
  // b with -0 as +0 (the keys' sums), one copy per piece rotation.  Copies
  // sit E + 32 words apart: the rows of a wave read their rotations' copies
  // with one 16-byte read per lane, and copies E words apart (a multiple of
  // the 64 banks) would put every row's reads on the same 32 banks.
  __shared__ float sh_bk[NQ][E + kBiasPad];
  __shared__ uint2 sh_rank[kRouteWaves][R][kRmax];   // (score bits, zbits << 16 | e) in rank order
  __shared__ int sh_pool_spent;                       // the group's pool has run out (pool mode)

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane % G, r = lane / G;
  // Row r of a wave visits its pieces in the order q ^ rr, so at any step the
  // rows of a wave work on different experts (distinct histogram slots).
  const int rr = r & (NQ - 1);

  // Step q of this lane covers experts ex(q) .. ex(q)+3 (piece q ^ rr), so the
  // G lanes of a row read 8*G contiguous bytes per step.  b is read from LDS,
  // four experts at a time (bias4: the keys' copy, bias4x: b as given); the
  // keys' copy is kept once per rotation, sh_bk[c][j] = b[j ^ 4Gc], so that a
  // lane reads its step q at a fixed offset from its own base.
  auto ex = [&](int q) -> int { return (q ^ rr) * 4 * G + g * 4; };
  // bytes 255 - e for the four experts of a piece (ex is a multiple of 4, no borrow)
  auto idxpk = [&](int q) -> uint32_t { return 0xFCFDFEFFu - (uint32_t)ex(q) * 0x01010101u; };
  auto bias4 = [&](int q) -> float4 { return *reinterpret_cast<const float4*>(&sh_bk[rr][q * 4 * G + g * 4]); };
  auto bias4x = [&](int q) -> float4 { return *reinterpret_cast<const float4*>(&sh_b[ex(q)]); };
  auto pick = [](const float4& v, int i) -> float { return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w; };

  // Rows of one step of a segment starting at zb and holding n rows: row
  // base + wave * R + r of the segment, a row past its end reading the last
  // row instead (processed as invalid: no output, no count).  Byte offsets
  // stay below 2^25; the piece index occupies bits that the row and lane
  // parts leave clear, so XOR selects piece q ^ rr.
  auto load_rows = [&](uint2 (&dst)[NQ], const uint16_t* zb, uint32_t wbase, uint32_t n) {
    uint32_t t = wbase + r;
    t = t < n ? t : n - 1;
    const uint32_t off = (t * (uint32_t)E + (uint32_t)g * 4u) * 2u + (uint32_t)rr * (8u * G);
#pragma unroll
    for (int q = 0; q < NQ; ++q) dst[q] = at<uint2>(zb, off ^ ((uint32_t)q * (8u * G)));
  };
  auto load_step = [&](uint2 (&dst)[NQ], const uint16_t* zb, uint32_t base, uint32_t n) {
    load_rows(dst, zb, base + wave * R, n);
  };

  // The first step of the block's first segment (as for_each_segment will
  // cut it) is loaded before the LDS set-up, so that its latency passes while
  // the histogram is zeroed and the bias is staged.
  const BlockPlan plan = block_plan(pt, T, rows_per_block);
  const int64_t r0 = plan.r0, r1 = plan.r1;
  const int64_t seg_max = plan.pool ? kSegPool : kSegMax;
  uint2 buf[NQ];
  if (r0 < r1) {
    int p = 0;
    while (p < pt.P - 1 && pt.off[p + 1] <= r0) ++p;
    int64_t end = pt.off[p + 1] < r1 ? pt.off[p + 1] : r1;
    if (end - r0 > seg_max) end = r0 + seg_max;
    load_step(buf, z + wave_uniform(r0) * E, 0, (uint32_t)(end - r0));
  }

  static_assert(fast_hist_words<E>() % 4 == 0, "16-byte zeroing");
  for (int w = threadIdx.x; w < fast_hist_words<E>() / 4; w += kRouteBlock)
    reinterpret_cast<uint4*>(sh_hist)[w] = make_uint4(0, 0, 0, 0);
  int fits = 1, bzero = 1;
  if (threadIdx.x == 0) sh_pool_spent = 0;
  for (int e = threadIdx.x; e < E; e += kRouteBlock) {
    sh_load[e] = 0;
    const float bv = b[e];
    sh_b[e] = bv;
    const float bk = (__float_as_uint(bv) == 0x80000000u) ? 0.0f : bv;
#pragma unroll
    for (int c = 0; c < NQ; ++c) sh_bk[c][e ^ (c * 4 * G)] = bk;
    fits &= (int)(fabsf(bv) < 0x1p119f);
    bzero &= (int)(bk == 0.0f);
  }
  // |z| <= 2^128 - 2^120 for a finite BF16 z, so with |b| < 2^119 every sum
  // z + b is finite and every key is a finite float.
  const bool bias_ok = __syncthreads_and(fits) != 0;
  // With a zero bias (the starting point of the balancing loop) every score
  // is a BF16 logit, so keys that agree in their top 24 bits hold equal
  // scores (for scores of either sign the index byte then orders them by
  // magnitude: lower index first for non-negative scores, last for negative
  // ones).
  const bool keys_exact = __syncthreads_and(bzero) != 0;

  uint2* myrank = sh_rank[wave][r];

  // key of element (q, i) from its widened logit
  auto key_of = [&](float zf, float bv, uint32_t ipk, int i) -> int {
    const uint32_t sb = __float_as_uint(zf + bv);
    return (int)__builtin_amdgcn_perm(sb, ipk, 0x07060500u | (uint32_t)i);
  };

  // Rebuild a lane's sorted list from its keys strictly below thr.
  auto rebuild = [&](const float (&zf)[N], int thr, int (&L)[kList]) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kList; ++j) L[j] = kKeyNone;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float4 bq = bias4(q);
      const uint32_t ipk = idxpk(q);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int x = key_of(zf[q * 4 + i], pick(bq, i), ipk, i);
        list_insert(L, key_lt(x, thr) ? x : kKeyNone);
      }
    }
  };

  // Base pointers of the current segment (at most kSegMax rows): rows are
  // addressed by a 32-bit offset from them, which the loads and stores take
  // directly next to a wave-uniform 64-bit base.
  const uint16_t* seg_z = z;
  int32_t* seg_idx = topk_idx;
  float* seg_score = topk_score;
  float* seg_tau = tau;

  // t: row index inside the current segment
  // raw holds this step's logits (loaded one step earlier); once they are
  // widened, refill(raw) issues the next step's loads into the same registers.
  // exact: std::true_type when the block's keys are exact (zero bias)
  auto process = [&](auto exact, uint2 (&raw)[NQ], uint32_t t, bool valid, auto&& refill)
                     __attribute__((always_inline)) {
    // ---- widen the logits once; build keys and the per-lane sorted list
    float4 bq = bias4(0);   // read first: its LDS latency passes during the widening
    float zf[N];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      zf[q * 4 + 0] = bf16_lo(raw[q].x);
      zf[q * 4 + 1] = bf16_hi(raw[q].x);
      zf[q * 4 + 2] = bf16_lo(raw[q].y);
      zf[q * 4 + 3] = bf16_hi(raw[q].y);
    }
    refill(raw);
    int L[kList];
#pragma unroll
    for (int j = 0; j < kList; ++j) L[j] = kKeyNone;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      // The next piece's bias is read while this piece is inserted; the
      // scheduling barrier keeps the compiler from sinking the read to its use.
      float4 bn = bq;
      if (q + 1 < NQ) bn = bias4(q + 1);
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t ipk = idxpk(q);
#pragma unroll
      for (int i = 0; i < 4; ++i) list_insert(L, key_of(zf[q * 4 + i], pick(bq, i), ipk, i));
      bq = bn;
    }

    // ---- extraction rounds: group maximum of the list heads, winner pops
    auto pop = [&](int M) {
      const bool win = (L[0] == M);
#pragma unroll
      for (int j = 0; j < kList - 1; ++j) L[j] = win ? L[j + 1] : L[j];
      L[kList - 1] = win ? kKeyNone : L[kList - 1];
    };
    // Rows whose ranks are staged in LDS: run past rank K+1, equal top-24-bit
    // keys or a list that ran dry; (slow) rows the keys cannot settle.
    bool staged = false, slow = false;
    int nrank = 0;
    float tv = 0.0f;          // tau of this lane's row (common rows)
    int rk[RSLOT];
    uint32_t zown[RSLOT];
#pragma unroll
    for (int s = 0; s < RSLOT; ++s) {
      rk[s] = kKeyNone;
      zown[s] = 0;
    }

    if constexpr (KT > 0) {
      int mK = kKeyNone, prev = kKeyNone;
      bool near = false;      // two adjacent extracted keys share their top 24 bits
      const int tail = L[kList - 1];   // the smallest key a lane can pop
#pragma unroll
      for (int k = 0; k <= KT; ++k) {
        const int M = group_max_key<G>(L[0]);
        pop(M);
        rk[k / G] = (g == k % G) ? M : rk[k / G];
        if (k > 0) near |= ((uint32_t)(M ^ prev) < 256u);
        prev = M;
        if (k == KT) mK = M;
      }
      // Rank K+1 is the largest list head left.  Whether it shares the top 24
      // bits of rank K is read off the heads directly; the rest of each list
      // is not needed past this point (a row that extends its run rebuilds
      // its lists), so the last rounds' pops only shift the entries that
      // later rounds read.
      // A lane whose list ran dry popped all of its kList keys and has no
      // head: its next key is the largest of its keys below the last one it
      // popped, found by one scan of its logits.  If that key ranks above
      // rank K, the rounds missed it and the row is extracted again; if not,
      // it is the lane's head.  A head of -inf (no key left) never matches:
      // no finite key has the top 24 bits of -inf.
      int hk = L[0];
      bool missed = false;
      if (__builtin_expect(__any(L[0] == kKeyNone), 0)) {
        const bool dry_lane = L[0] == kKeyNone;
        int nxt = kKeyNone;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const float4 bq = bias4(q);
          const uint32_t ipk = idxpk(q);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int x = key_of(zf[q * 4 + i], pick(bq, i), ipk, i);
            nxt = key_lt(x, tail) ? key_max(nxt, x) : nxt;
          }
        }
        hk = dry_lane ? nxt : hk;
        missed = dry_lane && key_lt(mK, nxt);
      }
      const int head = ((uint32_t)(hk ^ mK) < 256u) ? 1 : 0;
      const int rowflag = group_max_i32<G>(missed ? 2 : head);
      // z of the experts at this lane's ranks, recovered from their keys.
      // Every slot's bias is read before any is used, so the LDS latency is
      // paid once; one wave-wide test sends the failed recoveries to memory.
      int es[RSLOT];
      bool use[RSLOT], ok[RSLOT];
      float bks[RSLOT];
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        use[s] = valid && s * G + g <= KT;
        // below E for every key of the row; the clamp keeps a row whose
        // keys cannot be trusted (it goes slow) inside its own logits
        es[s] = use[s] ? min(255 - (rk[s] & 0xFF), E - 1) : 0;
        bks[s] = sh_bk[0][es[s]];
      }
      bool bad = false;
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        zown[s] = z_from_key(rk[s], bks[s], &ok[s]);
        ok[s] = ok[s] | !use[s];
        bad = bad | !ok[s];
      }
      if (__builtin_expect(__any(bad), 0)) {
        // The few failed recoveries are read one lane at a time with scalar
        // loads: their wait does not include the vector loads of the next
        // step, which are still in flight (vector loads complete in order, so
        // a vector fallback load would wait for all of them).
#pragma unroll
        for (int s = 0; s < RSLOT; ++s) {
          const uint32_t off = (t * (uint32_t)E + (uint32_t)es[s]) * 2u;   // < 2^25
          uint32_t zl = zown[s];
          uint64_t need = __ballot(!ok[s]);
          while (need) {
            const int l = __builtin_ctzll(need);
            const uint32_t o = __builtin_amdgcn_readlane(off, l);
            // the aligned word holding z (seg_z is 16-byte aligned)
            const uint32_t w = at<const uint32_t>(seg_z, o & ~3u);
            if (lane == l) zl = (w >> ((o & 2u) * 8u)) & 0xFFFFu;
            need &= need - 1;
          }
          zown[s] = zl;
        }
      }
      const int tauhi = mK >> 8;
      const bool dry = rowflag == 2;   // the rounds missed a key of a dry lane
      slow = valid && !bias_ok;
      staged = valid && !slow && (near || rowflag != 0);
      nrank = KT + 1;
      // A row is staged when adjacent ranks' keys agree in their top 24 bits
      // (their order may be wrong) or the run of rank K's top 24 bits
      // continues past it.  With exact keys such keys hold equal scores, and
      // for a non-negative rank K (every rank at or above it non-negative)
      // the index byte already orders them as the exact order does: only a
      // missed key needs the staged path.
      if constexpr (decltype(exact)::value) staged = staged && (dry || mK < 0);
      if (__builtin_expect(__any(staged), 0)) {
        // stage the keys, extend the run of rank K if it continues, then exact scores
#pragma unroll
        for (int s = 0; s < RSLOT; ++s) {
          const int k = s * G + g;
          if (staged && k <= KT) myrank[k].x = (uint32_t)rk[s];
        }
        // the keys past rank K are taken from lists rebuilt below mK, while
        // they share the top 24 bits of rank K
        bool ext = staged && rowflag == 1;
        bool bad = false;           // row-uniform: extraction can no longer be trusted
        if (__any(ext)) {
          rebuild(zf, mK, L);
          for (int k = KT + 1; k < kRmax; ++k) {
            if (!__any(ext)) break;
            // a lane whose list ran dry may hold the next key
            const bool dry_now = group_max_i32<G>((int)(L[0] == kKeyNone)) != 0;
            if (ext && dry_now) {
              bad = true;
              ext = false;
            }
            const int M = group_max_key<G>(L[0]);
            if (ext) {
              if (g == 0) myrank[k].x = (uint32_t)M;
              nrank = k + 1;
              if ((M >> 8) != tauhi) ext = false;
            }
            pop(M);
          }
        }
        bad = bad || ext;           // the run is longer than the rank buffer
        // Rows whose rounds missed a key (a lane held more of the top K+1
        // keys than its list) redo the extraction from fresh lists, refilling
        // a lane's list below its last key whenever it runs dry again (as the
        // generic-K loop does); only a run longer than the rank buffer still
        // goes to the exact 64-bit path.
        bool redo = staged && dry;
        if (__any(redo)) {
          if (redo) rebuild(zf, kKeyTop, L);
          bool done = !redo;
          int th = 0;
#pragma unroll 1
          for (int k = 0; k < kRmax; ++k) {
            if (!__any(!done)) break;
            const int M = group_max_key<G>(L[0]);
            pop(M);
            const bool dl = (L[0] == kKeyNone) && (M != kKeyNone);
            if (__any(dl && !done)) {
              if (dl && !done) rebuild(zf, M, L);
            }
            if (!done) {
              if (M == kKeyNone) {
                done = true;
              } else {
                if (g == 0) myrank[k].x = (uint32_t)M;
                nrank = k + 1;
                if (k == K) th = M >> 8;
                if (k > K && (M >> 8) != th) done = true;   // one key past the run of rank K
              }
            }
          }
          bad = bad || !done;
        }
        slow = slow || bad;
        staged = staged && !slow;
        lds_wave_sync();
#pragma unroll
        for (int s = 0; s < RSLOT; ++s) {
          const int k = s * G + g;
          if (staged && k < nrank) {
            const int key = (int)myrank[k].x;
            const int e = 255 - (key & 0xFF);
            bool ok;
            uint32_t zb = z_from_key(key, sh_bk[0][e], &ok);
            if (!ok) zb = seg_z[t * E + e];
            const uint32_t sb = __float_as_uint(__uint_as_float(zb << 16) + sh_b[e]);
            myrank[k] = make_uint2(sb, (zb << 16) | (uint32_t)e);
          }
        }
        lds_wave_sync();
      }
    } else {
      bool done = !valid;
      int tauhi = 0;
#pragma unroll 1
      for (int k = 0; k < kRmax; ++k) {
        if (!__any(!done)) break;
        const int M = group_max_key<G>(L[0]);
        pop(M);
        const bool dry = (L[0] == kKeyNone) && (M != kKeyNone);
        if (__any(dry && !done)) {
          if (dry && !done) rebuild(zf, M, L);
        }
        if (!done) {
          if (M == kKeyNone) {
            done = true;
          } else {
            if (g == 0) myrank[k].x = (uint32_t)M;
            nrank = k + 1;
            if (k == K) tauhi = M >> 8;
            if (k > K && (M >> 8) != tauhi) done = true;   // one key past the run of rank K
          }
        }
      }
      slow = valid && (!done || !bias_ok);
      staged = valid && !slow;
      lds_wave_sync();
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (staged && k < nrank) {
          const int e = 255 - (int)(myrank[k].x & 0xFF);
          const uint32_t zb = seg_z[t * E + e];
          const uint32_t sb = __float_as_uint(__uint_as_float(zb << 16) + sh_b[e]);
          myrank[k] = make_uint2(sb, (zb << 16) | (uint32_t)e);
        }
      }
      lds_wave_sync();
    }

    // ---- staged rows: sort the extracted ranks exactly where key order and
    // exact order differ (only inside a run of equal top-24-bit keys)
    // rank order of two staged entries: higher score, then lower expert
    auto before = [](uint2 a, uint2 c) -> bool {
      const float fa = __uint_as_float(a.x), fc = __uint_as_float(c.x);
      return fa > fc || (fa == fc && (a.y & 0xFF) < (c.y & 0xFF));
    };
    if (__builtin_expect(__any(staged), 0)) {
      bool coll = false;
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (staged && k + 1 < nrank) coll |= !before(myrank[k], myrank[k + 1]);
      }
      const bool coll_row = group_max_i32<G>((int)coll) != 0;
      if (coll_row && g == 0) {
        for (int i = 1; i < nrank; ++i) {
          const uint2 v = myrank[i];
          int j = i - 1;
          while (j >= 0) {
            const uint2 u = myrank[j];
            if (!before(v, u)) break;
            myrank[j + 1] = u;
            --j;
          }
          myrank[j + 1] = v;
        }
      }
      lds_wave_sync();
    }

    // ---- exact 64-bit extraction for rows flagged slow
    if (__builtin_expect(__any(slow), 0)) {
      if (slow) {
        uint64_t prevk = ~0ull;
        for (int k = 0; k <= K; ++k) {
          uint64_t m = 0;
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            const float4 bq = bias4x(q);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              // rebuilt every round instead of being held in 2*N registers
              float zq = zf[q * 4 + i];
              asm volatile("" : "+v"(zq));
              const uint32_t zb = __float_as_uint(zq) >> 16;
              const uint32_t sb = __float_as_uint(zq + pick(bq, i));
              const uint64_t key = exact_key(sb, ex(q) + i, zb);
              m = (key < prevk && key > m) ? key : m;
            }
          }
          m = group_max_u64<G>(m);
          prevk = m;
          if (g == 0)
            myrank[k] = make_uint2(exact_key_sbits(m), (exact_key_z(m) << 16) | (uint32_t)exact_key_expert(m));
        }
      }
      lds_wave_sync();
    }

    // ---- outputs: ranks 0..K-1, loads, tau
    const bool fromlds = staged || slow;
    if (KT > 0 && valid && !fromlds) {
      // rank k is held by lane k % G in slot k / G; its exact score is z + b of that expert
      float tk = 0.0f;
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (k <= K) {
          const int e = 255 - (rk[s] & 0xFF);
          const uint32_t zb = zown[s];
          if (k < K) {
            at<int32_t>(seg_idx, (t * K + k) * 4u) = e;
            at<float>(seg_score, (t * K + k) * 4u) = sigmoid_fast(__uint_as_float(zb << 16));
            if (load) atomicAdd(&sh_load[e], 1u);
          } else {
            tk = __uint_as_float(zb << 16) + sh_b[e];
          }
        }
      }
      tv = tk;
    }
    if constexpr (KT > 0) {
      // every lane of the row takes tau from the lane holding rank K
      tv = group_bcast<G, KT % G>(tv, g);
    }
    if (valid && fromlds) {
#pragma unroll
      for (int s = 0; s < RSLOT; ++s) {
        const int k = s * G + g;
        if (k < K) {
          const uint2 v = myrank[k];
          const int e = (int)(v.y & 0xFF);
          at<int32_t>(seg_idx, (t * K + k) * 4u) = e;
          at<float>(seg_score, (t * K + k) * 4u) = sigmoid_fast(__uint_as_float((v.y >> 16) << 16));
          if (load) atomicAdd(&sh_load[e], 1u);
        }
      }
      tv = __uint_as_float(myrank[K].x);
    }
    if (valid && g == 0) at<float>(seg_tau, t * 4u) = tv;

    // ---- coarse counts: raw high byte of bf16(tau - z), two margins per conversion
    if (hist && valid) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t p = bf16x2_bits(tv - zf[q * 4 + 2 * h], tv - zf[q * 4 + 2 * h + 1]);
          if constexpr (kSlotHist<E>) {
            // byte offsets: the raw high byte of either margin becomes byte 1
            if (h == 0) {
              const uint32_t ipk = idxpk(q);
              atomicAdd(&at<uint32_t>(sh_hist, __builtin_amdgcn_perm(ipk, p, 0x0C0C0107u)), 1u);
              atomicAdd(&at<uint32_t>(sh_hist, __builtin_amdgcn_perm(ipk, p, 0x0C0C0307u)), 1u << 16);
            } else {
              const uint32_t base = half1_base(idxpk(q), 0x10000u);
              atomicAdd(&at<uint32_t>(sh_hist, __builtin_amdgcn_perm(base, p, 0x0C060104u)), 1u);
              atomicAdd(&at<uint32_t>(sh_hist, __builtin_amdgcn_perm(base, p, 0x0C060304u)), 1u << 16);
            }
          } else {
            const uint32_t row = hist_row(ex(q)) + h * kHistStride;
            atomicAdd(&sh_hist[row + ((p >> 8) & 0xFFu)], 1u);
            atomicAdd(&sh_hist[row + (p >> 24)], 1u << 16);
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  };

  // The sweep is compiled twice, for exact keys (a zero bias) and for any
  // bias, so that neither carries the other's test in its per-row path.
  auto set_base = [&](int64_t s0) {
    const int64_t su = wave_uniform(s0);
    seg_z = z + su * E;
    seg_idx = topk_idx + su * K;
    seg_score = topk_score + su * K;
    seg_tau = tau + su;
  };
  // Adds the block's LDS counts (coarse bins, loads) of partition p to global
  // memory and clears them.
  auto flush_counts = [&](int p) {
    __syncthreads();
    if (hist) {
      if constexpr (kSlotHist<E>) {
        if (pt.slab16) flush_hist_slots16<E>(sh_hist, count_slab(hist, pt, p, E));
        else flush_hist_slots<E>(sh_hist, count_slab(hist, pt, p, E));
      } else {
        flush_hist<E, false>(sh_hist, count_slab(hist, pt, p, E), nullptr);
      }
    }
    if (load) {
      for (int e = threadIdx.x; e < E; e += kRouteBlock) {
        const uint32_t c = sh_load[e];
        if (c) atomicAdd(&load[(int64_t)p * E + e], (int32_t)c);
        sh_load[e] = 0;
      }
    }
    __syncthreads();
  };
  auto sweep = [&](auto exact) __attribute__((always_inline)) {
  bool first = true;
  for_each_segment(r0, r1, pt, [&](int p, int64_t s0, int64_t s1) {
    set_base(s0);
    const uint32_t n = (uint32_t)(s1 - s0);
    // The next step's loads are in flight while a step is processed: a step
    // widens the rows loaded one step earlier and then reuses their registers
    // for the next step's loads, so the only wait is for loads issued a whole
    // step before.  The last step also loads (the segment's last row, clamped
    // in load_step), which keeps the loads unconditional: the registers then
    // carry over to the next step without copies.  The first segment's first
    // step was loaded before the LDS set-up.
    if (!first) load_step(buf, seg_z, 0, n);
    first = false;
    for (uint32_t base = 0; base < n; base += ROWS) {
      const uint32_t t = base + wave * R + r;
      process(exact, buf, t, t < n, [&](uint2 (&dst)[NQ]) { load_step(dst, seg_z, base + ROWS, n); });
    }
    // in pool mode the last static segment's counts are flushed with the pool's
    if (!(plan.pool && s1 == r1)) flush_counts(p);
  }, seg_max);
  if (plan.pool) {
    // The group's pool, claimed by single waves in chunks of kChunk rows
    // (kChunkSteps wave steps).  A wave claims its next chunk when it starts
    // one and reads the claim at the start of the chunk's last step, whose
    // refill loads the next chunk's first rows; that read waits only for
    // loads the step waits for anyway.  A wave that draws past the pool
    // marks it spent in LDS, and the block's other waves then stop claiming.
    constexpr uint32_t kChunkSteps = 8;
    constexpr uint32_t kChunk = (uint32_t)R * kChunkSteps;
    set_base(plan.q0);
    const uint32_t nq = (uint32_t)(plan.q1 - plan.q0);
    const uint32_t nchunks = (nq + kChunk - 1) / kChunk;
    int32_t* ctr = pt.pool + (int64_t)plan.ctr * kPoolStride;
    volatile int* spent = &sh_pool_spent;
    auto claim = [&]() -> uint32_t {
      uint32_t v = nchunks;
      if (lane == 0 && *spent == 0) v = (uint32_t)atomicAdd(ctr, 1);
      return v;
    };
    auto take = [&](uint32_t v) -> uint32_t {
      const uint32_t c = __builtin_amdgcn_readfirstlane(v);
      if (c >= nchunks && lane == 0) *spent = 1;
      return c;
    };
    uint32_t c = take(claim());
    uint32_t pend = nchunks;
    if (c < nchunks) {
      load_rows(buf, seg_z, c * kChunk, nq);
      pend = claim();
    }
    while (c < nchunks) {
      uint32_t cn = nchunks;
#pragma unroll 1
      for (uint32_t j = 0; j < kChunkSteps; ++j) {
        const uint32_t wbase = c * kChunk + j * (uint32_t)R;
        uint32_t next = wbase + (uint32_t)R;
        if (j + 1 == kChunkSteps) {
          cn = take(pend);
          next = cn < nchunks ? cn * kChunk : wbase;
        }
        const uint32_t t = wbase + r;
        process(exact, buf, t, t < nq, [&](uint2 (&dst)[NQ]) { load_rows(dst, seg_z, next, nq); });
      }
      c = cn;
      if (c < nchunks) pend = claim();
    }
    flush_counts(plan.p);
  }
  };
  if (keys_exact) sweep(std::true_type{});
  else sweep(std::false_type{});
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
    if (hist) flush_hist<E, false>(sh_hist, count_slab(hist, pt, p, E), nullptr);
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
// Dynamic tails only for blocks of at least this many block steps: on
// shorter ranges the pool's claims cost more than the tail they remove
// (E = 128 with 4,096 rows per block: 3% slower; E = 256 with 16,384: 2%
// faster).
constexpr int64_t kPoolMinSteps = 64;

template <int E, int KT>
void launch_fast(const RouteArgs& a, hipStream_t s, bool* slab16_used) {
  int blocks;
  int64_t rpb;
  grid_for(a.T, kRouteWaves * (64 / FastCfg<E>::G), 1, &blocks, &rpb);
  PartTable pt = pool_table(a.pt, a.T, blocks, kPoolMinSteps * kRouteWaves * (64 / FastCfg<E>::G));
  pt.slab16 = (kSlotHist<E> && a.hist != nullptr && a.slab16_ok && pt.pool == nullptr &&
               slab_rows_bound(pt, rpb) <= kSegMax) ? 1 : 0;
  if (slab16_used) *slab16_used = pt.slab16 != 0;
  route_fast_kernel<E, KT><<<blocks, kRouteBlock, 0, s>>>(a.z, a.b, a.T, a.K, a.idx, a.score, a.tau, a.load,
                                                     a.hist, pt, rpb);
}

template <int E>
eqb_status launch_route_e(const RouteArgs& a, hipStream_t s, bool* slab16_used) {
  if (slab16_used) *slab16_used = false;
  if (a.K <= kFastKmax) {
    // the common MoE fan-outs get a kernel with the rounds unrolled
    if constexpr (E >= 64) {
      switch (a.K) {
        case 1: launch_fast<E, 1>(a, s, slab16_used); return launch_status();
        case 2: launch_fast<E, 2>(a, s, slab16_used); return launch_status();
        case 4: launch_fast<E, 4>(a, s, slab16_used); return launch_status();
        case 6: launch_fast<E, 6>(a, s, slab16_used); return launch_status();
        case 8: launch_fast<E, 8>(a, s, slab16_used); return launch_status();
        default: break;
      }
    }
    launch_fast<E, 0>(a, s, slab16_used);
  } else {
    int blocks;
    int64_t rpb;
    grid_for(a.T, kWaves * (64 / (E / 8)), 1, &blocks, &rpb);
    PartTable pt = a.pt;
    pt.pool = nullptr;   // static ranges only
    route_generic_kernel<E><<<blocks, kBlock, 0, s>>>(a.z, a.b, a.T, a.K, a.idx, a.score, a.tau, a.load,
                                                      a.hist, pt, rpb);
  }
  return launch_status();
}

eqb_status launch_route(const RouteArgs& a, hipStream_t s, bool* slab16_used) {
  switch (a.E) {
    case 8: return launch_route_e<8>(a, s, slab16_used);
    case 16: return launch_route_e<16>(a, s, slab16_used);
    case 32: return launch_route_e<32>(a, s, slab16_used);
    case 64: return launch_route_e<64>(a, s, slab16_used);
    case 128: return launch_route_e<128>(a, s, slab16_used);
    case 256: return launch_route_e<256>(a, s, slab16_used);
    default: return EQB_ERR_UNSUPPORTED;
  }
}

}  // namespace eqb
