// Device building blocks shared by the Prof-K kernels (gfx950, wave64).
//
//  * order-preserving keys (the total order every result is defined under);
//  * Philox4x64-10 (Salmon et al., SC'11) for the sample draws of stage 1;
//  * block-wide scans, an LDS radix select and an LDS bitonic sort used by
//    the threshold step (stage 2) and the exact refinement (stage 4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace profk {

constexpr int kWave = 64;

// ---------------------------------------------------------------- keys ----
// fp32: flip every bit of a negative pattern, set the sign bit otherwise, so
// unsigned key order is -NaN < -inf < ... < -0 < +0 < ... < +inf < +NaN.
__device__ __forceinline__ uint32_t key_f32(uint32_t u) {
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ uint32_t bits_from_key_f32(uint32_t k) {
  return (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
}
// bf16: the same rule on 16 bits; keys live in the low half of a uint32.
__device__ __forceinline__ uint32_t key_bf16(uint32_t h) {
  return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
}
__device__ __forceinline__ uint32_t bits_from_key_bf16(uint32_t k) {
  return (k & 0x8000u) ? (k & 0x7FFFu) : (~k & 0xFFFFu);
}

template <int DT> __device__ __forceinline__ uint32_t key_of(uint32_t raw);
template <> __device__ __forceinline__ uint32_t key_of<0>(uint32_t raw) { return key_f32(raw); }
template <> __device__ __forceinline__ uint32_t key_of<1>(uint32_t raw) { return key_bf16(raw); }
template <int DT> __device__ __forceinline__ uint32_t bits_of_key(uint32_t k);
template <> __device__ __forceinline__ uint32_t bits_of_key<0>(uint32_t k) { return bits_from_key_f32(k); }
template <> __device__ __forceinline__ uint32_t bits_of_key<1>(uint32_t k) { return bits_from_key_bf16(k); }

template <int DT> __device__ __forceinline__ uint32_t load_raw(const void* base, uint32_t i);
template <> __device__ __forceinline__ uint32_t load_raw<0>(const void* base, uint32_t i) {
  return static_cast<const uint32_t*>(base)[i];
}
template <> __device__ __forceinline__ uint32_t load_raw<1>(const void* base, uint32_t i) {
  return static_cast<const uint16_t*>(base)[i];
}

// ------------------------------------------------------------- philox ----
// Philox4x64-10: four 64-bit counter words, two 64-bit key words; each round
// multiplies words 0 and 2 by fixed odd constants and mixes the 128-bit
// products' halves with words 1, 3 and the key; the key advances by Weyl
// constants between rounds.
struct U64x4 { uint64_t w[4]; };

__device__ __forceinline__ U64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                               uint64_t c3, uint64_t k0, uint64_t k1) {
  constexpr uint64_t kMulA = 0xD2E7470EE14C6C93ull;
  constexpr uint64_t kMulB = 0xCA5A826395121157ull;
  constexpr uint64_t kWeyl0 = 0x9E3779B97F4A7C15ull;
  constexpr uint64_t kWeyl1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += kWeyl0; k1 += kWeyl1; }
    const uint64_t hi_a = __umul64hi(kMulA, c0), lo_a = kMulA * c0;
    const uint64_t hi_b = __umul64hi(kMulB, c2), lo_b = kMulB * c2;
    const uint64_t n0 = hi_b ^ c1 ^ k0, n2 = hi_a ^ c3 ^ k1;
    c0 = n0; c1 = lo_b; c2 = n2; c3 = lo_a;
  }
  U64x4 o; o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
  return o;
}

// Sample index from a 64-bit draw: floor(u * N / 2^64).
__device__ __forceinline__ uint32_t index_of_word(uint64_t u, uint64_t n) {
  return static_cast<uint32_t>(__umul64hi(u, n));
}

// ------------------------------------------------------------- scans ------
// Inclusive prefix sum over the lanes of a wave, in lane order, by DPP:
// shifts right by 1, 2, 4 and 8 lanes within each 16-lane row (lanes with no
// source add 0) give each row's own prefix sums; a broadcast of lane 15 into
// rows 1 and 3, then of lane 31 into rows 2 and 3, adds the rows below.
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Wave-wide maximum, uniform result: DPP exchanges inside each 16-lane row
// (quad swaps, half-row and row mirrors), then the four row results are read
// into scalars.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xB1, 0xF, 0xF, false)));
  x = max(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4E, 0xF, 0xF, false)));
  x = max(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x141, 0xF, 0xF, false)));
  x = max(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x140, 0xF, 0xF, false)));
  const uint32_t r0 = __builtin_amdgcn_readlane(static_cast<int>(x), 0);
  const uint32_t r1 = __builtin_amdgcn_readlane(static_cast<int>(x), 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(static_cast<int>(x), 32);
  const uint32_t r3 = __builtin_amdgcn_readlane(static_cast<int>(x), 48);
  return max(max(r0, r1), max(r2, r3));
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}

// Exclusive prefix sum over the threads of a block (thread order).  `wsum`
// is LDS scratch of at least BS/64 + 1 words.  Ends with a barrier so the
// scratch may be reused.
template <int BS>
__device__ __forceinline__ uint32_t block_excl_sum(uint32_t v, uint32_t* wsum, uint32_t* total) {
  constexpr int NW = BS / kWave;
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const uint32_t incl = wave_incl_sum(v);
  if (lane == kWave - 1) wsum[w] = incl;
  __syncthreads();
  if (w == 0) {
    uint32_t t = lane < NW ? wsum[lane] : 0u;
    t = wave_incl_sum(t);
    if (lane < NW) wsum[lane] = t;
    if (lane == NW - 1) wsum[NW] = t;
  }
  __syncthreads();
  const uint32_t r = (w ? wsum[w - 1] : 0u) + incl - v;
  if (total) *total = wsum[NW];
  __syncthreads();
  return r;
}

// The same for a pair of values in one pass (the same three barriers):
// e0/e1 the exclusive sums, t0/t1 the totals; wsum holds 2*(BS/64 + 1) words.
template <int BS>
__device__ __forceinline__ void block_excl_sum2(uint32_t v0, uint32_t v1, uint32_t* wsum, uint32_t& e0,
                                                uint32_t& e1, uint32_t& t0, uint32_t& t1) {
  constexpr int NW = BS / kWave;
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const uint32_t i0 = wave_incl_sum(v0), i1 = wave_incl_sum(v1);
  if (lane == kWave - 1) {
    wsum[w] = i0;
    wsum[NW + 1 + w] = i1;
  }
  __syncthreads();
  if (w == 0) {
    uint32_t a0 = lane < NW ? wsum[lane] : 0u, a1 = lane < NW ? wsum[NW + 1 + lane] : 0u;
    a0 = wave_incl_sum(a0);
    a1 = wave_incl_sum(a1);
    if (lane < NW) {
      wsum[lane] = a0;
      wsum[NW + 1 + lane] = a1;
    }
    if (lane == NW - 1) {
      wsum[NW] = a0;
      wsum[2 * NW + 1] = a1;
    }
  }
  __syncthreads();
  e0 = (w ? wsum[w - 1] : 0u) + i0 - v0;
  e1 = (w ? wsum[NW + 1 + w - 1] : 0u) + i1 - v1;
  t0 = wsum[NW];
  t1 = wsum[2 * NW + 1];
  __syncthreads();
}

template <int BS>
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* wsum) {
  uint32_t tot;
  block_excl_sum<BS>(v, wsum, &tot);
  return tot;
}

template <int BS>
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t* wsum) {
  constexpr int NW = BS / kWave;
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  v = wave_max_u32(v);
  if (lane == 0) wsum[w] = v;
  __syncthreads();
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) m = max(m, wsum[i]);
  __syncthreads();
  return m;
}

// ------------------------------------------------------- item iteration ---
// Calls body(i, load(i)) for every i in [0, n), BS*UNR items per sweep with
// all loads of a sweep issued before any body runs (memory-level
// parallelism for global sources).
// Offsets are compared with the remaining count, and the loop stops before
// base + BS*UNR could pass n, so n may be as large as 2^32 - 1.
template <int BS, int UNR, class Load, class Body>
__device__ __forceinline__ void for_items(uint32_t n, Load load, Body body) {
  for (uint32_t base = 0; base < n; base += BS * UNR) {
    const uint32_t rem = n - base;
    uint32_t v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t o = u * BS + threadIdx.x;
      v[u] = (o < rem) ? load(base + o) : 0u;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t o = u * BS + threadIdx.x;
      if (o < rem) body(base + o, v[u]);
    }
    if (rem <= static_cast<uint32_t>(BS * UNR)) break;
  }
}

// --------------------------------------------------------- radix select ---
// LDS workspace of the block radix select.
constexpr int kSelBins = 2048;
constexpr int kSelDigit = 11;

// Scratch of the block reductions and digit search.
struct SelectScratch {
  uint32_t wsum[20];
  uint32_t found[4];
};

struct alignas(16) SelectShared {
  uint32_t hist[kSelBins];
  uint32_t wsum[20];
  uint32_t found[4];
  __device__ __forceinline__ SelectScratch& scratch() { return *reinterpret_cast<SelectScratch*>(wsum); }
};

struct SelectResult {
  uint32_t kth;      // the kk-th largest selection key
  uint32_t above;    // items with a larger selection key
  uint32_t equal;    // items equal to kth
};

// Hand-over of results between the workgroups of one kernel.  A device-wide
// fence (__threadfence) writes back and invalidates the whole L2 of the
// calling XCD, and when every producer pays for one they serialise.
// Instead producers write the handed-over data with agent-scope stores
// (coherent across the XCDs' L2 caches) or atomics and wait for them to
// complete before taking a ticket; only the consumer that wins the ticket
// invalidates its L2 (an agent-scope acquire) before it reads.
// Why this orders the data before the ticket without a release fence: an
// agent-scope store is issued with the sc1 bit, so it is written through to
// the memory side shared by every XCD rather than kept in the producer's
// L2; vmcnt counts it until that write has been acknowledged, so after
// s_waitcnt vmcnt(0) (wait_memory) every such store of the wave is visible
// device-wide.  A workgroup barrier then covers the other waves' stores, and
// only after it does one lane take the ticket with an atomic, which is
// performed at the device-coherent level.  A consumer that sees the final
// ticket value therefore follows every producer's completed stores, and its
// acquire drops any stale lines its own L2 held.  The argument rests on the
// hardware's write-through and counter semantics rather than on a fence the
// language memory model names; the GPU tests of every hand-over (fallback
// merges, large-k radix passes, the lexicographic tie list) check it.
__device__ __forceinline__ void store_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_memory() { __builtin_amdgcn_s_waitcnt(0); }
__device__ __forceinline__ void acquire_agent() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

// LDS histogram increment of `bin` for the calling lanes with `active`
// set.  The lanes whose bin equals the first active lane's add with one
// atomic; the others add their own.  A digit most keys share (a plateau of
// equal values, candidates that all lie near the top) would otherwise
// serialise every lane on one LDS address.  May be called from divergent
// code: only the lanes that execute it take part.
__device__ __forceinline__ void hist_add(uint32_t* hist, uint32_t bin, bool active) {
  if (!active) return;
  // only the active lanes run this: the first of them is the leader, and its
  // bin is read as a scalar
  const uint32_t lb = __builtin_amdgcn_readfirstlane(bin);
  const bool same = bin == lb;
  const uint64_t sm = __ballot(same);
  if (same) {
    if (static_cast<int>(threadIdx.x & (kWave - 1)) == __ffsll(static_cast<unsigned long long>(sm)) - 1)
      atomicAdd(&hist[lb], static_cast<uint32_t>(__popcll(sm)));
  } else {
    atomicAdd(&hist[bin], 1u);
  }
}

// Slot in an LDS list for each calling lane with `take` set: one atomic on
// the list's counter per wave, slots in lane order.  Returns the slot
// (unspecified for lanes without `take`).  May be called from divergent
// code: only the lanes that execute it take part.
__device__ __forceinline__ uint32_t lds_append(uint32_t* counter, bool take) {
  const uint64_t m = __ballot(take);
  if (m == 0) return 0u;
  const int leader = __ffsll(static_cast<unsigned long long>(m)) - 1;
  const uint32_t lane = threadIdx.x & (kWave - 1);
  uint32_t base = 0;
  if (static_cast<int>(lane) == leader) base = atomicAdd(counter, static_cast<uint32_t>(__popcll(m)));
  base = __builtin_amdgcn_readlane(base, leader);
  const uint64_t below = lane == 0 ? 0ull : (m & (~0ull >> (kWave - lane)));
  return base + static_cast<uint32_t>(__popcll(below));
}

// Wave 0 of a block (the caller makes only lanes of one wave call it)
// finds the bin of `hist` (nb bins, a power of two, 16-byte aligned) that
// holds rank krem (1-based) counted from the highest bin, and stores
// sh.found = {bin, items in higher bins, items in the bin}.  Requires
// 1 <= krem <= the histogram's total.
__device__ __forceinline__ void rank_bin_search(const uint32_t* hist, uint32_t nb, uint32_t krem,
                                                SelectScratch& sh) {
  const int lane = threadIdx.x & (kWave - 1);
  if (nb >= static_cast<uint32_t>(4 * kWave)) {
    // lane L owns bins [nb - (L+1)*per, nb - L*per); lane 0 the highest
    const uint32_t per = nb / kWave;  // a multiple of 4
    const uint32_t base = nb - (lane + 1) * per;
    uint32_t loc = 0;
    for (uint32_t q = 0; q < per; q += 4) {
      const uint4 v4 = *reinterpret_cast<const uint4*>(&hist[base + q]);
      loc += v4.x + v4.y + v4.z + v4.w;
    }
    uint32_t run = wave_incl_sum(loc) - loc;
    if (run < krem && krem <= run + loc) {
      // the rank falls in this lane's bins: walk them from the top
      for (int q = static_cast<int>(per) - 4; q >= 0; q -= 4) {
        const uint4 v4 = *reinterpret_cast<const uint4*>(&hist[base + q]);
        const uint32_t c4[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
        for (int j = 3; j >= 0; --j) {
          if (run < krem && krem <= run + c4[j]) {
            sh.found[0] = base + q + j;
            sh.found[1] = run;
            sh.found[2] = c4[j];
          }
          run += c4[j];
        }
      }
    }
  } else {
    // at most 128 bins: lane L owns descending ranks [L*per, (L+1)*per)
    const uint32_t per = (nb + kWave - 1) / kWave;  // 1 or 2
    uint32_t hv[2];
    uint32_t loc = 0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const uint32_t r = lane * per + q;
      hv[q] = (static_cast<uint32_t>(q) < per && r < nb) ? hist[nb - 1 - r] : 0u;
      loc += hv[q];
    }
    uint32_t run = wave_incl_sum(loc) - loc;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const uint32_t r = lane * per + q;
      if (static_cast<uint32_t>(q) < per && r < nb) {
        if (run < krem && krem <= run + hv[q]) {
          sh.found[0] = nb - 1 - r;
          sh.found[1] = run;
          sh.found[2] = hv[q];
        }
        run += hv[q];
      }
    }
  }
}

// The kk-th largest (1-based, with multiplicity) of the selection keys
// produced by `visit`.  visit(f) must call f(skey) once for every item of
// the set, from any thread; every call site in the block calls it with the
// same set.  Only the low `nbits` bits may differ between items: the bits
// above are `prefix` for all of them.  Requires 1 <= kk <= |set|.
// Digits are DIGIT bits wide; `hist` is LDS of 2^DIGIT words (16-byte
// aligned).  Per digit pass: an LDS histogram, then wave 0 alone scans it
// from the top with 16-byte reads and wave prefix sums, so a pass costs
// three barriers.
template <int BS, int DIGIT, class Visit>
__device__ __forceinline__ SelectResult block_select_kth(Visit visit, uint32_t kk, int nbits,
                                                         uint32_t prefix, uint32_t* hist,
                                                         SelectScratch& sh) {
  static_assert(DIGIT >= 8 && DIGIT <= 13, "digit width");
  const uint32_t tid = threadIdx.x;
  uint32_t krem = kk, above_total = 0, eq = 0;
  int hi = nbits;
  if (hi == 0) {
    uint32_t cnt = 0;
    visit([&](uint32_t) { ++cnt; });
    eq = block_sum<BS>(cnt, sh.wsum);
  }
  while (hi > 0) {
    const int bits = hi < DIGIT ? hi : DIGIT;
    const int shift = hi - bits;
    const uint32_t nb = 1u << bits;
    const uint32_t hmask = (hi >= 32) ? 0u : ~((1u << hi) - 1u);
    for (uint32_t b = tid; b < nb; b += BS) hist[b] = 0;
    __syncthreads();
    const uint32_t pre = prefix & hmask;
    visit([&](uint32_t s) { hist_add(hist, (s >> shift) & (nb - 1), (s & hmask) == pre); });
    __syncthreads();
    if (tid < kWave) rank_bin_search(hist, nb, krem, sh);
    __syncthreads();
    const uint32_t d = sh.found[0], ab = sh.found[1];
    eq = sh.found[2];
    prefix = (prefix & hmask) | (d << shift);
    krem -= ab;
    above_total += ab;
    hi = shift;
  }
  __syncthreads();
  SelectResult res;
  res.kth = prefix;
  res.above = above_total;
  res.equal = eq;
  return res;
}

// The kk-th largest (1-based, with multiplicity) of m keys held in LDS, for
// short lists: each key counts the keys above it and equal to it (m^2
// compares in all, eight LDS reads in flight per step), and the keys with
// #above < kk <= #above + #equal, all equal to the answer, write out[0] =
// the key and out[1] = #above.  Requires 1 <= kk <= m; every thread of the
// block calls it, and the caller syncs before reading out.
constexpr uint32_t kListRankMax = 256;
template <int BS>
__device__ __forceinline__ void list_kth(const uint32_t* list, uint32_t m, uint32_t kk, uint32_t* out) {
  for (uint32_t i = threadIdx.x; i < m; i += BS) {
    const uint32_t c = list[i];
    uint32_t gt = 0, ge = 0, j = 0;
    for (; j + 8 <= m; j += 8) {
      uint32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = list[j + u];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        gt += v[u] > c ? 1u : 0u;
        ge += v[u] >= c ? 1u : 0u;
      }
    }
    for (; j < m; ++j) {
      const uint32_t v = list[j];
      gt += v > c ? 1u : 0u;
      ge += v >= c ? 1u : 0u;
    }
    if (gt < kk && kk <= ge) {
      out[0] = c;
      out[1] = gt;
    }
  }
}

// The common case: 11-bit digits in the SelectShared histogram.
template <int BS, class Visit>
__device__ __forceinline__ SelectResult block_select_kth(Visit visit, uint32_t kk, int nbits,
                                                         uint32_t prefix, SelectShared& sh) {
  return block_select_kth<BS, kSelDigit>(visit, kk, nbits, prefix, sh.hist, sh.scratch());
}

// Index of the lexicographic threshold pair (Sec. 3 stage 2 taken on
// (key, -index) pairs): with tau the t-th largest sampled key, the t-th
// largest sampled pair is (tau, -i) where i is the r-th smallest index, with
// multiplicity, among the draws whose key is tau, r = t - #draws above tau.
// draws(f) must call f(key, index) once per draw, from any thread of the
// block, identically on every call.  The indices of the tied draws are kept
// in `list` (cap words of LDS) when they fit, otherwise the draws are
// visited again on each select pass; `hist` is 2^DIGIT words of LDS.
// Returns 0xFFFFFFFF when no draw carries tau (not for a tau taken from the
// same draws).
template <int BS, int DIGIT, class Draws>
__device__ __forceinline__ uint32_t tau_pair_index(Draws draws, uint32_t tau, uint32_t t, uint32_t* list, uint32_t cap,
                                   uint32_t* hist, SelectScratch& scr, uint32_t* s_n) {
  if (threadIdx.x == 0) *s_n = 0;
  __syncthreads();
  uint32_t above = 0;
  draws([&](uint32_t key, uint32_t idx) {
    if (key > tau) {
      ++above;
    } else if (key == tau) {
      const uint32_t p = atomicAdd(s_n, 1u);
      if (p < cap) list[p] = idx;
    }
  });
  const uint32_t a = block_sum<BS>(above, scr.wsum);
  __syncthreads();
  const uint32_t ne = *s_n;
  if (ne == 0 || a >= t) return 0xFFFFFFFFu;
  const uint32_t r = min(t - a, ne);
  SelectResult res;
  if (ne <= cap) {
    res = block_select_kth<BS, DIGIT>(
        [&](auto f) {
          for (uint32_t i = threadIdx.x; i < ne; i += BS) f(~list[i]);
        },
        r, 32, 0u, hist, scr);
  } else {
    res = block_select_kth<BS, DIGIT>(
        [&](auto f) {
          draws([&](uint32_t key, uint32_t idx) {
            if (key == tau) f(~idx);
          });
        },
        r, 32, 0u, hist, scr);
  }
  return ~res.kth;
}

// Top-t of up to 64*E keys held by one wave (E per lane, `valid` bits mark
// which of a lane's slots hold keys): t rounds of a wave-wide max; the lowest
// lane holding the maximum gives up one copy and stores it to out[round]
// (out may be null).  Returns got = min(t, number of keys); `last` receives
// the got-th largest key in every lane.  v is left as it was.
//
// Each lane first sorts a copy of its keys in descending order (empty slots
// as 0, the lowest key: a lane's first n slots then hold its n keys, since a
// key of 0 and an empty slot are alike), so a round reads every lane's head
// and the lane that gives it up shifts its copy by one.
template <int E>
__device__ __forceinline__ uint32_t wave_top_t(const uint32_t (&v)[E], uint32_t valid, uint32_t t,
                                               uint32_t* out, uint32_t& last) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t s[E];
  uint32_t n = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool in = (valid >> e) & 1u;
    s[e] = in ? v[e] : 0u;
    n += in ? 1u : 0u;
  }
  // odd-even transposition sort, descending (E rounds sort E values)
#pragma unroll
  for (int r = 0; r < E; ++r)
#pragma unroll
    for (int j = r & 1; j + 1 < E; j += 2) {
      const uint32_t hi = max(s[j], s[j + 1]), lo = min(s[j], s[j + 1]);
      s[j] = hi;
      s[j + 1] = lo;
    }
  uint32_t got = 0;
  for (; got < t; ++got) {
    const bool have = n > 0;
    if (__ballot(have) == 0) break;
    const uint32_t wm = wave_max_u32(have ? s[0] : 0u);
    last = wm;
    // lanes whose head equals the wave maximum; the lowest one gives it up
    const uint64_t holders = __ballot(have && s[0] == wm);
    const int owner = __ffsll(static_cast<unsigned long long>(holders)) - 1;
    if (lane == owner) {
#pragma unroll
      for (int e = 0; e + 1 < E; ++e) s[e] = s[e + 1];
      s[E - 1] = 0;
      --n;
      if (out) out[got] = wm;
    }
  }
  return got;
}

// Number of leading bits shared by every value in [lo, hi] (lo <= hi),
// counted within the low `nbits` bits.
__device__ __forceinline__ int shared_prefix_bits(uint32_t lo, uint32_t hi, int nbits) {
  const uint32_t x = (lo ^ hi) << (32 - nbits);
  return x == 0 ? nbits : __clz(x);
}

// ----------------------------------------------------------- bitonic sort --
// Sorts P = E*BS 64-bit values descending.  Thread t holds positions
// e*BS + t (e < E) in v[e].  Compare-exchange partners at stride s are in the
// same thread (s >= BS), in another wave (64 <= s < BS: through LDS, one
// barrier per stage with two alternating buffers) or in the same wave
// (s < 64: lane shuffles).  `lds` holds 2*P values, or P with ONE_BUF (one
// more barrier per LDS stage).
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(x), m, kWave);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(x >> 32), m, kWave);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

template <int BS, int E, bool ONE_BUF = false>
__device__ __forceinline__ void bitonic_sort_regs_desc(uint64_t (&v)[E], uint64_t* lds) {
  constexpr uint32_t P = static_cast<uint32_t>(E) * BS;
  const uint32_t t = threadIdx.x;
  int buf = 0;
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= static_cast<uint32_t>(BS)) {
        const uint32_t es = stride / BS;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((static_cast<uint32_t>(e) & es) == 0) {
            const int f = e ^ static_cast<int>(es);
            const uint32_t p = static_cast<uint32_t>(e) * BS + t;
            const bool desc = (p & size) == 0;
            const uint64_t a = v[e], b = v[f];
            if ((a < b) == desc) { v[e] = b; v[f] = a; }
          }
        }
      } else if (stride >= static_cast<uint32_t>(kWave)) {
        uint64_t* cur = lds + (ONE_BUF ? 0 : (buf ? P : 0));
        buf ^= 1;
        if (ONE_BUF) __syncthreads();  // the previous stage's reads are done
#pragma unroll
        for (int e = 0; e < E; ++e) cur[static_cast<uint32_t>(e) * BS + t] = v[e];
        __syncthreads();
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint32_t p = static_cast<uint32_t>(e) * BS + t;
          const uint64_t o = cur[p ^ stride];
          const bool desc = (p & size) == 0;
          const bool lower = (p & stride) == 0;
          v[e] = (lower == desc) ? max(v[e], o) : min(v[e], o);
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint32_t p = static_cast<uint32_t>(e) * BS + t;
          const uint64_t o = shfl_xor_u64(v[e], static_cast<int>(stride));
          const bool desc = (p & size) == 0;
          const bool lower = (p & stride) == 0;
          v[e] = (lower == desc) ? max(v[e], o) : min(v[e], o);
        }
      }
    }
  }
}

// Monotone log-scale bin of a key distance d = key - tau, in
// [0, kLogBins): exact below 128, then 128 bins per octave (the 7 bits after
// the leading one).  Larger d never maps to a smaller bin, and a bin spans a
// relative width of at most 1/128 of its distance.
constexpr uint32_t kLogBins = 3328;
__device__ __forceinline__ uint32_t log_bin(uint32_t d) {
  if (d < 128u) return d;
  const uint32_t e = 31u - static_cast<uint32_t>(__clz(d));  // 7..31
  return (e - 6u) * 128u + ((d >> (e - 7u)) & 127u);
}
// Number of values in v[s, e) greater than c (v in LDS): eight reads are in
// flight per step, so a long run costs one LDS latency per eight values.
__device__ __forceinline__ uint32_t count_greater(const uint64_t* v, uint32_t s, uint32_t e, uint64_t c) {
  uint32_t r = 0, q = s;
  for (; q + 8 <= e; q += 8) {
    uint64_t t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = v[q + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) r += t[u] > c ? 1u : 0u;
  }
  for (; q < e; ++q) r += v[q] > c ? 1u : 0u;
  return r;
}

// The smallest d with log_bin(d) = b: log_bin(d) >= b exactly when
// d >= log_bin_edge(b) (b < kLogBins).
__device__ __forceinline__ uint32_t log_bin_edge(uint32_t b) {
  if (b < 128u) return b;
  const uint32_t e = b / 128u + 6u, m = b % 128u;
  return (1u << e) | (m << (e - 7u));
}

// Bitonic sort, descending, of P = E*T 64-bit values held E per thread in
// blocked order (thread t holds positions t*E .. t*E+E-1).  Strides below E
// are swaps within a thread, strides up to 32*E shuffles within a wave,
// larger ones go through `lds` (P values).  Waves holding no position only
// take part in the barriers.  Every thread of the block must call it with
// the same P (a power of two, at least E).
template <int E, int S>
__device__ __forceinline__ void bitonic_regs_step(uint64_t (&v)[E], uint32_t t, uint32_t size) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if ((e & S) == 0) {
      const uint32_t p = t * E + static_cast<uint32_t>(e);
      const bool desc = (p & size) == 0;
      const uint64_t x = v[e], y = v[e | S];
      const bool sw = desc ? (x < y) : (x > y);
      v[e] = sw ? y : x;
      v[e | S] = sw ? x : y;
    }
  }
}

template <int E>
__device__ __forceinline__ void bitonic_blocked_desc(uint64_t (&v)[E], uint32_t P, uint64_t* lds) {
  static_assert(E == 1 || E == 2 || E == 4 || E == 8 || E == 16, "elements per thread");
  const uint32_t t = threadIdx.x;
  const bool act = t * E < P;
  const bool wave_act = (t & ~static_cast<uint32_t>(kWave - 1)) * E < P;
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride < static_cast<uint32_t>(E)) {
        if (!wave_act) continue;
        if (E > 8 && stride == 8) bitonic_regs_step<E, (E > 8 ? 8 : 0)>(v, t, size);
        else if (E > 4 && stride == 4) bitonic_regs_step<E, (E > 4 ? 4 : 0)>(v, t, size);
        else if (E > 2 && stride == 2) bitonic_regs_step<E, (E > 2 ? 2 : 0)>(v, t, size);
        else if (E > 1 && stride == 1) bitonic_regs_step<E, (E > 1 ? 1 : 0)>(v, t, size);
        continue;
      }
      const uint32_t d = stride / E;  // partner thread distance
      const bool lower = (t & d) == 0;
      const bool desc = ((t * E) & size) == 0;
      if (d < static_cast<uint32_t>(kWave)) {
        if (!wave_act) continue;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint64_t o = shfl_xor_u64(v[e], static_cast<int>(d));
          v[e] = (lower == desc) ? max(v[e], o) : min(v[e], o);
        }
      } else {
        __syncthreads();
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) lds[t * E + e] = v[e];
        }
        __syncthreads();
        if (act) {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const uint64_t o = lds[(t * E + e) ^ stride];
            v[e] = (lower == desc) ? max(v[e], o) : min(v[e], o);
          }
        }
      }
    }
  }
}

// Composite ordering key: larger key first, then smaller index.
__device__ __forceinline__ uint64_t composite(uint32_t key, uint32_t idx) {
  return (static_cast<uint64_t>(key) << 32) | static_cast<uint64_t>(~idx);
}
__device__ __forceinline__ uint32_t comp_key(uint64_t c) { return static_cast<uint32_t>(c >> 32); }
__device__ __forceinline__ uint32_t comp_idx(uint64_t c) { return ~static_cast<uint32_t>(c); }

__device__ __forceinline__ uint32_t next_pow2(uint32_t x) {
  return x <= 1 ? 1u : (1u << (32 - __clz(x - 1)));
}

}  // namespace profk
