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
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t x) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) x = max(x, __shfl_xor(x, o, kWave));
  return x;
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
template <int BS, int UNR, class Load, class Body>
__device__ __forceinline__ void for_items(uint32_t n, Load load, Body body) {
  for (uint32_t base = 0; base < n; base += BS * UNR) {
    uint32_t v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t i = base + u * BS + threadIdx.x;
      v[u] = (i < n) ? load(i) : 0u;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const uint32_t i = base + u * BS + threadIdx.x;
      if (i < n) body(i, v[u]);
    }
  }
}

// --------------------------------------------------------- radix select ---
// LDS workspace of the block radix select.
constexpr int kSelBins = 2048;
constexpr int kSelDigit = 11;

struct SelectShared {
  uint32_t hist[kSelBins];
  uint32_t wsum[20];
  uint32_t found[4];
};

struct SelectResult {
  uint32_t kth;      // the kk-th largest selection key
  uint32_t above;    // items with a larger selection key
  uint32_t equal;    // items equal to kth
};

// The kk-th largest (1-based, with multiplicity) of the selection keys
// produced by `visit`.  visit(f) must call f(skey) once for every item of
// the set, from any thread; every call site in the block calls it with the
// same set.  Only the low `nbits` bits may differ between items: the bits
// above are `prefix` for all of them.  Requires 1 <= kk <= |set|.
template <int BS, class Visit>
__device__ SelectResult block_select_kth(Visit visit, uint32_t kk, int nbits,
                                         uint32_t prefix, SelectShared& sh) {
  uint32_t krem = kk, above_total = 0, eq = 0;
  int hi = nbits;
  if (hi == 0) {
    // every item equals the prefix
    uint32_t cnt = 0;
    visit([&](uint32_t) { ++cnt; });
    eq = block_sum<BS>(cnt, sh.wsum);
  }
  while (hi > 0) {
    const int bits = hi < kSelDigit ? hi : kSelDigit;
    const int shift = hi - bits;
    const uint32_t nb = 1u << bits;
    const uint32_t hmask = (hi >= 32) ? 0u : ~((1u << hi) - 1u);
    for (uint32_t b = threadIdx.x; b < nb; b += BS) sh.hist[b] = 0;
    __syncthreads();
    const uint32_t pre = prefix & hmask;
    visit([&](uint32_t s) {
      if ((s & hmask) == pre) atomicAdd(&sh.hist[(s >> shift) & (nb - 1)], 1u);
    });
    __syncthreads();
    // Each thread owns a run of bins in descending order; an exclusive scan
    // over threads gives the number of items in higher bins.
    const uint32_t per = (nb + BS - 1) / BS;
    const uint32_t r0 = threadIdx.x * per;   // descending rank of my first bin
    uint32_t loc = 0;
    for (uint32_t r = r0; r < r0 + per && r < nb; ++r) loc += sh.hist[nb - 1 - r];
    uint32_t run = block_excl_sum<BS>(loc, sh.wsum, nullptr);
    for (uint32_t r = r0; r < r0 + per && r < nb; ++r) {
      const uint32_t h = sh.hist[nb - 1 - r];
      if (run < krem && krem <= run + h) {
        sh.found[0] = nb - 1 - r;
        sh.found[1] = run;
        sh.found[2] = h;
      }
      run += h;
    }
    __syncthreads();
    const uint32_t d = sh.found[0], ab = sh.found[1];
    eq = sh.found[2];
    prefix = (prefix & hmask) | (d << shift);
    krem -= ab;
    above_total += ab;
    hi = shift;
    __syncthreads();
  }
  SelectResult res;
  res.kth = prefix;
  res.above = above_total;
  res.equal = eq;
  return res;
}

// Number of leading bits shared by every value in [lo, hi] (lo <= hi),
// counted within the low `nbits` bits.
__device__ __forceinline__ int shared_prefix_bits(uint32_t lo, uint32_t hi, int nbits) {
  const uint32_t x = (lo ^ hi) << (32 - nbits);
  return x == 0 ? nbits : __clz(x);
}

// ----------------------------------------------------------- bitonic sort --
// Sorts a[0..n) descending, n a power of two, in LDS.  Caller syncs before.
template <int BS>
__device__ void bitonic_sort_desc(uint64_t* a, uint32_t n) {
  for (uint32_t size = 2; size <= n; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (uint32_t i = threadIdx.x; i < n / 2; i += BS) {
        const uint32_t lo = 2 * i - (i & (stride - 1));
        const uint32_t hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const uint64_t x = a[lo], y = a[hi];
        if ((x < y) == desc) { a[lo] = y; a[hi] = x; }
      }
      __syncthreads();
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
