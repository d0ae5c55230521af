// Exact top-k of a candidate set by one workgroup (refinement, Sec. 3 stage
// 4, and the exact fallback), shared by the vector and per-row kernels.
//
// A candidate source exposes
//   visit<BS>(n, cache, f)  call f(i, key, idx_accessor) for every candidate
//                           i < n, keys from cache[i] when cache is given;
//   idx_at(i)               the input index of candidate i.
// Selection is a radix select on the keys (then on the indices of the tied
// keys when only part of the tie class fits), so the result is the unique
// top-k of the total order: larger key first, then smaller index.
#pragma once

#include "device_common.h"
#include "filter_tile.h"

namespace profk {

// Index accessors handed to candidate visitors: an index is loaded only
// when a visitor asks for it.
struct LoadIdx {
  const uint32_t* p;
  __device__ __forceinline__ uint32_t operator()() const { return *p; }
};
struct PosIdx {
  uint32_t v;
  __device__ __forceinline__ uint32_t operator()() const { return v; }
};

// Candidates held in LDS (keys of type K and indices).
template <class K = uint32_t>
struct LdsSrc {
  const K* key;
  const uint32_t* idx;
  template <int BS, class F>
  __device__ __forceinline__ void visit(uint32_t n, const uint32_t*, F f) const {
    for (uint32_t i = threadIdx.x; i < n; i += BS) f(i, key[i], LoadIdx{idx + i});
  }
  __device__ __forceinline__ uint32_t idx_at(uint32_t i) const { return idx[i]; }
};

// A contiguous range of the input starting at element `lo` of `values`;
// keys are computed on the fly.
template <int DT>
struct InputSrc {
  const void* values;
  uint32_t lo;
  template <int BS, class F>
  __device__ __forceinline__ void visit(uint32_t n, const uint32_t* cache, F f) const {
    for_items<BS, 8>(n, [&](uint32_t i) { return cache ? cache[i] : key_of<DT>(load_raw<DT>(values, lo + i)); },
                     [&](uint32_t i, uint32_t v) { f(i, v, PosIdx{lo + i}); });
  }
  __device__ __forceinline__ uint32_t idx_at(uint32_t i) const { return lo + i; }
};

// LDS the selection works in.  `collect` holds at least kk values; `hist`
// 2^DIGIT words, 16-byte aligned; `cache` (optional) cache_cap keys.
struct TopkSmem {
  uint32_t* cache;
  uint32_t cache_cap;
  uint32_t* hist;
  uint64_t* collect;
  SelectScratch* scratch;
  uint32_t* counter;
};

// Exact top-kk (kk <= n) of a candidate set under the total order, left
// unsorted as composites (key << 32 | ~index) in sm.collect[0..kk).  Every
// candidate key lies in [lo_key, hi_key], so the leading bits they share
// are skipped.  The collection first reserves slots for (key, candidate
// number) and then loads all selected indices at once.
template <int BS, int DIGIT, class Src>
__device__ __forceinline__ void block_topk(const Src& src, uint32_t n, uint32_t kk, uint32_t lo_key,
                                           uint32_t hi_key, int keybits, const TopkSmem& sm) {
  const uint32_t tid = threadIdx.x;
  const bool cached = sm.cache != nullptr && n <= sm.cache_cap;
  if (cached) {
    src.template visit<BS>(n, nullptr, [&](uint32_t i, uint32_t key, auto) { sm.cache[i] = key; });
    __syncthreads();
  }
  const uint32_t* cache = cached ? sm.cache : nullptr;
  auto keys_only = [&](auto f) {
    if (cached) {
      for (uint32_t i = tid; i < n; i += BS) f(sm.cache[i]);
    } else {
      src.template visit<BS>(n, nullptr, [&](uint32_t, uint32_t key, auto) { f(key); });
    }
  };
  const int shared = shared_prefix_bits(lo_key, hi_key, keybits);
  const SelectResult r =
      block_select_kth<BS, DIGIT>(keys_only, kk, keybits - shared, lo_key, sm.hist, *sm.scratch);
  const uint32_t kstar = r.kth;
  const uint32_t krem = kk - r.above;
  const bool cut = krem < r.equal;
  uint32_t istar = 0xFFFFFFFFu;
  if (cut) {
    // the krem smallest indices among the ties at kstar
    const SelectResult ri = block_select_kth<BS, DIGIT>(
        [&](auto f) {
          src.template visit<BS>(n, cache, [&](uint32_t, uint32_t key, auto idx) {
            if (key == kstar) f(~idx());
          });
        },
        krem, 32, 0u, sm.hist, *sm.scratch);
    istar = ~ri.kth;
  }
  if (tid == 0) *sm.counter = 0;
  __syncthreads();
  src.template visit<BS>(n, cache, [&](uint32_t i, uint32_t key, auto idx) {
    if (key > kstar || (key == kstar && (!cut || idx() <= istar))) {
      const uint32_t p = atomicAdd(sm.counter, 1u);
      if (p < kk) sm.collect[p] = (static_cast<uint64_t>(key) << 32) | i;
    }
  });
  __syncthreads();
  for (uint32_t p = tid; p < kk; p += BS) {
    const uint64_t e = sm.collect[p];
    sm.collect[p] = composite(static_cast<uint32_t>(e >> 32), src.idx_at(static_cast<uint32_t>(e)));
  }
  __syncthreads();
}

// Sorts collect[0..kk) descending (E*BS >= max(kk, k), a power of two) and
// writes k outputs: bit copies of the values and int64 indices; past kk,
// padding (-inf, -1).  `exch` holds 2*E*BS values and
// may alias nothing the caller still needs.
template <int DT, int BS, int E>
__device__ __forceinline__ void sort_write(const uint64_t* collect, uint32_t kk, uint32_t k, uint64_t* exch,
                                           void* out_vals, int64_t* out_idx) {
  const uint32_t tid = threadIdx.x;
  uint64_t v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t p = static_cast<uint32_t>(e) * BS + tid;
    v[e] = p < kk ? collect[p] : 0ull;
  }
  __syncthreads();
  bitonic_sort_regs_desc<BS, E>(v, exch);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t p = static_cast<uint32_t>(e) * BS + tid;
    if (p >= k) continue;
    uint32_t bits;
    int64_t id;
    if (p < kk) {
      bits = bits_of_key<DT>(comp_key(v[e]));
      id = comp_idx(v[e]);
    } else {
      bits = DT == 0 ? 0xFF800000u : 0xFF80u;  // -inf padding (relaxed recall)
      id = -1;
    }
    if (DT == 0) static_cast<uint32_t*>(out_vals)[p] = bits;
    else static_cast<uint16_t*>(out_vals)[p] = static_cast<uint16_t>(bits);
    out_idx[p] = id;
  }
}

// sort_write with E chosen from max(kk, k); supports up to 4*BS outputs.
template <int DT, int BS>
__device__ __forceinline__ void sort_write_any(const uint64_t* collect, uint32_t kk, uint32_t k,
                                               uint64_t* exch, void* out_vals, int64_t* out_idx) {
  const uint32_t P = next_pow2(max(kk, k));
  if (P <= static_cast<uint32_t>(BS)) sort_write<DT, BS, 1>(collect, kk, k, exch, out_vals, out_idx);
  else if (P <= 2u * BS) sort_write<DT, BS, 2>(collect, kk, k, exch, out_vals, out_idx);
  else sort_write<DT, BS, 4>(collect, kk, k, exch, out_vals, out_idx);
}

}  // namespace profk
