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

#include <type_traits>
#include <utility>

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
    // eight keys (and indices, where a visitor asks for them) read per
    // thread before any visitor runs
    constexpr int U = 8;
    for (uint32_t base = 0; base < n; base += BS * U) {
      uint32_t kv[U], iv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = base + u * BS + threadIdx.x;
        kv[u] = i < n ? static_cast<uint32_t>(key[i]) : 0u;
        iv[u] = i < n ? idx[i] : 0u;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = base + u * BS + threadIdx.x;
        if (i < n) f(i, kv[u], PosIdx{iv[u]});
      }
    }
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
//
// block_topk_core is the selection itself over `src` (keys cached in
// sm.cache when they fit); block_topk first copies keys and indices to LDS
// when both fit.  The two are separate functions so that neither calls
// itself: a recursive call could not be inlined, and its LDS arrays would
// then be reached through generic pointers (flat loads and atomics) from a
// stack frame.
template <int BS, int DIGIT, class Src>
__device__ __forceinline__ void block_topk_core(const Src& src, uint32_t n, uint32_t kk, uint32_t lo_key,
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
    const bool take = key > kstar || (key == kstar && (!cut || idx() <= istar));
    const uint32_t p = lds_append(sm.counter, take);
    if (take && p < kk) sm.collect[p] = (static_cast<uint64_t>(key) << 32) | i;
  });
  __syncthreads();
  for (uint32_t p = tid; p < kk; p += BS) {
    const uint64_t e = sm.collect[p];
    sm.collect[p] = composite(static_cast<uint32_t>(e >> 32), src.idx_at(static_cast<uint32_t>(e)));
  }
  __syncthreads();
}

// Sources with pair_at(i) (key and index of candidate i) give both in one
// load sweep.
template <class S, class = void>
struct HasPairAt : std::false_type {};
template <class S>
struct HasPairAt<S, std::void_t<decltype(std::declval<const S&>().pair_at(0u))>> : std::true_type {};

template <int BS, int DIGIT, class Src>
__device__ __forceinline__ void block_topk(const Src& src, uint32_t n, uint32_t kk, uint32_t lo_key,
                                           uint32_t hi_key, int keybits, const TopkSmem& sm) {
  if (sm.cache != nullptr && 2 * n <= sm.cache_cap) {
    // keys and indices both fit: copy them to LDS once (index loads batched)
    // and select there, so the passes on tied keys read no global memory
    uint32_t* const pk = sm.cache;
    uint32_t* const pi = sm.cache + n;
    if constexpr (HasPairAt<Src>::value) {
      // eight pairs per thread in flight per sweep (n is at most half the
      // cache, far below 2^32)
      constexpr int U = 8;
      for (uint32_t base = 0; base < n; base += BS * U) {
        uint2 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const uint32_t i = base + u * BS + threadIdx.x;
          v[u] = i < n ? src.pair_at(i) : uint2{0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const uint32_t i = base + u * BS + threadIdx.x;
          if (i < n) {
            pk[i] = v[u].x;
            pi[i] = v[u].y;
          }
        }
      }
    } else {
      src.template visit<BS>(n, nullptr, [&](uint32_t i, uint32_t key, auto) { pk[i] = key; });
      for_items<BS, 8>(n, [&](uint32_t i) { return src.idx_at(i); }, [&](uint32_t i, uint32_t v) { pi[i] = v; });
    }
    __syncthreads();
    TopkSmem lds = sm;
    lds.cache = nullptr;
    lds.cache_cap = 0;
    block_topk_core<BS, DIGIT>(LdsSrc<uint32_t>{pk, pi}, n, kk, lo_key, hi_key, keybits, lds);
    return;
  }
  block_topk_core<BS, DIGIT>(src, n, kk, lo_key, hi_key, keybits, sm);
}

// Exact top-kk of an item set too large for LDS, read in a few passes.
// Histogram passes over DIGIT-bit digits narrow a window of keys (a fixed
// prefix of the leading bits) that holds rank kk, until the items with key
// at or above the window's lowest key fit in LDS as (key, index) pairs
// (sm.cache_cap / 2 of them); one pass collects them and block_topk selects
// among them in LDS.  When the window is down to a single key whose tie
// class does not fit, the items above it are collected and the tie class is
// cut in index order (the smallest indices first) by src.ties_in_order.
// Leaves the kk composites unsorted in sm.collect[0..kk), as block_topk.
// Src provides
//   keys(f)                  f(pos, key) for every item, from any thread;
//   idx_of(pos)              the input index of item pos;
//   ties_in_order(key, m, g) g(pos, r) for the m items of that key with the
//                            smallest indices, r = 0..m-1 each once
//                            (block-wide; may use sm.hist and sm.scratch).
template <int BS, int DIGIT, class Src>
__device__ __forceinline__ void window_topk(const Src& src, uint32_t kk, int keybits, const TopkSmem& sm) {
  const uint32_t tid = threadIdx.x;
  const uint32_t cap = sm.cache_cap / 2;
  uint32_t* const pk = sm.cache;
  uint32_t* const pi = sm.cache + cap;
  SelectScratch& sc = *sm.scratch;
  uint32_t prefix = 0, above = 0, eq = 0;
  int hi = keybits;
  do {
    const int bits = hi < DIGIT ? hi : DIGIT;
    const int shift = hi - bits;
    const uint32_t nb = 1u << bits;
    const uint32_t hmask = hi >= 32 ? 0u : ~((1u << hi) - 1u);
    for (uint32_t b = tid; b < nb; b += BS) sm.hist[b] = 0;
    __syncthreads();
    src.keys([&](uint32_t, uint32_t key) { hist_add(sm.hist, (key >> shift) & (nb - 1), (key & hmask) == prefix); });
    __syncthreads();
    if (tid < kWave) rank_bin_search(sm.hist, nb, kk - above, sc);
    __syncthreads();
    prefix |= sc.found[0] << shift;
    above += sc.found[1];
    eq = sc.found[2];
    hi = shift;
  } while (above + eq > cap && hi > 0);
  // the window is [prefix, prefix + 2^hi); `above` items lie above it
  const bool cut = above + eq > cap;  // one key, too many ties
  if (tid == 0) *sm.counter = 0;
  __syncthreads();
  uint32_t mx = prefix;
  src.keys([&](uint32_t pos, uint32_t key) {
    const bool take = cut ? key > prefix : key >= prefix;
    const uint32_t p = lds_append(sm.counter, take);
    if (take) {
      pk[p] = key;
      pi[p] = pos;
      mx = max(mx, key);
    }
  });
  mx = block_max<BS>(mx, sc.wsum);
  uint32_t n2 = above + eq;
  if (cut) {
    src.ties_in_order(prefix, kk - above, [&](uint32_t pos, uint32_t r) {
      pk[above + r] = prefix;
      pi[above + r] = pos;
    });
    n2 = kk;
    __syncthreads();
  }
  // positions to input indices, every load of a sweep in flight at once
  for_items<BS, 8>(n2, [&](uint32_t p) { return src.idx_of(pi[p]); }, [&](uint32_t p, uint32_t v) { pi[p] = v; });
  __syncthreads();
  TopkSmem lds = sm;
  lds.cache = nullptr;
  lds.cache_cap = 0;
  block_topk_core<BS, DIGIT>(LdsSrc<uint32_t>{pk, pi}, n2, kk, prefix, mx, keybits, lds);
}

// Sorts collect[0..kk) descending (E*BS >= max(kk, n_out), a power of two)
// and calls f(p, composite, p < kk) for output positions p < n_out (past
// kk the composite is 0).  `exch` holds 2*E*BS values and may alias
// nothing the caller still needs.
template <int BS, int E, class F>
__device__ __forceinline__ void sort_desc_each(const uint64_t* collect, uint32_t kk, uint32_t n_out,
                                               uint64_t* exch, F f) {
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
    if (p < n_out) f(p, v[e], p < kk);
  }
}

// sort_desc_each with E chosen from max(kk, n_out); up to 4*BS outputs.
template <int BS, class F>
__device__ __forceinline__ void sort_desc_each_any(const uint64_t* collect, uint32_t kk, uint32_t n_out,
                                                   uint64_t* exch, F f) {
  const uint32_t P = next_pow2(max(kk, n_out));
  if (P <= static_cast<uint32_t>(BS)) sort_desc_each<BS, 1>(collect, kk, n_out, exch, f);
  else if (P <= 2u * BS) sort_desc_each<BS, 2>(collect, kk, n_out, exch, f);
  else sort_desc_each<BS, 4>(collect, kk, n_out, exch, f);
}

// Sorts collect[0..kk) descending and writes k outputs: bit copies of the
// values and int64 indices; past kk, padding (-inf, -1).  `exch` as for
// sort_desc_each; supports up to 4*BS outputs.
template <int DT, int BS>
__device__ __forceinline__ void sort_write_any(const uint64_t* collect, uint32_t kk, uint32_t k,
                                               uint64_t* exch, void* out_vals, int64_t* out_idx) {
  sort_desc_each_any<BS>(collect, kk, k, exch, [&](uint32_t p, uint64_t c, bool valid) {
    uint32_t bits;
    int64_t id;
    if (valid) {
      bits = bits_of_key<DT>(comp_key(c));
      id = comp_idx(c);
    } else {
      bits = DT == 0 ? 0xFF800000u : 0xFF80u;  // -inf padding (relaxed recall)
      id = -1;
    }
    if (DT == 0) static_cast<uint32_t*>(out_vals)[p] = bits;
    else static_cast<uint16_t*>(out_vals)[p] = static_cast<uint16_t>(bits);
    out_idx[p] = id;
  });
}

}  // namespace profk
