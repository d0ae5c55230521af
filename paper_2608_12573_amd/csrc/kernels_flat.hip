// Prof-K on one vector: sampling (stage 1), threshold (stage 2), the
// filter-and-compact pass (stage 3) and refinement with fallback (stage 4),
// Sec. 3 "The Prof-K Algorithm".
//
// Kernel sequence of one call, all on the caller's stream:
//   k_sample      ceil(S/1024) blocks (ceil(S/4096) of 1024 threads when
//                 t > 32): Philox draws, gathers, and each block's local
//                 top-t sample keys (the t-th largest of the whole sample is
//                 among the union of the blocks' top-t).
//   k_select_tau  only when that union is large: one block picks tau.
//   k_tau_index   lexicographic plans only: the sample blocks list the draws
//                 that carry tau, and the last one picks the threshold pair.
//   k_filter      the filter-and-compact pass (kernels_filter.hip).
//   k_finish      reads the segment counts; when k_req <= count <= M one
//                 block refines the candidates exactly, otherwise every
//                 block computes the exact top-k of its chunk of the input,
//                 the last of each group of 16 chunks to finish merges the
//                 group's, and the last group to finish merges the groups'.
#include <climits>
#include <cmath>

#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"
#include "sample_union.h"
#include "topk_block.h"

namespace profk {

// ------------------------------------------------------------ stage 1 -----
struct SampleArgs {
  const void* values;
  uint64_t n, seed, row;
  uint32_t S, t, tcap;
  uint32_t* union_keys;
  CallState* st;
  uint32_t* seg_cnt;
  uint32_t* fhist;
  uint32_t* bcur;   // null unless the call takes the large-k path
  uint32_t* ghist;  // null unless the call takes the large-k path
  // capped lists (t is then their length): each block's cut key, and every
  // draw's key at its draw number; null otherwise
  uint32_t* cut;
  uint32_t* all_keys;
};

template <int DT, int BS>
__global__ __launch_bounds__(BS) void k_sample(SampleArgs a) {
  constexpr uint32_t kPer = 4 * BS;  // four draws per thread
  __shared__ SampleUnionShared<BS> sh;
  const uint32_t b = blockIdx.x, tid = threadIdx.x;
  if (b == 0) reset_state(a.st, a.seg_cnt, a.fhist, a.bcur, a.ghist);
  const uint32_t j0 = b * kPer;
  const uint32_t nb = min(kPer, a.S - j0);
  uint32_t kv[4];
  uint32_t valid = 0;
  {
    // draw j = j0 + 4*tid + q is word q of Philox block (j0/4 + tid)
    const U64x4 r = philox4x64_10(static_cast<uint64_t>(j0 / 4) + tid, a.row, 0, 0, a.seed, 0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t j = 4 * tid + q;
      kv[q] = 0;
      if (j < nb) {
        kv[q] = key_of<DT>(load_raw<DT>(a.values, index_of_word(r.w[q], a.n)));
        valid |= 1u << q;
      }
    }
  }
  if (a.all_keys) {
    if (4 * tid + 3 < nb) {
      *reinterpret_cast<uint4*>(a.all_keys + j0 + 4 * tid) = uint4{kv[0], kv[1], kv[2], kv[3]};
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((valid >> q) & 1u) a.all_keys[j0 + 4 * tid + q] = kv[q];
    }
  }
  sample_block_top<BS, Elem<DT>::KEYBITS>(kv, valid, nb, a.t, a.union_keys + static_cast<size_t>(b) * a.tcap, sh,
                                           a.cut ? a.cut + b : nullptr);
}

// Per-block top-t of keys already in memory (the SAE path's sampled
// latents, 32-bit keys): block b takes keys [4*BS*b, 4*BS*(b+1)) and writes
// its top min(t, nb) to union_keys + b * tcap, as k_sample does for its
// draws, so that one block then selects tau from a union much smaller than
// the sample.
template <int BS>
__global__ __launch_bounds__(BS) void k_key_union(const uint32_t* keys, uint32_t n, uint32_t t, uint32_t tcap,
                                                  uint32_t* union_keys) {
  __shared__ SampleUnionShared<BS> sh;
  const uint32_t b = blockIdx.x, tid = threadIdx.x;
  const uint32_t j0 = b * 4 * BS, nb = min(4u * BS, n - j0);
  uint32_t kv[4];
  uint32_t valid = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t j = 4 * tid + q;
    kv[q] = j < nb ? keys[j0 + j] : 0u;
    if (j < nb) valid |= 1u << q;
  }
  sample_block_top<BS, 32>(kv, valid, nb, t, union_keys + static_cast<size_t>(b) * tcap, sh);
}

// ------------------------------------------------------------ stage 2 -----
// tau = t-th largest key of the union.  Used when the union is too large
// for the filter blocks to select from it themselves.
constexpr uint32_t kTauCache = 32768;
constexpr uint32_t kTauList = 2048;  // keys of the bin holding rank t

struct TauArgs {
  const uint32_t* keys;
  uint32_t n, t;
  int keybits;
  CallState* st;
  // capped sample lists (null otherwise): the n_cut blocks' cut keys, and
  // all n_all sample keys to select from when a cut key reaches the result
  const uint32_t* cut;
  uint32_t n_cut;
  const uint32_t* all_keys;
  uint32_t n_all;
};

__global__ __launch_bounds__(kTauBS) void k_select_tau(TauArgs a) {
  constexpr int NW = kTauBS / kWave;
  constexpr int E = 8;  // union keys per lane on the wave path
  __shared__ uint32_t cache[kTauCache];
  __shared__ SelectShared sel;
  __shared__ uint32_t lists[NW][kWaveTopMax];
  __shared__ uint32_t list_n[NW];
  __shared__ uint32_t tlist[kTauList];
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  if (a.t <= kWaveTopMax && a.n <= static_cast<uint32_t>(kTauBS * E)) {
    // every wave keeps the top t of its share, wave 0 merges the lists
    uint32_t v[E];
    uint32_t valid = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint32_t i = w * (kWave * E) + e * kWave + lane;
      v[e] = i < a.n ? a.keys[i] : 0u;
      if (i < a.n) valid |= 1u << e;
    }
    uint32_t last = 0;
    const uint32_t got = wave_top_t<E>(v, valid, a.t, lists[w], last);
    if (lane == 0) list_n[w] = got;
    __syncthreads();
    if (w == 0) {
      constexpr int E2 = NW * kWaveTopMax / kWave;
      uint32_t v2[E2];
      uint32_t valid2 = 0;
#pragma unroll
      for (int e = 0; e < E2; ++e) {
        uint32_t c = lane + kWave * e, li = 0;
        v2[e] = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i)
          if (li == static_cast<uint32_t>(i) && c >= list_n[i]) { c -= list_n[i]; li = i + 1; }
        if (li < NW) { v2[e] = lists[li][c]; valid2 |= 1u << e; }
      }
      wave_top_t<E2>(v2, valid2, a.t, nullptr, last);
      if (lane == 0) a.st->tau_key = last;
    }
    return;
  }
  // Capped sample lists: the t-th largest of the union is the sample's
  // unless a block that dropped keys has its cut key at or above it (every
  // dropped key is at most its block's cut key).  With C the largest cut
  // key, that is the case exactly when fewer than t union keys exceed C; the
  // select then takes all sample keys instead.
  const uint32_t* keys = a.keys;
  uint32_t n = a.n;
  if (a.cut) {
    // the first 4*kTauBS union keys are loaded with the cut keys
    constexpr int U = 4;
    uint32_t u[U];
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const uint32_t i = j * kTauBS + tid;
      u[j] = i < a.n ? a.keys[i] : 0u;
    }
    uint32_t c = 0;
    for (uint32_t i = tid; i < a.n_cut; i += kTauBS) c = max(c, a.cut[i]);
    c = block_max<kTauBS>(c, sel.wsum);
    uint32_t above = 0;
#pragma unroll
    for (int j = 0; j < U; ++j) above += (j * kTauBS + tid < a.n && u[j] > c) ? 1u : 0u;
    for (uint32_t i = U * kTauBS + tid; i < a.n; i += kTauBS) above += a.keys[i] > c ? 1u : 0u;
    // (the same in every thread: readfirstlane keeps the source uniform for
    // the compiler)
    if (__builtin_amdgcn_readfirstlane(block_sum<kTauBS>(above, sel.wsum)) < a.t) {
      keys = a.all_keys;
      n = a.n_all;
    }
  }
  auto gload = [&](uint32_t i) { return keys[i]; };
  const bool cached = n <= kTauCache;
  // every key of the union, from LDS when it fits (eight reads per thread
  // issued before any visitor runs)
  auto all = [&](auto f) {
    if (cached) for_items<kTauBS, 8>(n, [&](uint32_t i) { return cache[i]; }, [&](uint32_t, uint32_t v) { f(v); });
    else for_items<kTauBS, 8>(n, gload, [&](uint32_t, uint32_t v) { f(v); });
  };
  uint32_t mn = 0xFFFFFFFFu, mx = 0u;
  for_items<kTauBS, 16>(n, gload, [&](uint32_t i, uint32_t v) {
    if (cached) cache[i] = v;
    mn = min(mn, v);
    mx = max(mx, v);
  });
  // The high bits all keys share need no digit pass, and the first pass
  // then spreads the keys over its bins instead of piling them into a few.
  mx = block_max<kTauBS>(mx, sel.wsum);
  mn = ~block_max<kTauBS>(~mn, sel.wsum);
  const int nbits = a.keybits - shared_prefix_bits(mn, mx, a.keybits);
  SelectResult r;
  bool done = false;
  if (nbits > kSelDigit) {
    // One digit pass over the whole union finds the bin that holds rank t;
    // t is a small part of the union, so that bin holds few keys.  They are
    // copied to a short list and the remaining digits are taken on the list
    // alone.  A bin too full for the list falls through to the passes below.
    const int shift = nbits - kSelDigit;
    const uint32_t hmask = nbits >= 32 ? 0u : ~((1u << nbits) - 1u);
    const uint32_t pre = mn & hmask;
    for (uint32_t i = tid; i < static_cast<uint32_t>(kSelBins); i += kTauBS) sel.hist[i] = 0;
    __syncthreads();
    // Keys equal to the minimum (a sample of ReLU outputs is mostly +0) are
    // counted apart and added to their bin once: on one LDS address every
    // wave's increment would wait for the others'.
    uint32_t n_min = 0;
    all([&](uint32_t v) {
      if (v == mn) ++n_min;
      else hist_add(sel.hist, (v >> shift) & (kSelBins - 1), true);
    });
    n_min = block_sum<kTauBS>(n_min, sel.wsum);
    if (tid == 0 && n_min) sel.hist[(mn >> shift) & (kSelBins - 1)] += n_min;
    __syncthreads();
    if (tid < kWave) rank_bin_search(sel.hist, kSelBins, a.t, sel.scratch());
    __syncthreads();
    const uint32_t d = sel.found[0], above = sel.found[1], eq = sel.found[2];
    if (eq <= kTauList) {
      if (tid == 0) list_n[0] = 0;
      __syncthreads();
      all([&](uint32_t v) {
        const bool take = ((v >> shift) & (kSelBins - 1)) == d;
        const uint32_t p = lds_append(&list_n[0], take);
        if (take) tlist[p] = v;
      });
      __syncthreads();
      if (eq <= kListRankMax) {
        list_kth<kTauBS>(tlist, eq, a.t - above, &list_n[1]);
        __syncthreads();
        r.kth = list_n[1];
      } else {
        r = block_select_kth<kTauBS>(
            [&](auto f) {
              for (uint32_t i = tid; i < eq; i += kTauBS) f(tlist[i]);
            },
            a.t - above, shift, pre | (d << shift), sel);
      }
      done = true;
    }
  }
  if (!done) r = block_select_kth<kTauBS>(all, a.t, nbits, mn, sel);
  if (tid == 0) a.st->tau_key = r.kth;
}

// ------------------------------------------------------ stage 2, pairs ----
// Lexicographic plans: once tau is in the call state, every sample block
// draws its 1024 draws again (Philox words and gathers, as k_sample), counts
// those above tau and lists the indices of those equal to it (one atomic
// per block for each); the last block to finish takes i_tau, the
// (t - above)-th smallest listed index, with multiplicity.
struct TauIdxArgs {
  const void* values;
  uint64_t n, seed, row;
  uint32_t S, t;
  CallState* st;
  uint32_t* list;  // S entries
};

template <int DT>
__global__ __launch_bounds__(kSampBS) void k_tau_index(TauIdxArgs a) {
  __shared__ uint32_t s_list[kSampPerBlock];
  __shared__ SelectShared sel;
  __shared__ uint32_t s_n, s_base, s_last;
  const uint32_t tid = threadIdx.x, tau = a.st->tau_key;
  const uint32_t j0 = blockIdx.x * kSampPerBlock;
  if (tid == 0) s_n = 0;
  __syncthreads();
  uint32_t above = 0;
  {
    const U64x4 r = philox4x64_10(static_cast<uint64_t>(j0 / 4) + tid, a.row, 0, 0, a.seed, 0);
    uint32_t raw[4], ix[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool in = j0 + 4 * tid + q < a.S;
      ix[q] = in ? index_of_word(r.w[q], a.n) : 0u;
      raw[q] = in ? load_raw<DT>(a.values, ix[q]) : 0u;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (j0 + 4 * tid + q >= a.S) continue;
      const uint32_t key = key_of<DT>(raw[q]);
      if (key > tau) ++above;
      else if (key == tau) s_list[atomicAdd(&s_n, 1u)] = ix[q];
    }
  }
  const uint32_t blk_above = block_sum<kSampBS>(above, sel.wsum);
  __syncthreads();
  const uint32_t nb = s_n;
  if (tid == 0) {
    if (blk_above) atomicAdd(&a.st->tie_above, blk_above);
    s_base = nb ? atomicAdd(&a.st->tie_n, nb) : 0u;
  }
  __syncthreads();
  for (uint32_t i = tid; i < nb; i += kSampBS) store_agent(&a.list[s_base + i], s_list[i]);
  wait_memory();
  __syncthreads();
  if (tid == 0) s_last = atomicAdd(&a.st->tie_ticket, 1u) == gridDim.x - 1 ? 1u : 0u;
  __syncthreads();
  if (!s_last) return;
  acquire_agent();
  const uint32_t a_tot = a.st->tie_above, ne = a.st->tie_n;
  uint32_t i_tau = 0xFFFFFFFFu;
  if (ne > 0 && a_tot < a.t) {
    const uint32_t r = min(a.t - a_tot, ne);
    const uint32_t* list = a.list;
    i_tau = ~block_select_kth<kSampBS>(
                 [&](auto f) {
                   for (uint32_t i = tid; i < ne; i += kSampBS) f(~list[i]);
                 },
                 r, 32, 0u, sel)
                 .kth;
  }
  if (tid == 0) a.st->tau_idx = i_tau;
}

struct InitArgs {
  CallState* st;
  uint32_t* seg_cnt;
  uint32_t* fhist;
  uint32_t* bcur;   // null unless the call takes the large-k path
  uint32_t* ghist;  // null unless the call takes the large-k path
  uint32_t tau_key;
};

__global__ void k_init_state(InitArgs a) {
  reset_state(a.st, a.seg_cnt, a.fhist, a.bcur, a.ghist);
  if (threadIdx.x == 0) a.st->tau_key = a.tau_key;
}

// ------------------------------------------------------------ stage 4 -----
constexpr uint32_t kFinCache = 28672;
// The bucket refinement reads the candidate keys segment by segment as
// aligned 16-byte vectors: kPreThreads threads per segment, kPreV vectors
// each loaded before the segment counts are known, kSweepV per later sweep.
// A vector may start up to 3 entries before its segment (the previous
// segment's) or end up to 3 past its capacity (still within the workspace);
// such entries are skipped by their index.
constexpr uint32_t kPreThreads = kFinBS / kSegs;
constexpr int kPreV = 4;
constexpr int kSweepV = 8;
static_assert(kPreThreads * kSegs == kFinBS, "threads per segment");
constexpr int kFinDigit = 12;
// The bucket refinement spreads the buckets at or above the bucket of rank k
// over up to kFinRefMax workgroups, one per kFinRefWork units of work (a
// bucket of m candidates weighs m^2 + kFinRankW*m: its ranking compares and
// the placing, gathering and writing of its entries).  Every workgroup
// derives the same partition from the histogram, scans all candidates and
// keeps those of its own buckets: no workgroup hands anything to another.
constexpr uint32_t kFinRefMax = 32;
constexpr uint32_t kFinRefWork = 16384;
constexpr uint32_t kFinRankW = 64;

// LDS of the general refinement (radix select over the candidates).
struct FinShared {
  uint32_t cache[kFinCache];       // candidate keys; later the sort's exchange buffers
  uint64_t sortbuf[kFinMaxK];      // radix histogram, then the collected top k
  SelectScratch sel;
  uint32_t misc[8];
  __device__ __forceinline__ TopkSmem topk() {
    return TopkSmem{cache, kFinCache, reinterpret_cast<uint32_t*>(sortbuf), sortbuf, &sel, &misc[0]};
  }
};

// LDS of the bucket refinement: the candidates at or above the bucket of
// rank k, placed bucket by bucket in descending bucket order.
struct BucketShared {
  alignas(16) uint32_t off[kLogBins];   // first slot of each bucket
  alignas(16) uint32_t fill[kLogBins];  // entries placed in each bucket
  uint64_t comp[kFastCap];         // (key, ~index) composites
};

union FinLds {
  FinShared gen;
  BucketShared bkt;
  uint32_t hist[kLogBins];         // a block's histogram of its slice
};

// The filter's candidates: segment x holds n_x entries at x*cap; candidate i
// is entry i - pre[x] of the segment with pre[x] <= i < pre[x+1].
struct SegSrc {
  const uint32_t *key, *idx;
  uint32_t cap;
  const uint32_t* pre;  // LDS, kSegs + 1 entries
  __device__ __forceinline__ size_t pos(uint32_t i) const {
    uint32_t x = 0;
#pragma unroll
    for (int j = 1; j < kSegs; ++j) x += (i >= pre[j]) ? 1u : 0u;
    return static_cast<size_t>(x) * cap + (i - pre[x]);
  }
  template <int BS, class F>
  __device__ __forceinline__ void visit(uint32_t n, const uint32_t* cache, F f) const {
    // two loops, so that each load has one address space (a pointer chosen
    // between the LDS cache and the segments would be loaded as generic)
    auto body = [&](uint32_t i, uint32_t v) { f(i, v, LoadIdx{idx + pos(i)}); };
    if (cache) for_items<BS, 8>(n, [&](uint32_t i) { return cache[i]; }, body);
    else for_items<BS, 8>(n, [&](uint32_t i) { return key[pos(i)]; }, body);
  }
  __device__ __forceinline__ uint32_t idx_at(uint32_t i) const { return idx[pos(i)]; }
  __device__ __forceinline__ uint2 pair_at(uint32_t i) const {
    const size_t p = pos(i);
    return uint2{key[p], idx[p]};
  }
};

// The part of the input one fallback block owns, in index order: chunk b
// holds the aligned 16-byte vectors [v0, v1) (v0 = b*cv; the last chunk
// runs to the last vector); chunk 0 also holds the `head` elements before
// the first aligned vector and the last chunk the elements after the last
// one (fewer than a vector each).
template <int DT, int BS>
struct ChunkSrc {
  static constexpr int EPV = Elem<DT>::EPV, ES = Elem<DT>::ES;
  const void* values;
  uint32_t n, head, v0, v1;
  bool first, last;
  uint32_t* counter;  // one LDS word
  uint32_t* wsum;     // LDS scratch of block_excl_sum
  __device__ __forceinline__ const u32x4* vec() const {
    return reinterpret_cast<const u32x4*>(static_cast<const char*>(values) + static_cast<size_t>(head) * ES);
  }
  static __device__ __forceinline__ uint32_t raw_of(const u32x4& x, int e) {
    return DT == 0 ? x[e] : (x[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
  }
  __device__ __forceinline__ uint32_t tail0() const { return head + v1 * EPV; }
  template <class F>
  __device__ __forceinline__ void keys(F f) const {
    constexpr int U = 8;
    const u32x4* vp = vec();
    const uint32_t tid = threadIdx.x;
    for (uint32_t vb = v0; vb < v1; vb += BS * U) {
      u32x4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t vi = vb + u * BS + tid;
        x[u] = vi < v1 ? vp[vi] : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t vi = vb + u * BS + tid;
        if (vi < v1) {
#pragma unroll
          for (int e = 0; e < EPV; ++e) f(head + vi * EPV + e, key_of<DT>(raw_of(x[u], e)));
        }
      }
    }
    if (first)
      for (uint32_t i = tid; i < head; i += BS) f(i, key_of<DT>(load_raw<DT>(values, i)));
    if (last)  // fewer than a vector's elements, so no offset passes 2^32
      for (uint32_t o = tid; o < n - tail0(); o += BS) f(tail0() + o, key_of<DT>(load_raw<DT>(values, tail0() + o)));
  }
  __device__ __forceinline__ uint32_t idx_of(uint32_t pos) const { return pos; }
  // g(index, r) for the m elements equal to `key` of smallest index: one
  // vector per thread per sweep, ranked by a block-wide exclusive scan
  template <class G>
  __device__ __forceinline__ void ties_in_order(uint32_t key, uint32_t m, G g) const {
    const uint32_t tid = threadIdx.x;
    uint32_t taken = 0;
    auto scalar = [&](uint32_t s0, uint32_t s1) {  // fewer than EPV elements: one thread
      if (tid == 0) {
        uint32_t c = taken;
        for (uint32_t i = s0; i < s1; ++i)
          if (c < m && key_of<DT>(load_raw<DT>(values, i)) == key) g(i, c++);
        *counter = c;
      }
      __syncthreads();
      taken = *counter;
      __syncthreads();
    };
    if (first) scalar(0u, head);
    const u32x4* vp = vec();
    for (uint32_t vb = v0; vb < v1 && taken < m; vb += BS) {
      const uint32_t vi = vb + tid;
      uint32_t mask = 0;
      if (vi < v1) {
        const u32x4 x = vp[vi];
#pragma unroll
        for (int e = 0; e < EPV; ++e) mask |= (key_of<DT>(raw_of(x, e)) == key ? 1u : 0u) << e;
      }
      uint32_t tot;
      uint32_t r = taken + block_excl_sum<BS>(static_cast<uint32_t>(__popc(mask)), wsum, &tot);
      while (mask) {
        const uint32_t e = __builtin_ctz(mask);
        mask &= mask - 1;
        if (r < m) g(head + vi * EPV + e, r);
        ++r;
      }
      taken += tot;
    }
    if (last && taken < m) scalar(tail0(), n);
  }
};

// A run of R (key, index) pairs at positions [off, off + R) of two global
// arrays: results of fallback chunks or chunk groups, k pairs each, in no
// particular order.  Keys are read as aligned 16-byte vectors, which may
// reach up to 3 words on either side of the run (the arrays have slack).
template <int BS>
struct CandSrc {
  const uint32_t *key, *idx;
  uint32_t off, R;
  uint32_t* hist;       // LDS, 2^kSelDigit words, for ties_in_order
  SelectScratch* scr;   // LDS scratch of the select
  uint32_t* counter;    // one LDS word
  template <class F>
  __device__ __forceinline__ void keys(F f) const {
    constexpr int U = 8;
    const u32x4* kv = reinterpret_cast<const u32x4*>(key);
    const uint32_t end = off + R, vb0 = off / 4, nv = (end + 3) / 4, tid = threadIdx.x;
    for (uint32_t vb = vb0; vb < nv; vb += BS * U) {
      u32x4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t vi = vb + u * BS + tid;
        x[u] = vi < nv ? kv[vi] : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t vi = vb + u * BS + tid;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t p = vi * 4 + e;
          if (vi < nv && p >= off && p < end) f(p, x[u][e]);
        }
      }
    }
  }
  __device__ __forceinline__ uint32_t idx_of(uint32_t pos) const { return idx[pos]; }
  // the m smallest indices among the pairs with key kv: a radix select on
  // ~index over those pairs, then one collect pass
  template <class G>
  __device__ __forceinline__ void ties_in_order(uint32_t kv, uint32_t m, G g) const {
    const SelectResult r = block_select_kth<BS, kSelDigit>(
        [&](auto f) {
          keys([&](uint32_t pos, uint32_t k) {
            if (k == kv) f(~idx[pos]);
          });
        },
        m, 32, 0u, hist, *scr);
    const uint32_t istar = ~r.kth;
    if (threadIdx.x == 0) *counter = 0;
    __syncthreads();
    keys([&](uint32_t pos, uint32_t k) {
      const bool take = k == kv && idx[pos] <= istar;
      const uint32_t q = lds_append(counter, take);
      if (take) g(pos, q);
    });
    __syncthreads();
  }
};

struct FinishArgs {
  const void* values;
  uint32_t n, k, k_req, M;
  int direct;
  uint32_t G_f, seg_cap;
  const uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  CallState* st;
  uint32_t head, nvec, cv;          // fallback chunks: see ChunkSrc
  uint32_t *cand_key, *cand_idx;    // each chunk's top k, chunk b at b*k
  uint32_t *grp_key, *grp_idx;      // each chunk group's top k, group g at g*k
  const uint32_t* fhist;           // the filter's histogram of log_bin(key - tau)
  void* out_vals;
  int64_t* out_idx;
  profk_info_t* info;
};

// Refinement of a filtered call (k_req <= total <= M), from the filter's
// histogram of log_bin(key - tau) over the candidates:
//   1. find the bucket b* holding rank kk;
//   2. when the candidates at or above b* are few and ranking them within
//      their buckets takes few comparisons (the squares of the bucket sizes),
//      share those buckets out among the first G' workgroups (b < G'); each
//      places the candidates of its buckets in LDS, bucket by bucket, and
//      ranks each one within its bucket by comparison: its output position
//      is the bucket's first slot plus the number of larger composites in
//      the bucket;
//   3. otherwise workgroup 0 runs the general radix refinement.
// Called by workgroups b < kFinRefMax; b = 0 also writes the report.
template <int DT>
__device__ __forceinline__ void finish_filtered(const FinishArgs& a, FinLds& sh, const uint32_t* seg_pre,
                                                const uint32_t* seg_n, uint32_t total, SelectScratch& fs,
                                                const uint32_t (&h)[4], const uint4 (&pv)[kPreV], uint32_t b,
                                                uint32_t* tmp) {
  constexpr int KB = Elem<DT>::KEYBITS;
  const uint32_t tid = threadIdx.x;
  const uint32_t tau = a.st->tau_key;
  const SegSrc src{a.seg_key, a.seg_idx, a.seg_cap, seg_pre};
  const uint32_t kk = min(a.k, total);

  // 1. bucket offsets and weight prefixes in descending bucket order:
  //    thread t owns buckets [kLogBins - 4(t+1), kLogBins - 4t).  The weight
  //    of a bucket of m candidates is m^2, the compares that rank them, plus
  //    kFinRankW*m.  A prefix from the top covers higher buckets only, so the
  //    prefixes and the total W through b* cannot wrap when
  //    n_sel <= kFastCap (W <= n_sel^2 + kFinRankW*n_sel); the sums below b*
  //    may, and are not used.
  constexpr uint32_t kOwners = kLogBins / 4;
  static_assert(kLogBins % 4 == 0 && kOwners <= kFinBS, "bucket ownership");
  const uint32_t bbase = kLogBins - 4 * (tid + 1);  // h: loaded by the caller
  uint32_t* const own = tmp;
  uint32_t wt[4], wsum = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    wt[j] = h[j] * h[j] + kFinRankW * h[j];
    wsum += wt[j];
  }
  uint32_t above_me, wabove, tot_n, tot_w;
  block_excl_sum2<kFinBS>(h[0] + h[1] + h[2] + h[3], wsum, tmp + 4, above_me, wabove, tot_n, tot_w);
  if (tid < kOwners) {
    uint32_t run = above_me, wrun = wabove, o[4];
#pragma unroll
    for (int j = 3; j >= 0; --j) {
      o[j] = run;
      if (run < kk && kk <= run + h[j]) {
        fs.found[0] = bbase + j;
        fs.found[1] = run;
        fs.found[2] = h[j];
        fs.found[3] = wrun + wt[j];
      }
      run += h[j];
      wrun += wt[j];
    }
    // one 16-byte write per array (4-byte writes at a 16-byte stride would
    // collide on the LDS banks)
    *reinterpret_cast<uint4*>(&sh.bkt.off[bbase]) = uint4{o[0], o[1], o[2], o[3]};
    *reinterpret_cast<uint4*>(&sh.bkt.fill[bbase]) = uint4{0u, 0u, 0u, 0u};
  }
  if (tid == 0) {
    own[0] = kLogBins;
    own[1] = 0;
    own[2] = 0xFFFFFFFFu;
    own[3] = 0;
  }
  __syncthreads();
  const uint32_t bstar = fs.found[0], n_sel = fs.found[1] + fs.found[2], W = fs.found[3];

  if (n_sel <= kFastCap && W - kFinRankW * n_sel <= kFastCost) {
    // Partition: bucket j (descending order) goes to workgroup
    // min(G' - 1, floor(G' * W_j / W)), W_j the weight of the buckets above
    // it, so each workgroup holds a run of consecutive buckets: bins
    // [own[0], own[1]] and output slots [own[2], own[3]).
    const uint32_t G = min(min(gridDim.x, kFinRefMax), max(1u, (W + kFinRefWork - 1) / kFinRefWork));
    if (b >= G) return;
    uint32_t lo = kLogBins, hi = 0, s0 = 0xFFFFFFFFu, s1 = 0;
    if (G == 1) {
      // one workgroup: every bucket at or above b*, slots [0, n_sel)
      lo = bstar;
      hi = kLogBins - 1;
      s0 = 0;
      s1 = n_sel;
    } else if (tid < kOwners) {
      uint32_t run = above_me, wrun = wabove;
      // part == b exactly when b*W <= G*W_j < (b+1)*W (the last part takes
      // the rest); every product is below 2^32 since W <= 2^26 + 2^19
      const uint32_t lo_w = b * W, hi_w = b + 1 < G ? (b + 1) * W : 0xFFFFFFFFu;
#pragma unroll
      for (int j = 3; j >= 0; --j) {
        const uint32_t gw = wrun * G;
        if (h[j] > 0 && bbase + j >= bstar && gw >= lo_w && (gw < hi_w || b + 1 == G)) {
          lo = min(lo, bbase + j);
          hi = max(hi, bbase + j);
          s0 = min(s0, run);
          s1 = max(s1, run + h[j]);
        }
        run += h[j];
        wrun += wt[j];
      }
    }
    if (G > 1) {
      lo = ~wave_max_u32(~lo);
      hi = wave_max_u32(hi);
      s0 = ~wave_max_u32(~s0);
      s1 = wave_max_u32(s1);
      if ((tid & (kWave - 1)) == 0 && lo <= hi) {
        atomicMin(&own[0], lo);
        atomicMax(&own[1], hi);
        atomicMin(&own[2], s0);
        atomicMax(&own[3], s1);
      }
      __syncthreads();
      lo = own[0];
      hi = own[1];
      s0 = own[2];
      s1 = own[3];
      if (lo > hi) return;  // every bucket of this share lies in a heavier neighbour's
    }
    const uint32_t bin_lo = lo, bin_hi = hi, slo = s0, n_own = s1 - s0;
    // place (key, candidate number) of the buckets [bin_lo, bin_hi]: thread t takes
    // vectors t % kPreThreads + kPreThreads * u of segment t / kPreThreads,
    // the first kPreV of them already in registers
    const uint32_t x = tid / kPreThreads, l = tid % kPreThreads;
    const uint32_t nx = seg_n[x], px = seg_pre[x];
    const uint32_t b0 = x * a.seg_cap;                  // the segment's first entry
    const uint32_t v0 = b0 / 4, v1 = (b0 + nx + 3) / 4;  // vectors that cover its entries
    // Every candidate's key is >= tau, and one lies in a bucket >= bin_lo
    // exactly when key - tau >= log_bin_edge(bin_lo), i.e. key >= thr: the
    // sum cannot wrap, since bucket bin_lo holds a candidate.  Most vectors
    // hold no such key and cost four compares.
    const uint32_t thr = tau + log_bin_edge(bin_lo);
    auto place_vec = [&](uint32_t v, const uint4& q) {
      if (__builtin_expect((q.x >= thr) | (q.y >= thr) | (q.z >= thr) | (q.w >= thr), 0)) {
        const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t i = 4 * v + e, key = w4[e];
          if (key >= thr && i >= b0 && i < b0 + nx) {
            const uint32_t bin = log_bin(key - tau);
            if (bin <= bin_hi) {
              const uint32_t slot = sh.bkt.off[bin] - slo + atomicAdd(&sh.bkt.fill[bin], 1u);
              sh.bkt.comp[slot] = (static_cast<uint64_t>(key) << 32) | (px + i - b0);
            }
          }
        }
      }
    };
#pragma unroll
    for (int u = 0; u < kPreV; ++u) {
      const uint32_t v = v0 + l + kPreThreads * u;
      if (v < v1) place_vec(v, pv[u]);
    }
    const uint4* const kv4 = reinterpret_cast<const uint4*>(a.seg_key);
    for (uint32_t vb = v0 + kPreThreads * kPreV; vb < v1; vb += kPreThreads * kSweepV) {
      uint4 q[kSweepV];
#pragma unroll
      for (int u = 0; u < kSweepV; ++u) {
        const uint32_t v = vb + l + kPreThreads * u;
        q[u] = v < v1 ? kv4[v] : uint4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < kSweepV; ++u) {
        const uint32_t v = vb + l + kPreThreads * u;
        if (v < v1) place_vec(v, q[u]);
      }
    }
    __syncthreads();
    // ... then turn them into composites, all index loads in flight at once
    constexpr int PER = kFastCap / kFinBS;
    uint32_t ix[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const uint32_t p = u * kFinBS + tid;
      ix[u] = p < n_own ? a.seg_idx[src.pos(static_cast<uint32_t>(sh.bkt.comp[p]))] : 0u;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const uint32_t p = u * kFinBS + tid;
      if (p < n_own) sh.bkt.comp[p] = composite(static_cast<uint32_t>(sh.bkt.comp[p] >> 32), ix[u]);
    }
    __syncthreads();
    // rank within the bucket, write the kk largest
    for (uint32_t p = tid; p < n_own; p += kFinBS) {
      const uint64_t c = sh.bkt.comp[p];
      const uint32_t bin = log_bin(comp_key(c) - tau);
      const uint32_t s = sh.bkt.off[bin] - slo, m = sh.bkt.fill[bin];
      const uint32_t dst = sh.bkt.off[bin] + count_greater(sh.bkt.comp, s, s + m, c);
      if (dst < kk) {
        const uint32_t bits = bits_of_key<DT>(comp_key(c));
        if (DT == 0) static_cast<uint32_t*>(a.out_vals)[dst] = bits;
        else static_cast<uint16_t*>(a.out_vals)[dst] = static_cast<uint16_t>(bits);
        a.out_idx[dst] = comp_idx(c);
      }
    }
    if (b == 0)
      for (uint32_t p = kk + tid; p < a.k; p += kFinBS) {  // relaxed recall: padding
        if (DT == 0) static_cast<uint32_t*>(a.out_vals)[p] = 0xFF800000u;
        else static_cast<uint16_t*>(a.out_vals)[p] = 0xFF80u;
        a.out_idx[p] = -1;
      }
  } else {
    if (b != 0) return;
    __syncthreads();
    uint32_t bm = 0;
    for (uint32_t i = tid; i < a.G_f; i += kFinBS) bm = max(bm, a.blk_max[i]);
    const uint32_t gmax = block_max<kFinBS>(bm, fs.wsum);
    block_topk<kFinBS, kFinDigit>(src, total, kk, tau, max(gmax, tau), KB, sh.gen.topk());
    sort_write_any<DT, kFinBS>(sh.gen.sortbuf, kk, a.k, reinterpret_cast<uint64_t*>(sh.gen.cache),
                               a.out_vals, a.out_idx);
  }
  if (b == 0 && tid == 0) {
    a.st->status = PROFK_STATUS_FILTERED;
    if (a.info) {
      a.info->count = total;
      a.info->tau_key = tau;
      a.info->status = PROFK_STATUS_FILTERED;
      a.info->n_valid = kk;
    }
  }
}

template <int DT>
__global__ __launch_bounds__(kFinBS) void k_finish(FinishArgs a) {
  __shared__ FinLds sh;
  __shared__ SelectScratch fs;
  __shared__ uint32_t seg_n[kSegs], seg_pre[kSegs + 1], flag;
  __shared__ uint32_t fin_tmp[4 + 2 * (kFinBS / kWave + 1)];
  constexpr int KB = Elem<DT>::KEYBITS;
  const uint32_t tid = threadIdx.x, b = blockIdx.x;
  uint32_t total = 0, status = PROFK_STATUS_DIRECT;
  // Blocks b < kFinRefMax load the bucket histogram and the first kPreV
  // vectors of candidate keys of every segment together with the segment
  // counts, before they know them, so the three latencies overlap (reads past
  // a segment's count stay within its capacity and are ignored).
  uint32_t h[4] = {0u, 0u, 0u, 0u};
  uint4 pv[kPreV];
  if (!a.direct && b < kFinRefMax) {
    const uint32_t bbase = kLogBins - 4 * (tid + 1);
    if (tid < kLogBins / 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(a.fhist + bbase);
      h[0] = v.x; h[1] = v.y; h[2] = v.z; h[3] = v.w;
    }
    // vectors that start within the segment's capacity (they end at most 3
    // entries past it)
    const uint32_t x = tid / kPreThreads, l = tid % kPreThreads;
    const uint32_t v0 = x * a.seg_cap / 4;
#pragma unroll
    for (int u = 0; u < kPreV; ++u) {
      const uint32_t v = v0 + l + kPreThreads * u;
      pv[u] = 4 * v < (x + 1) * a.seg_cap ? reinterpret_cast<const uint4*>(a.seg_key)[v] : uint4{0u, 0u, 0u, 0u};
    }
  }
  if (!a.direct) {
    if (tid < kWave) {
      const uint32_t c = tid < kSegs ? a.seg_cnt[tid * kSegStride] : 0u;
      const uint32_t incl = wave_incl_sum(c);
      if (tid < kSegs) {
        seg_n[tid] = c;
        seg_pre[tid] = incl - c;
      }
      if (tid == kSegs - 1) seg_pre[kSegs] = incl;
    }
    __syncthreads();
    total = seg_pre[kSegs];
    status = total < a.k_req ? PROFK_STATUS_UNDERFLOW
                             : (total > a.M ? PROFK_STATUS_OVERFLOW : PROFK_STATUS_FILTERED);
    if (status == PROFK_STATUS_FILTERED) {
      if (b < kFinRefMax) {
        finish_filtered<DT>(a, sh, seg_pre, seg_n, total, fs, h, pv, b, fin_tmp);
      } else {
        // The other workgroups have no work here: they read the candidates'
        // keys and indices, so that the refining ones find them in L2 and
        // not in HBM, which the filter's stream has flushed them to.  Each
        // XCD has an L2 of its own and workgroup b runs on XCD b % kXcds
        // (round-robin dispatch), so the idle workgroups of each XCD read
        // every line between them.  Each segment's vectors are those that
        // cover its entries (they end at most 3 entries past it, within the
        // workspace).
        static_assert(kFinRefMax % kXcds == 0, "idle workgroups start on XCD 0");
        const uint32_t xcd = b % kXcds, nx = (gridDim.x - kFinRefMax - xcd + kXcds - 1) / kXcds;
        const uint32_t nthr = nx * kFinBS, g = (b - kFinRefMax) / kXcds * kFinBS + tid;
        const uint4* const kv4 = reinterpret_cast<const uint4*>(a.seg_key);
        const uint4* const iv4 = reinterpret_cast<const uint4*>(a.seg_idx);
        uint32_t fold = 0;
        for (int x = 0; x < kSegs; ++x) {
          const uint32_t b0 = x * a.seg_cap, v0 = b0 / 4, v1 = (b0 + seg_n[x] + 3) / 4;
          for (uint32_t v = v0 + g; v < v1; v += nthr) {
            const uint4 q = kv4[v], r = iv4[v];
            fold ^= q.x ^ r.x;
          }
        }
        asm volatile("" : : "v"(fold));  // the loads are kept: their lines are the point
      }
      return;
    }
  }
  // Exact fallback: each block takes the exact top-k of its chunk ...
  constexpr int EPV = Elem<DT>::EPV;
  const uint32_t G = gridDim.x;
  const uint32_t tail = a.n - (a.head + a.nvec * EPV);
  // elements of chunk c (ChunkSrc's partition)
  auto chunk_n = [&](uint32_t c) {
    const uint32_t v0 = min(c * a.cv, a.nvec);
    const uint32_t v1 = c == G - 1 ? a.nvec : min(v0 + a.cv, a.nvec);
    return (v1 - v0) * EPV + (c == 0 ? a.head : 0u) + (c == G - 1 ? tail : 0u);
  };
  const TopkSmem sm = sh.gen.topk();
  {
    const uint32_t v0 = min(b * a.cv, a.nvec);
    const uint32_t v1 = b == G - 1 ? a.nvec : min(v0 + a.cv, a.nvec);
    const uint32_t kb = min(a.k, chunk_n(b));  // k for every chunk but possibly the last
    if (kb) {
      const ChunkSrc<DT, kFinBS> src{a.values, a.n, a.head, v0, v1, b == 0, b == G - 1, sm.counter, fs.wsum};
      window_topk<kFinBS, kFinDigit>(src, kb, KB, sm);
      for (uint32_t p = tid; p < kb; p += kFinBS) {
        const uint64_t c = sh.gen.sortbuf[p];
        store_agent(&a.cand_key[static_cast<size_t>(b) * a.k + p], comp_key(c));
        store_agent(&a.cand_idx[static_cast<size_t>(b) * a.k + p], comp_idx(c));
      }
    }
  }
  // ... the last chunk of each group of kFbGroup to finish merges the
  // group's results, and the last group to finish merges the groups'.
  const uint32_t NG = (G + kFbGroup - 1) / kFbGroup, gi = b / kFbGroup;
  const uint32_t g0 = gi * kFbGroup, gn = min(G - g0, static_cast<uint32_t>(kFbGroup));
  wait_memory();
  __syncthreads();
  if (tid == 0) flag = (atomicAdd(&a.st->grp_ticket[gi], 1u) == gn - 1) ? 1u : 0u;
  __syncthreads();
  if (!flag) return;
  acquire_agent();
  // pairs of the group: k from each chunk but the last, which holds fewer
  // only when it is the last chunk of the input
  const uint32_t rg = (gn - 1) * a.k + min(a.k, chunk_n(g0 + gn - 1));
  const CandSrc<kFinBS> group{a.cand_key, a.cand_idx, g0 * a.k, rg, sm.hist, sm.scratch, sm.counter};
  uint64_t* const exch = reinterpret_cast<uint64_t*>(sh.gen.cache);
  if (NG > 1) {
    const uint32_t kg = min(a.k, rg);
    window_topk<kFinBS, kFinDigit>(group, kg, KB, sm);
    for (uint32_t p = tid; p < kg; p += kFinBS) {
      const uint64_t c = sh.gen.sortbuf[p];
      store_agent(&a.grp_key[static_cast<size_t>(gi) * a.k + p], comp_key(c));
      store_agent(&a.grp_idx[static_cast<size_t>(gi) * a.k + p], comp_idx(c));
    }
    wait_memory();
    __syncthreads();
    if (tid == 0) flag = (atomicAdd(&a.st->ticket, 1u) == NG - 1) ? 1u : 0u;
    __syncthreads();
    if (!flag) return;
    acquire_agent();
    // every group but the last holds k; the last holds min(k, its pairs)
    const uint32_t gl = (NG - 1) * kFbGroup;
    const uint32_t rl = (G - gl - 1) * a.k + min(a.k, chunk_n(G - 1));
    const CandSrc<kFinBS> groups{a.grp_key, a.grp_idx, 0u, (NG - 1) * a.k + min(a.k, rl), sm.hist, sm.scratch,
                                 sm.counter};
    window_topk<kFinBS, kFinDigit>(groups, a.k, KB, sm);
  } else {
    window_topk<kFinBS, kFinDigit>(group, a.k, KB, sm);
  }
  sort_write_any<DT, kFinBS>(sh.gen.sortbuf, a.k, a.k, exch, a.out_vals, a.out_idx);
  if (tid == 0) {
    a.st->status = status;
    if (a.info) {
      a.info->count = a.direct ? 0u : total;
      a.info->tau_key = a.direct ? 0u : a.st->tau_key;
      a.info->status = static_cast<int32_t>(status);
      a.info->n_valid = a.k;
    }
  }
}

// ------------------------------------------------------ inspection ---------
__global__ void k_sample_indices(uint64_t seed, uint64_t row, uint32_t S, uint64_t n, int64_t* out) {
  const uint32_t blk = blockIdx.x * blockDim.x + threadIdx.x;
  if (static_cast<uint64_t>(blk) * 4 >= S) return;
  const U64x4 w = philox4x64_10(blk, row, 0, 0, seed, 0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint64_t j = static_cast<uint64_t>(blk) * 4 + q;
    if (j < S) out[j] = index_of_word(w.w[q], n);
  }
}

// Gathers the candidate segments into one contiguous buffer.
__global__ __launch_bounds__(1024) void k_gather_buffer(uint32_t cap, const uint32_t* seg_cnt,
                                                        const uint32_t* seg_key, const uint32_t* seg_idx,
                                                        uint32_t* out_key, uint32_t* out_idx, uint32_t* count) {
  __shared__ uint32_t pre[kSegs + 1];
  const uint32_t tid = threadIdx.x;
  if (tid == 0) {
    uint32_t run = 0;
    for (int x = 0; x < kSegs; ++x) {
      pre[x] = run;
      run += min(seg_cnt[x * kSegStride], cap);
    }
    pre[kSegs] = run;
    uint32_t total = 0;
    for (int x = 0; x < kSegs; ++x) total += seg_cnt[x * kSegStride];
    *count = total;
  }
  __syncthreads();
  SegSrc src{seg_key, seg_idx, cap, pre};
  const uint32_t stored = min(pre[kSegs], cap);
  src.visit<1024>(stored, nullptr, [&](uint32_t i, uint32_t key, auto idx) {
    out_key[i] = key;
    out_idx[i] = idx();
  });
}

// ------------------------------------------------------------- host -------
static inline uint32_t cdiv(uint64_t a, uint64_t b) { return static_cast<uint32_t>((a + b - 1) / b); }
static inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Length of the capped sample lists for a key-rule plan with t >
// kWaveTopMax, or 0 when the draws of a block in the top t are too many for
// kWaveTopMax to hold them with a margin of eight standard deviations.
static uint32_t capped_list_len(uint32_t S, uint32_t t, bool lex) {
  if (lex || t <= kWaveTopMax || S < 2u * kSampPerBlock) return 0;
  const double mu = static_cast<double>(kSampPerBlock) * t / S;
  const double need = mu + 8.0 * std::sqrt(mu) + 2.0;
  return need <= kCapListSmall ? kCapListSmall : (need <= kWaveTopMax ? kWaveTopMax : 0u);
}

FlatLayout flat_layout(const profk_plan_t& p, int dtype, int num_cus) {
  FlatLayout L;
  const uint64_t N = static_cast<uint64_t>(p.N);
  const uint32_t epv = dtype == PROFK_F32 ? 4 : 8;
  const uint32_t S = static_cast<uint32_t>(p.S), t = static_cast<uint32_t>(p.t);
  const uint32_t M = static_cast<uint32_t>(p.M), k = static_cast<uint32_t>(p.k);
  L.cap_list = capped_list_len(S, t, p.lexicographic != 0);
  L.samp_bs = (!p.lexicographic && t > kWaveTopMax && !L.cap_list) ? kSampWideBS : kSampBS;
  const uint32_t spb = 4u * L.samp_bs;
  const uint32_t tl = L.cap_list ? L.cap_list : t;  // length of a block's list
  L.G_s = cdiv(S, spb);
  L.tcap = tl < spb ? tl : spb;
  const uint32_t last_nb = S - (L.G_s - 1) * spb;
  L.union_n = (L.G_s - 1) * L.tcap + (tl < last_nb ? tl : last_nb);
  // Expected survivors per element are about t / (S + 1).
  const bool sparse = N * (dtype == PROFK_F32 ? 4u : 2u) >= kFiltSparseMinBytes &&
                      static_cast<uint64_t>(t) * kFiltSparseInvDensity < static_cast<uint64_t>(S) + 1;
  const int per_cu = filter_blocks_per_cu(dtype, sparse ? kFiltPerCuSparse : kFiltPerCuDense);
  const uint32_t maxg = static_cast<uint32_t>(num_cus * per_cu < kFiltMaxBlocks ? num_cus * per_cu : kFiltMaxBlocks);
  L.filt_u = N * (dtype == PROFK_F32 ? 4u : 2u) >= kFiltSparseMinBytes ? kFiltULarge : kFiltUSmall;
  L.filt_db = !sparse;
  uint32_t g = cdiv(cdiv(N, epv), kFiltBS * static_cast<uint32_t>(L.filt_u));
  L.G_f = g < 1 ? 1 : (g > maxg ? maxg : g);
  L.seg_cap = M;
  const uint32_t fbmax = static_cast<uint32_t>(num_cus < kFbMaxBlocks ? num_cus : kFbMaxBlocks);
  uint32_t gb = cdiv(N, kFbMinChunk);
  L.G_fb = gb < 1 ? 1 : (gb > fbmax ? fbmax : gb);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  L.off_state = take(sizeof(CallState));
  L.off_segcnt = take(static_cast<size_t>(kSegs) * kSegStride * 4);
  L.off_union = take(static_cast<size_t>(L.G_s) * L.tcap * 4);
  if (L.cap_list) {
    L.off_cut = take(static_cast<size_t>(L.G_s) * 4);
    L.off_all_keys = take(static_cast<size_t>(S) * 4);
  }
  L.off_blk_max = take(static_cast<size_t>(L.G_f) * 4);
  L.off_seg_key = take(static_cast<size_t>(kSegs) * M * 4);
  L.off_seg_idx = take(static_cast<size_t>(kSegs) * M * 4);
  L.big = k > static_cast<uint32_t>(kFinMaxK);
  if (L.big) {
    const size_t P = static_cast<size_t>(cdiv(k, kBigSortTile)) * kBigSortTile;
    L.G_big = static_cast<uint32_t>(num_cus < kBigMaxBlocks ? num_cus : kBigMaxBlocks);
    L.off_big_state = take(256);
    L.off_ghist = take(static_cast<size_t>(kBigBins) * 4);
    L.off_staging = take((P + kBktCap) * 8);
    L.off_runs = take(P * 8);
    L.off_bcur = take(static_cast<size_t>(kLogBins) * kBktPad * 4);
    L.off_blist = take(static_cast<size_t>(kLogBins) * 16);
  } else {
    // the merges read keys as aligned 16-byte vectors: 4 words of slack
    const size_t NG = (L.G_fb + kFbGroup - 1) / kFbGroup;
    L.off_cand_key = take((static_cast<size_t>(L.G_fb) * k + 4) * 4);
    L.off_cand_idx = take(static_cast<size_t>(L.G_fb) * k * 4);
    L.off_grp_key = take((NG * k + 4) * 4);
    L.off_grp_idx = take(NG * k * 4);
  }
  L.off_fhist = take(static_cast<size_t>(kLogBins) * 4);
  if (p.lexicographic) L.off_tie = take(static_cast<size_t>(S) * 4);
  L.bytes = off;
  return L;
}

template <class T> static T* at(uint8_t* ws, size_t off) { return reinterpret_cast<T*>(ws + off); }

// Stages 4 and 5 on the candidates the filter left in the workspace (G_f
// workgroups wrote blk_max); the fallback reads c.values.
template <int DT>
static hipError_t launch_refine_t(const FlatCall& c, bool direct, uint32_t G_f) {
  const FlatLayout& L = c.L;
  const profk_plan_t& p = *c.plan;
  CallState* st = at<CallState>(c.ws, L.off_state);
  uint32_t* seg_cnt = at<uint32_t>(c.ws, L.off_segcnt);
  uint32_t* fhist = at<uint32_t>(c.ws, L.off_fhist);
  if (L.big) {
    BigCall bc{DT, c.values, c.n, c.k, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.M),
               direct ? 1 : 0, seg_cnt, at<uint32_t>(c.ws, L.off_seg_key), at<uint32_t>(c.ws, L.off_seg_idx),
               at<uint32_t>(c.ws, L.off_blk_max), L.seg_cap, G_f, st, c.ws + L.off_big_state,
               at<uint32_t>(c.ws, L.off_ghist), at<uint64_t>(c.ws, L.off_staging), at<uint64_t>(c.ws, L.off_runs),
               fhist, at<uint32_t>(c.ws, L.off_bcur),
               at<uint32_t>(c.ws, L.off_blist),
               L.G_big, c.out_vals, c.out_idx, c.info, c.stream};
    return launch_big(bc);
  }
  // Fallback chunks (ChunkSrc): whole 16-byte vectors after the unaligned
  // head, as the filter splits the input, and at least max(k, kFbMinChunk)
  // elements each, so that every chunk but the last holds k of the top.
  constexpr int ES = Elem<DT>::ES, EPV = Elem<DT>::EPV;
  const uintptr_t addr = reinterpret_cast<uintptr_t>(c.values);
  uint32_t head = static_cast<uint32_t>(((16 - (addr & 15)) & 15) / ES);
  if (head > c.n) head = c.n;
  const uint32_t nvec = (c.n - head) / EPV;
  const uint64_t min_chunk = c.k > kFbMinChunk ? c.k : kFbMinChunk;
  const uint64_t gmax = static_cast<uint64_t>(nvec) * EPV / min_chunk;
  const uint32_t G_fb = gmax < 1 ? 1u : (gmax < L.G_fb ? static_cast<uint32_t>(gmax) : L.G_fb);
  FinishArgs fa{c.values, c.n, c.k, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.M),
                direct ? 1 : 0, G_f, L.seg_cap,
                seg_cnt, at<uint32_t>(c.ws, L.off_seg_key), at<uint32_t>(c.ws, L.off_seg_idx),
                at<uint32_t>(c.ws, L.off_blk_max), st,
                head, nvec, cdiv(nvec, G_fb), at<uint32_t>(c.ws, L.off_cand_key), at<uint32_t>(c.ws, L.off_cand_idx),
                at<uint32_t>(c.ws, L.off_grp_key), at<uint32_t>(c.ws, L.off_grp_idx),
                fhist, c.out_vals, c.out_idx, c.info};
  hipLaunchKernelGGL(k_finish<DT>, dim3(G_fb), dim3(kFinBS), 0, c.stream, fa);
  return hipGetLastError();
}

template <int DT>
static hipError_t launch_flat_t(const FlatCall& c) {
  const FlatLayout& L = c.L;
  const profk_plan_t& p = *c.plan;
  CallState* st = at<CallState>(c.ws, L.off_state);
  uint32_t* seg_cnt = at<uint32_t>(c.ws, L.off_segcnt);
  const bool direct = p.mode == PROFK_MODE_DIRECT && !c.use_tau;
  const bool lex = p.lexicographic && !direct && !c.use_tau;  // a caller's tau: the key rule
  uint32_t* fhist = at<uint32_t>(c.ws, L.off_fhist);
  uint32_t* bcur = L.big ? at<uint32_t>(c.ws, L.off_bcur) : nullptr;
  uint32_t* ghist = L.big ? at<uint32_t>(c.ws, L.off_ghist) : nullptr;
  const uint32_t* union_for_filter = nullptr;
  hipError_t e;
  if (direct || c.use_tau) {
    hipLaunchKernelGGL(k_init_state, dim3(1), dim3(64), 0, c.stream,
                       InitArgs{st, seg_cnt, fhist, bcur, ghist, c.use_tau ? c.tau_key : 0u});
  } else {
    uint32_t* uk = at<uint32_t>(c.ws, L.off_union);
    SampleArgs sa{c.values, c.n, c.seed, c.row, static_cast<uint32_t>(p.S),
                  L.cap_list ? L.cap_list : static_cast<uint32_t>(p.t), L.tcap, uk, st, seg_cnt, fhist, bcur, ghist,
                  L.cap_list ? at<uint32_t>(c.ws, L.off_cut) : nullptr,
                  L.cap_list ? at<uint32_t>(c.ws, L.off_all_keys) : nullptr};
    if (L.samp_bs == kSampWideBS) hipLaunchKernelGGL((k_sample<DT, kSampWideBS>), dim3(L.G_s), dim3(kSampWideBS), 0, c.stream, sa);
    else hipLaunchKernelGGL((k_sample<DT, kSampBS>), dim3(L.G_s), dim3(kSampBS), 0, c.stream, sa);
    if (!lex && L.union_n <= kFiltTauMax && static_cast<uint32_t>(p.t) <= kFiltTauInMaxT) {
      union_for_filter = uk;
    } else {
      TauArgs ta{uk, L.union_n, static_cast<uint32_t>(p.t), Elem<DT>::KEYBITS, st,
                 L.cap_list ? at<uint32_t>(c.ws, L.off_cut) : nullptr, L.G_s,
                 L.cap_list ? at<uint32_t>(c.ws, L.off_all_keys) : nullptr, static_cast<uint32_t>(p.S)};
      hipLaunchKernelGGL(k_select_tau, dim3(1), dim3(kTauBS), 0, c.stream, ta);
      if (lex) {
        TauIdxArgs ti{c.values, c.n, c.seed, c.row, static_cast<uint32_t>(p.S), static_cast<uint32_t>(p.t), st,
                      at<uint32_t>(c.ws, L.off_tie)};
        hipLaunchKernelGGL(k_tau_index<DT>, dim3(L.G_s), dim3(kSampBS), 0, c.stream, ti);
      }
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!direct && (e = launch_filter(c, st, union_for_filter, lex)) != hipSuccess) return e;
  return launch_refine_t<DT>(c, direct, L.G_f);
}

hipError_t launch_flat(const FlatCall& c) {
  (void)hipGetLastError();  // report only errors of this call's launches
  return c.dtype == PROFK_F32 ? launch_flat_t<0>(c) : launch_flat_t<1>(c);
}

hipError_t launch_refine(const FlatCall& c, uint32_t G_f) {
  return c.dtype == PROFK_F32 ? launch_refine_t<0>(c, false, G_f) : launch_refine_t<1>(c, false, G_f);
}

hipError_t launch_select_tau(const uint32_t* union_keys, uint32_t n, uint32_t t, int keybits, CallState* st,
                             hipStream_t s) {
  TauArgs ta{union_keys, n, t, keybits, st};
  hipLaunchKernelGGL(k_select_tau, dim3(1), dim3(kTauBS), 0, s, ta);
  return hipGetLastError();
}

hipError_t launch_select_tau_keys(const uint32_t* keys, uint32_t n, uint32_t t, uint32_t* union_keys,
                                  size_t union_words, CallState* st, hipStream_t s) {
  constexpr uint32_t spb = 4u * kSampWideBS;
  const uint32_t G = cdiv(n, spb), tcap = t < spb ? t : spb;
  const uint32_t last_nb = n - (G - 1) * spb;
  const uint32_t un = (G - 1) * tcap + (t < last_nb ? t : last_nb);
  if (static_cast<uint64_t>(un) * 2 > n || static_cast<size_t>(G) * tcap > union_words)
    return launch_select_tau(keys, n, t, 32, st, s);  // no real reduction: select over the keys
  hipLaunchKernelGGL(k_key_union<kSampWideBS>, dim3(G), dim3(kSampWideBS), 0, s, keys, n, t, tcap, union_keys);
  return launch_select_tau(union_keys, un, t, 32, st, s);
}

hipError_t launch_sample_indices(uint64_t seed, uint64_t row, uint32_t S, uint64_t N, int64_t* out,
                                 hipStream_t s) {
  const uint32_t nblk = cdiv(S, 4);
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_sample_indices, dim3(cdiv(nblk, 256)), dim3(256), 0, s, seed, row, S, N, out);
  return hipGetLastError();
}

hipError_t launch_debug_filter(const FlatCall& c, uint32_t* buf_key, uint32_t* buf_idx,
                               uint32_t* count_dev) {
  const FlatLayout& L = c.L;
  CallState* st = at<CallState>(c.ws, L.off_state);
  uint32_t* seg_cnt = at<uint32_t>(c.ws, L.off_segcnt);
  (void)hipGetLastError();
  uint32_t* fhist = at<uint32_t>(c.ws, L.off_fhist);
  hipLaunchKernelGGL(k_init_state, dim3(1), dim3(64), 0, c.stream,
                     InitArgs{st, seg_cnt, fhist, L.big ? at<uint32_t>(c.ws, L.off_bcur) : nullptr,
                              L.big ? at<uint32_t>(c.ws, L.off_ghist) : nullptr, c.tau_key});
  hipError_t e = launch_filter(c, st, nullptr, false);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_gather_buffer, dim3(1), dim3(1024), 0, c.stream, L.seg_cap, seg_cnt,
                     at<uint32_t>(c.ws, L.off_seg_key), at<uint32_t>(c.ws, L.off_seg_idx),
                     buf_key, buf_idx, count_dev);
  return hipGetLastError();
}

int device_cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

}  // namespace profk
