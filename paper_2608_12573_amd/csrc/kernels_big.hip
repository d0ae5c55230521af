// Refinement and fallback for k above what one workgroup can hold (the
// BatchTopK case of Sec. 5: K = B*k of a flattened latent matrix).
//
// Same result as the one-block path -- the exact top-k under the total
// order, sorted -- computed across the GPU.  A filtered call whose
// candidates spread over small buckets takes the bucket path:
//   k_bkt_scatter  in every block, the status, bucket offsets in descending
//                  bucket order from the filter's histogram of
//                  log_bin(key - tau) and the bucket b* holding rank k
//                  (block 0 records the plan); then every candidate of a
//                  bucket >= b* into its bucket's range of the staging array.
//                  When the bucket path does not apply, the blocks run the
//                  radix path's first key digit pass instead;
//   k_bkt_sort     one block per bucket sorts it in LDS and writes the
//                  outputs at the bucket's offset.
// Every other call (a fallback, DIRECT, or a bucket larger than kBktCap)
// takes the radix path, whose kernels return at once after a bucket call
// (its source is the candidate segments, or the whole input on fallback):
//   radix passes   one radix digit per launch: block histograms are merged
//                  into a global histogram and the last block (ticket) picks
//                  the digit holding rank k.  Key digits first, then, if the
//                  tie class at the k-th key is split, digits of ~index.  The
//                  first two key digits are taken by the k_bkt_scatter and
//                  k_bkt_sort launches, the others by k_big_pass.
//   k_big_collect  every item of the top k, as a composite key, into a
//                  staging array (one atomic per block).
//   k_big_tile     sorts tiles of 16384 composites in LDS.
//   k_big_merge    merge-path passes doubling the sorted run length; the
//                  last pass (or the tile sort, for a single tile) writes
//                  values, indices and the per-call report.
#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"

namespace profk {

struct BigState {
  uint32_t status;     // PROFK_STATUS_* of the call
  uint32_t n_src;      // items in the source
  uint32_t from_input; // 1: the source is the input itself
  uint32_t kk;         // how many to select
  uint32_t total;      // filter survivors
  uint32_t tau;
  // key stage
  uint32_t prefix, krem, above, equal;
  int32_t hi;
  uint32_t kstar;
  // index stage (on ~index among keys equal to kstar)
  uint32_t cut;
  uint32_t iprefix, ikrem;
  int32_t ihi;
  uint32_t istar;
  uint32_t out_count;
  uint32_t mode;       // kModeRadix or kModeBucket
  uint32_t bstar;      // bucket path: the bucket holding rank kk
  uint32_t nlist;      // bucket path: entries of the bucket list
  uint32_t pad[43];
};
constexpr uint32_t kModeRadix = 0, kModeBucket = 1;
static_assert(sizeof(BigState) <= 256, "state size");

struct BigArgs {
  const void* values;
  uint32_t n, k, k_req, M;
  int direct;
  const uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  uint32_t seg_cap, G_f;
  CallState* st;
  BigState* bs;
  uint32_t* ghist;     // kBigBins
  uint64_t* staging;   // P
  uint64_t* runs;      // P
  const uint32_t* fhist;  // kLogBins: the filter's histogram of log_bin(key - tau)
  uint32_t* bcur;      // kLogBins * kBktPad: entries placed in bucket b at b * kBktPad
  uint4* blist;        // kLogBins: the non-empty buckets >= b*, descending: {bucket, first slot, size, 0}
  uint32_t P;          // padded length: k rounded up to kBigSortTile
  void* out_vals;
  int64_t* out_idx;
  profk_info_t* info;
};

// Candidate i of the segments: segment x holds n_x entries at x*cap.
struct SegPos {
  const uint32_t* n;  // kSegs counts (already capped)
  uint32_t cap;
  __device__ __forceinline__ size_t operator()(uint32_t i) const {
    uint32_t x = 0, base = 0;
#pragma unroll
    for (int j = 0; j < kSegs - 1; ++j) {
      if (x == static_cast<uint32_t>(j) && i >= base + n[j]) { base += n[j]; ++x; }
    }
    return static_cast<size_t>(x) * cap + (i - base);
  }
};

// Grid-stride visit of the call's source: f(key, index) for every item.
// Offsets are compared with the remaining count and a block stops before
// its next sweep could pass n, so n may be as large as 2^32 - 1.
template <int DT, int BS, class F>
__device__ __forceinline__ void big_visit(const BigArgs& a, uint32_t n, uint32_t from_input, const uint32_t* segn,
                                          F f) {
  const uint32_t stride = gridDim.x * BS * 8;
  if (from_input) {
    for (uint32_t base = blockIdx.x * BS * 8; base < n; base += stride) {
      const uint32_t rem = n - base;
      uint32_t kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t o = u * BS + threadIdx.x;
        kv[u] = o < rem ? key_of<DT>(load_raw<DT>(a.values, base + o)) : 0u;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t o = u * BS + threadIdx.x;
        if (o < rem) f(kv[u], base + o);
      }
      if (rem <= stride) break;
    }
  } else {
    const SegPos pos{segn, a.seg_cap};
    for (uint32_t base = blockIdx.x * BS * 8; base < n; base += stride) {
      const uint32_t rem = n - base;
      uint32_t kv[8], iv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t o = u * BS + threadIdx.x;
        if (o < rem) {
          const size_t p = pos(base + o);
          kv[u] = a.seg_key[p];
          iv[u] = a.seg_idx[p];
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t o = u * BS + threadIdx.x;
        if (o < rem) f(kv[u], iv[u]);
      }
      if (rem <= stride) break;
    }
  }
}

__device__ __forceinline__ void load_segn(const BigArgs& a, uint32_t* segn) {
  if (threadIdx.x < kSegs) segn[threadIdx.x] = min(a.seg_cnt[threadIdx.x * kSegStride], a.seg_cap);
  __syncthreads();
}

// ------------------------------------------------------------ radix path ---
// The radix path's state: what is selected from where (the header), and the
// digit state of the key stage and of the index stage (digits of ~index
// among the items whose key is kstar, when that tie class is split).
struct RadixHead {
  uint32_t status, total, tau, from_input, n_src, kk;
};
struct RadixVals {
  uint32_t prefix, krem, above, equal;
  int32_t hi;
  uint32_t kstar, cut, iprefix, ikrem;
  int32_t ihi;
  uint32_t istar;
};

__device__ __forceinline__ RadixHead radix_load_head(const BigState* s) {
  return RadixHead{s->status, s->total, s->tau, s->from_input, s->n_src, s->kk};
}
__device__ __forceinline__ RadixVals radix_load(const BigState* s) {
  return RadixVals{s->prefix, s->krem, s->above, s->equal, s->hi, s->kstar,
                   s->cut, s->iprefix, s->ikrem, s->ihi, s->istar};
}
__device__ __forceinline__ void radix_store_head(BigState* s, const RadixHead& h) {
  s->mode = kModeRadix;
  s->status = h.status;
  s->total = h.total;
  s->tau = h.tau;
  s->from_input = h.from_input;
  s->n_src = h.n_src;
  s->kk = h.kk;
  s->out_count = 0;
}
__device__ __forceinline__ void radix_store(BigState* s, const RadixVals& v) {
  s->prefix = v.prefix;
  s->krem = v.krem;
  s->above = v.above;
  s->equal = v.equal;
  s->hi = v.hi;
  s->kstar = v.kstar;
  s->cut = v.cut;
  s->iprefix = v.iprefix;
  s->ikrem = v.ikrem;
  s->ihi = v.ihi;
  s->istar = v.istar;
}

// The starting state from the call's status.  Every thread of a block of
// BS calls it, and every block derives the same values.
template <int DT, int BS>
__device__ __forceinline__ void radix_init(const BigArgs& a, uint32_t status, uint32_t total, uint32_t* wsum,
                                           RadixHead& h, RadixVals& v) {
  constexpr int KB = Elem<DT>::KEYBITS;
  const uint32_t key_max = KB == 32 ? 0xFFFFFFFFu : 0xFFFFu;
  const bool filtered = status == PROFK_STATUS_FILTERED;
  uint32_t lo = 0, hi = key_max;
  if (filtered) {
    lo = a.st->tau_key;
    uint32_t bm = 0;
    for (uint32_t i = threadIdx.x; i < a.G_f; i += BS) bm = max(bm, a.blk_max[i]);
    hi = max(lo, block_max<BS>(bm, wsum));
  }
  h.status = status;
  h.total = total;
  h.tau = a.direct ? 0u : a.st->tau_key;
  h.from_input = filtered ? 0u : 1u;
  h.n_src = filtered ? total : a.n;
  h.kk = filtered ? min(a.k, total) : a.k;
  v.prefix = lo;
  v.krem = h.kk;
  v.above = 0;
  v.equal = 0;
  v.hi = KB - shared_prefix_bits(lo, hi, KB);
  v.kstar = lo;
  v.cut = 0;
  v.iprefix = 0;
  v.ikrem = 0;
  v.ihi = 0;
  v.istar = 0xFFFFFFFFu;
  if (v.hi == 0) {
    // every candidate carries the same key: only the index cut is left
    v.equal = h.n_src;
    if (h.kk < h.n_src) {
      v.cut = 1;
      v.ikrem = h.kk;
      v.ihi = 32;
    }
  }
}

struct PassShared {
  uint32_t hist[1 << kBigDigit];
  uint32_t segn[kSegs];
  uint32_t wsum[20];
  uint32_t last, found[3];
};

// Whether a digit pass of STAGE has work in state v.
template <int STAGE>
__device__ __forceinline__ bool radix_pending(const RadixVals& v) {
  return STAGE == 0 ? v.hi > 0 : (v.cut && v.ihi > 0);
}

// One radix digit pass by a grid of BS-thread blocks from the state (h, v)
// that every block holds (STAGE 0: a digit of the key; STAGE 1: a digit of
// ~index among the items whose key is kstar).  Block histograms are merged
// into ghist (zero on entry); the last block to finish (ticket) picks the
// digit holding the remaining rank, clears ghist and the ticket, and writes
// the state after the pass: the digit state, and the header too when
// `head` (nothing had written the state before this pass).
template <int DT, int STAGE, int BS>
__device__ __forceinline__ void radix_pass(const BigArgs& a, const RadixHead& h, RadixVals v, bool head, PassShared& sh) {
  const int hi = STAGE == 0 ? v.hi : v.ihi;
  const uint32_t tid = threadIdx.x;
  const int bits = hi < kBigDigit ? hi : kBigDigit;
  const int shift = hi - bits;
  const uint32_t nb = 1u << bits;
  const uint32_t hmask = hi >= 32 ? 0u : ~((1u << hi) - 1u);
  const uint32_t pre = (STAGE == 0 ? v.prefix : v.iprefix) & hmask;
  const uint32_t kstar = v.kstar;
  for (uint32_t b = tid; b < nb; b += BS) sh.hist[b] = 0;
  if (!h.from_input) load_segn(a, sh.segn); else __syncthreads();
  big_visit<DT, BS>(a, h.n_src, h.from_input, sh.segn, [&](uint32_t key, uint32_t idx) {
    uint32_t x = key;
    if (STAGE == 1) {
      if (key != kstar) return;
      x = ~idx;
    }
    if ((x & hmask) == pre) atomicAdd(&sh.hist[(x >> shift) & (nb - 1)], 1u);
  });
  __syncthreads();
  for (uint32_t b = tid; b < nb; b += BS)
    if (sh.hist[b]) atomicAdd(&a.ghist[b], sh.hist[b]);
  wait_memory();  // the histogram is handed over through atomics
  __syncthreads();
  if (tid == 0) sh.last = (atomicAdd(&a.st->big_ticket, 1u) == gridDim.x - 1) ? 1u : 0u;
  __syncthreads();
  if (!sh.last) return;
  acquire_agent();
  // The last block finds the digit holding the remaining rank.
  const uint32_t krem = STAGE == 0 ? v.krem : v.ikrem;
  const uint32_t per = (nb + BS - 1) / BS;  // bins per thread, descending
  uint32_t loc = 0;
  for (uint32_t r = tid * per; r < (tid + 1) * per && r < nb; ++r) loc += a.ghist[nb - 1 - r];
  uint32_t run = block_excl_sum<BS>(loc, sh.wsum, nullptr);
  for (uint32_t r = tid * per; r < (tid + 1) * per && r < nb; ++r) {
    const uint32_t c = a.ghist[nb - 1 - r];
    if (run < krem && krem <= run + c) {
      sh.found[0] = nb - 1 - r;
      sh.found[1] = run;
      sh.found[2] = c;
    }
    run += c;
  }
  __syncthreads();
  for (uint32_t b = tid; b < nb; b += BS) a.ghist[b] = 0;
  if (tid == 0) {
    const uint32_t d = sh.found[0], ab = sh.found[1], eq = sh.found[2];
    const uint32_t np = (pre & hmask) | (d << shift);
    if (STAGE == 0) {
      v.prefix = np;
      v.krem = krem - ab;
      v.above += ab;
      v.equal = eq;
      v.hi = shift;
      if (shift == 0) {
        v.kstar = np;
        const bool cut = v.krem < eq;
        v.cut = cut ? 1u : 0u;
        if (cut) {
          v.ikrem = v.krem;
          v.ihi = 32;
          v.iprefix = 0;
        }
      }
    } else {
      v.iprefix = np;
      v.ikrem = krem - ab;
      v.ihi = shift;
      if (shift == 0) v.istar = ~np;
    }
    if (head) radix_store_head(a.bs, h);
    radix_store(a.bs, v);
    a.st->big_ticket = 0;
  }
}

// ----------------------------------------------------------- bucket path ---
// Candidates are placed sweep by sweep: a block counts one sweep's items per
// bucket in LDS, reserves each bucket's range with one global atomic, and
// writes every item at its range base plus its rank within the block.
//
// The plan comes first, in every block: the status from the segment
// counters, then, for a filtered call, bucket offsets in descending bucket
// order from the filter's histogram of log_bin(key - tau), the bucket b*
// holding rank kk, and whether every bucket >= b* fits one sort block.  All
// blocks read the same counts and so derive the same plan; none waits for
// another.  Block 0 also records it for the kernels after this one: the
// bucket path's state, bucket list, padding and report.  When the bucket
// path does not apply, the blocks run the radix path's first key digit pass
// instead (the sort launch runs the second).  The fill counters (bcur), the
// digit histogram and its ticket are zeroed at the start of the call.
constexpr int kScatBS = 1024, kScatU = 4;

// The radix path from the scatter's blocks: its first key digit pass runs
// there, or, when no key digit is left, block 0 records the starting state.
template <int DT>
__device__ __forceinline__ void radix_start(const BigArgs& a, uint32_t status, uint32_t total, uint32_t* wsum,
                                            PassShared& ps) {
  RadixHead h;
  RadixVals v;
  radix_init<DT, kScatBS>(a, status, total, wsum, h, v);
  if (radix_pending<0>(v)) {
    radix_pass<DT, 0, kScatBS>(a, h, v, true, ps);
  } else if (blockIdx.x == 0 && threadIdx.x == 0) {
    radix_store_head(a.bs, h);
    radix_store(a.bs, v);
  }
}

template <int DT>
__global__ __launch_bounds__(kScatBS) void k_bkt_scatter(BigArgs a) {
  __shared__ uint32_t hist[kLogBins];  // counts of the sweep, then its range bases
  __shared__ uint32_t boff[kLogBins];  // first slot of each bucket (descending bucket order)
  __shared__ uint32_t segn[kSegs], s_cnt[kSegs];
  __shared__ SelectScratch fs;
  __shared__ PassShared ps;  // the radix path's first key digit pass
  BigState* s = a.bs;
  const uint32_t tid = threadIdx.x;
  const bool lead = blockIdx.x == 0;
  // thread t owns buckets [kLogBins - 4(t+1), kLogBins - 4t)
  constexpr uint32_t kOwners = kLogBins / 4;
  static_assert(kLogBins % 4 == 0 && kOwners <= kScatBS, "bucket ownership");
  const bool owner = tid < kOwners;
  const uint32_t bbase = owner ? kLogBins - 4 * (tid + 1) : 0u;
  // the segment counters and the histogram in one round trip
  uint4 hv{0u, 0u, 0u, 0u};
  if (!a.direct) {
    if (owner) hv = *reinterpret_cast<const uint4*>(a.fhist + bbase);
    if (tid < kSegs) s_cnt[tid] = a.seg_cnt[tid * kSegStride];
    if (tid == 0) fs.found[0] = 0;
  }
  __syncthreads();
  uint32_t total = 0, status = PROFK_STATUS_DIRECT;
  if (!a.direct) {
#pragma unroll
    for (int x = 0; x < kSegs; ++x) total += s_cnt[x];
    status = total < a.k_req ? PROFK_STATUS_UNDERFLOW
                             : (total > a.M ? PROFK_STATUS_OVERFLOW : PROFK_STATUS_FILTERED);
  }
  if (status != PROFK_STATUS_FILTERED) {  // uniform over the grid
    radix_start<DT>(a, status, total, fs.wsum, ps);
    return;
  }
  if (tid < kSegs) segn[tid] = min(s_cnt[tid], a.seg_cap);
  __syncthreads();
  const uint32_t n = total;
  const SegPos pos{segn, a.seg_cap};
  constexpr uint32_t per = kScatBS * kScatU;
  uint32_t key[kScatU], idx[kScatU];
  auto load_sweep = [&](uint32_t base) {
#pragma unroll
    for (int u = 0; u < kScatU; ++u) {
      const uint32_t i = base + u * kScatBS + tid;
      key[u] = 0;
      idx[u] = 0;
      if (i < n) {
        const size_t p = pos(i);
        key[u] = a.seg_key[p];
        idx[u] = a.seg_idx[p];
      }
    }
  };
  // the first sweep's candidates load while the plan is computed
  const uint32_t base0 = blockIdx.x * per;
  if (base0 < n) load_sweep(base0);
  const uint32_t kk = min(a.k, total);
  const uint32_t h[4] = {hv.x, hv.y, hv.z, hv.w};
  const uint32_t above_me = block_excl_sum<kScatBS>(h[0] + h[1] + h[2] + h[3], fs.wsum, nullptr);
  if (owner) {
    uint32_t run = above_me;
#pragma unroll
    for (int j = 3; j >= 0; --j) {
      boff[bbase + j] = run;
      if (run < kk && kk <= run + h[j]) fs.found[0] = bbase + j;
      run += h[j];
    }
  }
  __syncthreads();
  const uint32_t bstar = fs.found[0];
  uint32_t big = 0, nonempty = 0;
  if (owner) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (bbase + j >= bstar) {
        big = max(big, h[j]);
        nonempty += h[j] ? 1u : 0u;
      }
  }
  big = block_max<kScatBS>(big, fs.wsum);
  if (big > kBktCap) {  // uniform over the grid: the radix path
    radix_start<DT>(a, status, total, fs.wsum, ps);
    return;
  }
  const uint32_t tau = a.st->tau_key;
  if (lead) {
    // the non-empty buckets >= b*, in descending bucket order, with their
    // first slot and size (every candidate of such a bucket is placed)
    uint32_t nlist = 0;
    uint32_t lpos = block_excl_sum<kScatBS>(nonempty, fs.wsum, &nlist);
    if (owner) {
#pragma unroll
      for (int j = 3; j >= 0; --j)
        if (bbase + j >= bstar && h[j]) a.blist[lpos++] = uint4{bbase + j, boff[bbase + j], h[j], 0u};
    }
    if (tid == 0) {
      s->mode = kModeBucket;
      s->bstar = bstar;
      s->nlist = nlist;
      s->status = status;
      s->total = total;
      s->tau = tau;
      s->n_src = total;
      s->from_input = 0;
      s->kk = kk;
    }
    for (uint32_t p = kk + tid; p < a.k; p += kScatBS) {  // relaxed recall: padding
      if (DT == 0) static_cast<uint32_t*>(a.out_vals)[p] = 0xFF800000u;
      else static_cast<uint16_t*>(a.out_vals)[p] = 0xFF80u;
      a.out_idx[p] = -1;
    }
    if (tid == 0 && a.info) {
      a.info->count = total;
      a.info->tau_key = tau;
      a.info->status = static_cast<int32_t>(status);
      a.info->n_valid = kk;
    }
  }
  for (uint32_t base = base0; base < n; base += gridDim.x * per) {
    if (base != base0) load_sweep(base);
    for (uint32_t b = tid; b < kLogBins; b += kScatBS) hist[b] = 0;
    __syncthreads();
    uint32_t bin[kScatU], rank[kScatU];
#pragma unroll
    for (int u = 0; u < kScatU; ++u) {
      const uint32_t i = base + u * kScatBS + tid;
      bin[u] = i < n ? log_bin(key[u] - tau) : 0u;
      rank[u] = (i < n && bin[u] >= bstar) ? atomicAdd(&hist[bin[u]], 1u) : 0u;
    }
    __syncthreads();
    for (uint32_t b = tid; b < kLogBins; b += kScatBS) {
      const uint32_t c = hist[b];
      if (c) hist[b] = boff[b] + atomicAdd(&a.bcur[b * kBktPad], c);
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kScatU; ++u) {
      const uint32_t i = base + u * kScatBS + tid;
      if (i < n && bin[u] >= bstar) a.staging[hist[bin[u]] + rank[u]] = composite(key[u], idx[u]);
    }
    __syncthreads();
  }
}

// The bucket-sort blocks loop over the bucket list.  A bucket b >= 128
// holds the distances d = key - tau in [dlo(b), dlo(b) + 2^(e-7)), e =
// b/128 + 6; it is split into 256 sub-bins by the next 8 bits of d - dlo,
// counted and placed in LDS in descending sub-bin order, and each item is
// ranked within its sub-bin by comparison (a bucket b < 128 holds a single
// key, so it is one sub-bin).  A bucket whose largest sub-bin exceeds
// kSubMax is sorted whole instead (blocked bitonic sort).
constexpr int kSortBS = 256;
constexpr uint32_t kSubBins = 256, kSubMax = 64;

__device__ __forceinline__ uint32_t sub_bin(uint32_t d, uint32_t b) {
  if (b < 128u) return 0u;
  const uint32_t e = (b >> 7) + 6u;                       // d in [2^e, 2^(e+1))
  const uint32_t dlo = (128u + (b & 127u)) << (e - 7u);  // bucket start
  const uint32_t shift = e > 15u ? e - 15u : 0u;          // bucket width 2^(e-7) -> 256 sub-bins
  return (d - dlo) >> shift;
}

template <int DT>
__device__ __forceinline__ void bkt_write(const BigArgs& a, uint32_t dst, uint64_t c) {
  const uint32_t bits = bits_of_key<DT>(comp_key(c));
  if (DT == 0) static_cast<uint32_t*>(a.out_vals)[dst] = bits;
  else static_cast<uint16_t*>(a.out_vals)[dst] = static_cast<uint16_t>(bits);
  a.out_idx[dst] = comp_idx(c);
}

template <int DT>
__global__ __launch_bounds__(kSortBS) void k_bkt_sort(BigArgs a) {
  constexpr int PER = kBktCap / kSortBS;  // items per thread
  __shared__ uint64_t A[kBktCap], Bv[kBktCap];
  __shared__ uint32_t cnt[kSubBins], off[kSubBins];
  __shared__ SelectScratch scr;
  __shared__ PassShared ps;  // the radix path's second key digit pass
  const BigState* s = a.bs;
  // this block's first list entry loads with the state: it is read before
  // the list length is known (the list has kLogBins entries, so the read is
  // in bounds) and used only when it is in the list
  const uint4 e0 = blockIdx.x < kLogBins ? a.blist[blockIdx.x] : uint4{0u, 0u, 0u, 0u};
  if (s->mode != kModeBucket) {
    const RadixVals v = radix_load(s);
    if (radix_pending<0>(v)) radix_pass<DT, 0, kSortBS>(a, radix_load_head(s), v, false, ps);
    return;
  }
  const uint32_t kk = s->kk, nlist = s->nlist, tau = s->tau, t = threadIdx.x;
  for (uint32_t l = blockIdx.x; l < nlist; l += gridDim.x) {
    const uint4 e = l == blockIdx.x ? e0 : a.blist[l];
    const uint32_t b = e.x, start = e.y, m = e.z;
    if (start >= kk) continue;
    cnt[t] = 0;
    __syncthreads();
    uint32_t rk[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const uint32_t i = u * kSortBS + t;
      rk[u] = 0;
      if (i < m) {
        const uint64_t c = a.staging[start + i];
        A[i] = c;
        rk[u] = atomicAdd(&cnt[sub_bin(comp_key(c) - tau, b)], 1u);
      }
    }
    __syncthreads();
    // descending sub-bin order: thread t owns sub-bin 255 - t
    const uint32_t mine = cnt[kSubBins - 1 - t];
    const uint32_t before = block_excl_sum<kSortBS>(mine, scr.wsum, nullptr);
    off[kSubBins - 1 - t] = before;
    const uint32_t biggest = block_max<kSortBS>(mine, scr.wsum);  // (syncs: off is visible after)
    if (biggest <= kSubMax) {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const uint32_t i = u * kSortBS + t;
        if (i < m) Bv[off[sub_bin(comp_key(A[i]) - tau, b)] + rk[u]] = A[i];
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const uint32_t p = u * kSortBS + t;
        if (p < m) {
          const uint64_t c = Bv[p];
          const uint32_t sb = sub_bin(comp_key(c) - tau, b);
          const uint32_t s0 = off[sb], s1 = s0 + cnt[sb];
          const uint32_t r = count_greater(Bv, s0, s1, c);
          if (start + s0 + r < kk) bkt_write<DT>(a, start + s0 + r, c);
        }
      }
    } else {
      constexpr int E = kBktCap / kSortBS;  // 16
      uint64_t v[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t p = t * E + e;
        v[e] = p < m ? A[p] : 0ull;
      }
      __syncthreads();
      bitonic_blocked_desc<E>(v, max(static_cast<uint32_t>(E), next_pow2(m)), Bv);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t p = t * E + e;
        if (p < m && start + p < kk) bkt_write<DT>(a, start + p, v[e]);
      }
    }
    __syncthreads();  // the next bucket reuses the LDS
  }
}

// ------------------------------------------------------------ one digit ---
// One radix digit pass per launch (radix_pass), after the two that the
// scatter and the sort launches run.
template <int DT, int STAGE>
__global__ __launch_bounds__(kBigBS) void k_big_pass(BigArgs a) {
  __shared__ PassShared sh;
  const BigState* s = a.bs;
  if (s->mode == kModeBucket) return;
  const RadixVals v = radix_load(s);
  if (!radix_pending<STAGE>(v)) return;  // uniform: nothing left to resolve
  radix_pass<DT, STAGE, kBigBS>(a, radix_load_head(s), v, false, sh);
}

// -------------------------------------------------------------- collect ---
template <int DT>
__global__ __launch_bounds__(kBigBS) void k_big_collect(BigArgs a) {
  __shared__ uint64_t stage[kBigStage];
  __shared__ uint32_t segn[kSegs];
  __shared__ uint32_t s_cnt, s_base;
  const BigState* s = a.bs;
  if (s->mode == kModeBucket) return;
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1);
  const uint32_t kstar = s->kstar, istar = s->istar, cut = s->cut;
  if (tid == 0) s_cnt = 0;
  if (!s->from_input) load_segn(a, segn); else __syncthreads();
  BigState* sw = a.bs;
  big_visit<DT, kBigBS>(a, s->n_src, s->from_input, segn, [&](uint32_t key, uint32_t idx) {
    const bool take = key > kstar || (key == kstar && (!cut || idx <= istar));
    const uint64_t bal = __ballot(take);
    if (bal == 0) return;
    const uint32_t total = __popcll(bal);
    const uint32_t rank = __popcll(bal & ((1ull << lane) - 1ull));
    uint32_t base = 0;
    if (lane == __ffsll(static_cast<unsigned long long>(bal)) - 1) base = atomicAdd(&s_cnt, total);
    base = __shfl(base, __ffsll(static_cast<unsigned long long>(bal)) - 1, kWave);
    if (take) {
      const uint32_t slot = base + rank;
      const uint64_t c = composite(key, idx);
      if (slot < kBigStage) {
        stage[slot] = c;
      } else {
        // overflow of the LDS stage: one global atomic per such item (rare)
        const uint32_t g = atomicAdd(&sw->out_count, 1u);
        if (g < a.P) a.staging[g] = c;
      }
    }
  });
  __syncthreads();
  const uint32_t n_st = min(s_cnt, static_cast<uint32_t>(kBigStage));
  if (tid == 0) s_base = n_st ? atomicAdd(&sw->out_count, n_st) : 0u;
  __syncthreads();
  for (uint32_t i = tid; i < n_st; i += kBigBS) {
    const uint32_t g = s_base + i;
    if (g < a.P) a.staging[g] = stage[i];
  }
}

// ---------------------------------------------------------------- write ---
// Output i of the radix path from the i-th composite of the sorted order
// (the last sorting pass calls it): value and index for i < kk, the padding
// of a relaxed call after that, and the per-call report from output 0.
template <int DT>
__device__ __forceinline__ void big_out(const BigArgs& a, const BigState* s, uint32_t kk, uint32_t i, uint64_t c) {
  if (i >= a.k) return;
  uint32_t bits;
  int64_t id;
  if (i < kk) {
    bits = bits_of_key<DT>(comp_key(c));
    id = comp_idx(c);
  } else {
    bits = DT == 0 ? 0xFF800000u : 0xFF80u;
    id = -1;
  }
  if (DT == 0) static_cast<uint32_t*>(a.out_vals)[i] = bits;
  else static_cast<uint16_t*>(a.out_vals)[i] = static_cast<uint16_t>(bits);
  a.out_idx[i] = id;
  if (i == 0 && a.info) {
    a.info->count = s->total;
    a.info->tau_key = s->tau;
    a.info->status = static_cast<int32_t>(s->status);
    a.info->n_valid = kk;
  }
}

// ----------------------------------------------------------------- sort ---
// Sorts each tile of kBigSortTile composites descending; entries past kk are
// zero (they sort last).  One LDS buffer of the tile (128 KiB).  FINAL (a
// single tile, no merge after it): the outputs are written from the tile.
template <int DT, bool FINAL>
__global__ __launch_bounds__(1024) void k_big_tile(BigArgs a) {
  __shared__ uint64_t exch[kBigSortTile];
  const BigState* s = a.bs;
  if (s->mode == kModeBucket) return;
  const uint32_t kk = s->kk;
  const uint32_t t0 = blockIdx.x * kBigSortTile;
  constexpr int E = kBigSortTile / 1024;
  uint64_t v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t p = t0 + e * 1024 + threadIdx.x;
    v[e] = p < kk ? a.staging[p] : 0ull;
  }
  bitonic_sort_regs_desc<1024, E, true>(v, exch);
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t p = t0 + e * 1024 + threadIdx.x;
    if constexpr (FINAL) big_out<DT>(a, s, kk, p, v[e]);
    else a.runs[p] = v[e];
  }
}

// One merge-path pass: sorted runs of length L in `in` become runs of 2L in
// `out`.  Block b writes outputs [b*kBigTile, (b+1)*kBigTile), which lie in
// one pair of runs; the split points are found by a wave-parallel search
// on the runs in memory, the block's slices are staged in LDS, and each
// thread merges kBigTile/1024 outputs from its own split.  FINAL (the last
// pass, one run of P after it): the outputs are written instead of `out`.
__device__ __forceinline__ bool take_more_a(const uint64_t* A, uint32_t la, const uint64_t* B, uint32_t lb,
                                            uint32_t o, uint32_t i) {
  // With i items from A among the first o outputs, should there be more?
  const uint32_t j = o - i;
  return i < la && j > 0 && (j > lb || A[i] > B[j - 1]);
}

__device__ __forceinline__ uint32_t corank_wave(const uint64_t* A, uint32_t la, const uint64_t* B, uint32_t lb,
                                                uint32_t o) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  uint32_t lo = o > lb ? o - lb : 0u;   // smallest feasible i
  uint32_t hi = o < la ? o : la;         // largest feasible i
  // find the smallest i in [lo, hi] with take_more_a false
  while (hi > lo) {
    const uint32_t span = hi - lo;
    const uint32_t step = (span + kWave - 1) / kWave;
    const uint32_t i = lo + lane * step;
    const bool more = i < hi && take_more_a(A, la, B, lb, o, i);
    const uint64_t m = __ballot(more);
    // lanes 0..c-1 say "more": the answer is in (lo + (c-1)*step, lo + c*step]
    const uint32_t c = __popcll(m);
    if (c == 0) {
      hi = lo;
    } else {
      lo = lo + (c - 1) * step + 1;
      const uint32_t nhi = lo - 1 + step;
      hi = nhi < hi ? nhi : hi;
    }
  }
  return lo;
}

template <int DT, bool FINAL>
__global__ __launch_bounds__(1024) void k_big_merge(BigArgs a, const uint64_t* in, uint64_t* out, uint32_t L) {
  __shared__ uint64_t sa[kBigTile], sb[kBigTile];
  __shared__ uint32_t s_i[2];
  const BigState* s = a.bs;
  if (s->mode == kModeBucket) return;
  const uint32_t P = a.P;
  const uint32_t tid = threadIdx.x;
  const uint32_t o_begin = blockIdx.x * kBigTile;
  const uint32_t pair0 = (o_begin / (2 * L)) * (2 * L);
  const uint64_t* A = in + pair0;
  const uint32_t la = min(L, P - pair0);
  const uint64_t* B = A + la;
  const uint32_t lb = min(L, P - pair0 - la);
  const uint32_t o0 = o_begin - pair0;
  const uint32_t o1 = o0 + kBigTile;
  if (tid < 2 * kWave) {
    const uint32_t i = corank_wave(A, la, B, lb, tid < kWave ? o0 : o1);
    if ((tid & (kWave - 1)) == 0) s_i[tid / kWave] = i;
  }
  __syncthreads();
  const uint32_t i0 = s_i[0], i1 = s_i[1];
  const uint32_t j0 = o0 - i0, j1 = o1 - i1;
  const uint32_t na = i1 - i0, nbb = j1 - j0;
  for (uint32_t p = tid; p < na; p += 1024) sa[p] = A[i0 + p];
  for (uint32_t p = tid; p < nbb; p += 1024) sb[p] = B[j0 + p];
  __syncthreads();
  // each thread: outputs [q0, q0 + E) of this block's tile
  constexpr uint32_t E = kBigTile / 1024;
  const uint32_t q0 = tid * E;
  uint32_t lo = q0 > nbb ? q0 - nbb : 0u, hi = q0 < na ? q0 : na;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (take_more_a(sa, na, sb, nbb, q0, mid)) lo = mid + 1; else hi = mid;
  }
  uint32_t ia = lo, ib = q0 - lo;
#pragma unroll
  for (uint32_t q = 0; q < E; ++q) {
    uint64_t v;
    if (ib >= nbb || (ia < na && sa[ia] > sb[ib])) v = sa[ia++];
    else v = sb[ib++];
    if constexpr (FINAL) big_out<DT>(a, s, s->kk, o_begin + q0 + q, v);
    else out[o_begin + q0 + q] = v;
  }
}

// ------------------------------------------------------------- host -------
static inline uint32_t cdiv_u(uint64_t a, uint64_t b) { return static_cast<uint32_t>((a + b - 1) / b); }

template <int DT>
static hipError_t launch_big_t(const BigCall& c) {
  constexpr int KB = Elem<DT>::KEYBITS;
  const uint32_t P = cdiv_u(c.k, kBigSortTile) * kBigSortTile;
  BigArgs a{c.values, c.n, c.k, c.k_req, c.M, c.direct, c.seg_cnt, c.seg_key, c.seg_idx, c.blk_max,
            c.seg_cap, c.G_f, c.st, reinterpret_cast<BigState*>(c.big_state), c.ghist, c.staging, c.runs,
            c.fhist, c.bcur, reinterpret_cast<uint4*>(c.blist), P, c.out_vals, c.out_idx, c.info};
  hipLaunchKernelGGL(k_bkt_scatter<DT>, dim3(c.G_big), dim3(kScatBS), 0, c.stream, a);
  hipLaunchKernelGGL(k_bkt_sort<DT>, dim3(kBktSortBlocks), dim3(kSortBS), 0, c.stream, a);
  // key digit passes after the scatter's and the sort's (one each)
  const uint32_t key_passes = cdiv_u(KB, kBigDigit) > 2 ? cdiv_u(KB, kBigDigit) - 2 : 0u;
  for (uint32_t p = 0; p < key_passes; ++p)
    hipLaunchKernelGGL((k_big_pass<DT, 0>), dim3(c.G_big), dim3(kBigBS), 0, c.stream, a);
  for (uint32_t p = 0; p < cdiv_u(32, kBigDigit); ++p)
    hipLaunchKernelGGL((k_big_pass<DT, 1>), dim3(c.G_big), dim3(kBigBS), 0, c.stream, a);
  hipLaunchKernelGGL(k_big_collect<DT>, dim3(c.G_big), dim3(kBigBS), 0, c.stream, a);
  // tile sorts, then merge passes; the last of them writes the outputs
  const uint32_t tiles = P / kBigTile;
  if (P == kBigSortTile) {
    hipLaunchKernelGGL((k_big_tile<DT, true>), dim3(1), dim3(1024), 0, c.stream, a);
  } else {
    hipLaunchKernelGGL((k_big_tile<DT, false>), dim3(P / kBigSortTile), dim3(1024), 0, c.stream, a);
    uint64_t* src = c.runs;
    uint64_t* dst = c.staging;
    for (uint32_t L = kBigSortTile; L < P; L *= 2) {
      if (2 * L < P) hipLaunchKernelGGL((k_big_merge<DT, false>), dim3(tiles), dim3(1024), 0, c.stream, a, src, dst, L);
      else hipLaunchKernelGGL((k_big_merge<DT, true>), dim3(tiles), dim3(1024), 0, c.stream, a, src, dst, L);
      uint64_t* t = src;
      src = dst;
      dst = t;
    }
  }
  return hipGetLastError();
}

hipError_t launch_big(const BigCall& c) {
  return c.dtype == PROFK_F32 ? launch_big_t<0>(c) : launch_big_t<1>(c);
}

}  // namespace profk
