// Stage 1 of Sec. 3, the per-workgroup half of the threshold: a sample
// workgroup of BS threads holds up to 4*BS draws, 4 per thread (draw
// 4*tid + q in kv[q]), and keeps its own top-t of them.  The t-th largest
// key of the whole sample (with multiplicity) is among the union of the
// workgroups' lists, so stage 2 selects from that union only.
#pragma once

#include "device_common.h"
#include "launch.h"

namespace profk {

// Clears the per-call counters; fhist (kLogBins words, or null) is the
// refinement histogram the filter accumulates into.
// (bcur: the large-k path's bucket fill counters, one per kBktPad words, and
// ghist its radix digit histogram, kBigBins words; both null when the call
// does not take that path)
__device__ __forceinline__ void reset_state(CallState* st, uint32_t* seg_cnt, uint32_t* fhist, uint32_t* bcur,
                                            uint32_t* ghist) {
  if (threadIdx.x < kSegs) seg_cnt[threadIdx.x * kSegStride] = 0;
  if (fhist)
    for (uint32_t i = threadIdx.x; i < kLogBins; i += blockDim.x) fhist[i] = 0;
  if (bcur)
    for (uint32_t i = threadIdx.x; i < kLogBins; i += blockDim.x) bcur[i * kBktPad] = 0;
  if (ghist)
    for (uint32_t i = threadIdx.x; i < kBigBins; i += blockDim.x) ghist[i] = 0;
  if (threadIdx.x == 0) {
    st->ticket = 0;
    st->status = 0;
    st->tie_above = 0;
    st->tie_n = 0;
    st->tie_ticket = 0;
    st->big_ticket = 0;
  }
  if (threadIdx.x < 16) st->grp_ticket[threadIdx.x] = 0;
}

template <int BS>
struct SampleUnionShared {
  uint32_t keys[4 * BS];
  uint32_t lists[BS / kWave][kWaveTopMax];
  uint32_t list_n[BS / kWave];
  uint32_t bin_list[kListRankMax];  // t > kWaveTopMax: the keys of the bin holding rank t
  uint32_t kth[2];
  SelectShared sel;
  uint32_t emitted;
};

// Writes the workgroup's top-min(t, nb) draws to dst (nb: draws it holds,
// valid bit q of `valid` for kv[q]).  Every thread of the workgroup calls it.
// With t <= kWaveTopMax, *cut (when not null) receives the t-th largest
// draw if the workgroup dropped any (nb > t), else 0.
template <int BS, int KEYBITS>
__device__ __forceinline__ void sample_block_top(uint32_t (&kv)[4], uint32_t valid, uint32_t nb, uint32_t t,
                                                 uint32_t* dst, SampleUnionShared<BS>& sh,
                                                 uint32_t* cut = nullptr) {
  constexpr int NW = BS / kWave;
  static_assert(NW * kWaveTopMax % kWave == 0, "union of the wave lists");
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const uint32_t tl = min(t, nb);
  if (t <= kWaveTopMax) {
    // each wave keeps its top-tl draws, then wave 0 merges the NW lists
    uint32_t last;
    const uint32_t got = wave_top_t<4>(kv, valid, tl, sh.lists[w], last);
    if (lane == 0) sh.list_n[w] = got;
    __syncthreads();
    if (w == 0) {
      constexpr int E2 = NW * kWaveTopMax / kWave;
      uint32_t v2[E2];
      uint32_t valid2 = 0;
#pragma unroll
      for (int e = 0; e < E2; ++e) {
        // concatenated list position c = lane + 64*e
        uint32_t c = lane + kWave * e, li = 0;
        v2[e] = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i)
          if (li == static_cast<uint32_t>(i) && c >= sh.list_n[i]) { c -= sh.list_n[i]; li = i + 1; }
        if (li < NW) { v2[e] = sh.lists[li][c]; valid2 |= 1u << e; }
      }
      wave_top_t<E2>(v2, valid2, tl, dst, last);
      if (cut && lane == 0) *cut = nb > tl ? last : 0u;
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if ((valid >> q) & 1u) sh.keys[4 * tid + q] = kv[q];
  __syncthreads();
  if (tl == nb) {
    for (uint32_t j = tid; j < nb; j += BS) dst[j] = sh.keys[j];
    return;
  }
  // One digit pass over the top key bits finds the bin holding rank tl;
  // when it holds few keys they are ranked by counting, otherwise the
  // remaining digits are taken over all keys.
  constexpr int SHIFT = KEYBITS - kSelDigit;
  for (uint32_t i = tid; i < static_cast<uint32_t>(kSelBins); i += BS) sh.sel.hist[i] = 0;
  if (tid == 0) {
    sh.emitted = 0;
    sh.list_n[0] = 0;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) hist_add(sh.sel.hist, kv[q] >> SHIFT, (valid >> q) & 1u);
  __syncthreads();
  if (tid < kWave) rank_bin_search(sh.sel.hist, kSelBins, tl, sh.sel.scratch());
  __syncthreads();
  const uint32_t d = sh.sel.found[0], above = sh.sel.found[1], eq = sh.sel.found[2];
  uint32_t kth, above_kth;
  if (eq <= kListRankMax) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool take = ((valid >> q) & 1u) && (kv[q] >> SHIFT) == d;
      const uint32_t slot = lds_append(&sh.list_n[0], take);
      if (take) sh.bin_list[slot] = kv[q];
    }
    __syncthreads();
    list_kth<BS>(sh.bin_list, eq, tl - above, sh.kth);
    __syncthreads();
    kth = sh.kth[0];
    above_kth = above + sh.kth[1];
  } else {
    auto visit = [&](auto f) {
      for (uint32_t j = tid; j < nb; j += BS) f(sh.keys[j]);
    };
    const SelectResult r = block_select_kth<BS>(visit, tl - above, SHIFT, d << SHIFT, sh.sel);
    kth = r.kth;
    above_kth = above + r.above;
  }
  // the keys above the tl-th, then copies of it up to tl
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool take = ((valid >> q) & 1u) && kv[q] > kth;
    const uint32_t slot = lds_append(&sh.emitted, take);
    if (take) dst[slot] = kv[q];
  }
  for (uint32_t j = above_kth + tid; j < tl; j += BS) dst[j] = kth;
}

}  // namespace profk
