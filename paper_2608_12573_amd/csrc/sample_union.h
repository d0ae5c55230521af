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
__device__ __forceinline__ void reset_state(CallState* st, uint32_t* seg_cnt, uint32_t* fhist) {
  if (threadIdx.x < kSegs) seg_cnt[threadIdx.x * kSegStride] = 0;
  if (fhist)
    for (uint32_t i = threadIdx.x; i < kLogBins; i += blockDim.x) fhist[i] = 0;
  if (threadIdx.x == 0) {
    st->ticket = 0;
    st->status = 0;
    st->tie_above = 0;
    st->tie_n = 0;
    st->tie_ticket = 0;
  }
  if (threadIdx.x < 16) st->grp_ticket[threadIdx.x] = 0;
}

template <int BS>
struct SampleUnionShared {
  uint32_t keys[4 * BS];
  uint32_t lists[BS / kWave][kWaveTopMax];
  uint32_t list_n[BS / kWave];
  SelectShared sel;
  uint32_t emitted;
};

// Writes the workgroup's top-min(t, nb) draws to dst (nb: draws it holds,
// valid bit q of `valid` for kv[q]).  Every thread of the workgroup calls it.
template <int BS, int KEYBITS>
__device__ __forceinline__ void sample_block_top(uint32_t (&kv)[4], uint32_t valid, uint32_t nb, uint32_t t,
                                                 uint32_t* dst, SampleUnionShared<BS>& sh) {
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
  auto visit = [&](auto f) {
    for (uint32_t j = tid; j < nb; j += BS) f(sh.keys[j]);
  };
  const SelectResult r = block_select_kth<BS>(visit, tl, KEYBITS, 0u, sh.sel);
  if (tid == 0) sh.emitted = 0;
  __syncthreads();
  for (uint32_t j = tid; j < nb; j += BS)
    if (sh.keys[j] > r.kth) dst[atomicAdd(&sh.emitted, 1u)] = sh.keys[j];
  for (uint32_t j = r.above + tid; j < tl; j += BS) dst[j] = r.kth;
}

}  // namespace profk
