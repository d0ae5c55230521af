// The filter-and-compact pass of Prof-K (Sec. 3, stage 3): every element is
// compared with the threshold tau and the survivors are compacted into a
// bounded candidate buffer, counting all of them.
//
// k_filter: a persistent grid streaming the input with 16-byte nontemporal
// loads; tiles of the input are dealt to the workgroups in turn, so that the
// survivors of a sorted or clustered input spread over every workgroup.  When the sample union
// is small every workgroup first selects tau from it itself.  Survivors are
// staged in LDS and appended to one of eight candidate segments with one
// atomic per workgroup, because same-address global atomics serialise across
// the chip.
#include <climits>

#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"

namespace profk {

static inline uint32_t cdiv(uint64_t a, uint64_t b) { return static_cast<uint32_t>((a + b - 1) / b); }
template <class T> static T* at(uint8_t* ws, size_t off) { return reinterpret_cast<T*>(ws + off); }

// ------------------------------------------------------------ stage 3 -----
struct FilterArgs {
  const void* values;
  uint32_t n, head, nvec;
  uint32_t seg_cap;
  CallState* st;
  const uint32_t* union_keys;  // sample union to select tau from, or null: tau in st
  uint32_t union_n, t;
  uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  uint32_t* fhist;             // refinement histogram (or null), zero on entry
};

// The filter pass; the survival test is in filter_tile.h.
// U: 16-byte loads per lane and step.  DB: the next step's loads are issued
// before the current step is tested, which pays where most steps take the
// survivor path and costs a little on the sparse stream of a large input.
template <int DT, bool LEX, int U, bool DB>
__global__ __launch_bounds__(kFiltBS) void k_filter(FilterArgs a) {
  constexpr int EPV = Elem<DT>::EPV;
  constexpr int ES = Elem<DT>::ES;
  __shared__ uint32_t s_skey[kStage], s_sidx[kStage];
  // the waves' top-t lists while tau is chosen, then the block's log-bin
  // histogram of its survivors
  __shared__ __align__(16) uint32_t s_pool[kLogBins];
  static_assert(kFiltBS / kWave * kWaveTopMax <= kLogBins, "tau lists");
  uint32_t* const s_lists = s_pool;
  __shared__ uint32_t s_found[kFiltBS / kWave];
  __shared__ uint32_t s_cnt, s_tau, s_base;
  __shared__ uint32_t s_wmax[kFiltBS / kWave];
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), b = blockIdx.x;
  const uint32_t seg = b & (kSegs - 1);
  if (tid == 0) s_cnt = 0;

  // The sample union (when this block selects tau) is loaded first and the
  // block's first step after it: a wave's loads return in order, so the
  // union arrives at once and tau is chosen while the step is in flight.
  const u32x4* vec = reinterpret_cast<const u32x4*>(static_cast<const char*>(a.values) +
                                                    static_cast<size_t>(a.head) * ES);
  // step s of block b reads tile s * gridDim.x + b (kFiltBS * U vectors);
  // nvec + the stride stays below 2^32 for every input the C ABI accepts
  constexpr uint32_t kTile = kFiltBS * U;
  const uint32_t vbeg = b * kTile;
  const uint32_t vend = a.nvec;
  const uint32_t vstride = gridDim.x * kTile;
  constexpr int E = kFiltTauMax / kFiltBS;
  const bool one_wave = a.union_n <= kWave * kFiltTauWave;
  uint32_t uk[E];
  uint32_t valid = 0;
  if (a.union_n) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      // one wave: lane + 64 e for e < kFiltTauWave; four waves: tid + 256 e
      const uint32_t i = one_wave ? lane + kWave * e : tid + kFiltBS * e;
      const bool in = (one_wave ? (tid < kWave && e < static_cast<int>(kFiltTauWave)) : true) && i < a.union_n;
      uk[e] = in ? a.union_keys[i] : 0u;
      if (in) valid |= 1u << e;
    }
  }
  u32x4 v[U];
  auto load_step = [&](uint32_t vb, uint32_t fill) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t vi = vb + u * kFiltBS + tid;
      if (vi < vend) v[u] = __builtin_nontemporal_load(vec + vi);
      else v[u] = u32x4{fill, fill, fill, fill};
    }
  };
  // 0xFFFFFFFF is the lowest key: it fails the fast test unless every key
  // passes, and the exact test skips slots past the end anyway.
  load_step(vbeg, 0xFFFFFFFFu);

  // ---- threshold (stage 2) when the sample union is small (t <= 32)
  uint32_t tau;
  if (a.union_n) {
    uint32_t last = 0;
    if (one_wave) {
      // one wave holds the whole union in registers
      if (tid < kWave) {
        wave_top_t<E>(uk, valid, a.t, nullptr, last);
        if (lane == 0) s_tau = last;
      }
    } else {
      // every wave keeps the top t of its share, wave 0 merges the lists
      constexpr int NW = kFiltBS / kWave;
      const uint32_t w = tid / kWave;
      const uint32_t got = wave_top_t<E>(uk, valid, a.t, s_lists + w * kWaveTopMax, last);
      if (lane == 0) s_found[w] = got;
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
            if (li == static_cast<uint32_t>(i) && c >= s_found[i]) { c -= s_found[i]; li = i + 1; }
          if (li < NW) { v2[e] = s_lists[li * kWaveTopMax + c]; valid2 |= 1u << e; }
        }
        wave_top_t<E2>(v2, valid2, a.t, nullptr, last);
        if (lane == 0) s_tau = last;
      }
    }
    __syncthreads();
    tau = s_tau;
    if (b == 0 && tid == 0) a.st->tau_key = tau;
  } else {
    tau = a.st->tau_key;
  }

  const Thresh<DT> th(tau, LEX ? a.st->tau_idx : 0xFFFFFFFFu);
  uint32_t* const s_hist = s_pool;
  if (a.fhist)
    for (uint32_t i = tid; i < kLogBins; i += kFiltBS) s_hist[i] = 0;
  __syncthreads();

  uint32_t* const seg_counter = a.seg_cnt + seg * kSegStride;
  uint32_t* const seg_key = a.seg_key + static_cast<size_t>(seg) * a.seg_cap;
  uint32_t* const seg_idx = a.seg_idx + static_cast<size_t>(seg) * a.seg_cap;
  uint32_t my_max = 0;
  // Reserve consecutive staging slots for one wave; slots past the LDS
  // stage go straight to the block's segment.
  auto reserve = [&](uint32_t cnt, uint32_t& slot, uint32_t& first_over, uint32_t& gbase) {
    const uint32_t incl = wave_incl_sum(cnt);
    const uint32_t total = __builtin_amdgcn_readlane(incl, kWave - 1);  // (scalar reads, no lane permute)
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(&s_cnt, total);
    base = __builtin_amdgcn_readlane(base, 0);
    const uint32_t n_in = base < kStage ? min(total, kStage - base) : 0u;
    const uint32_t n_over = total - n_in;
    gbase = 0;
    if (n_over) {
      if (lane == 0) gbase = atomicAdd(seg_counter, n_over);
      gbase = __builtin_amdgcn_readlane(gbase, 0);
    }
    first_over = base + n_in;
    slot = base + incl - cnt;
  };
  auto store = [&](uint32_t slot, uint32_t first_over, uint32_t gbase, uint32_t key, uint32_t idx) {
    my_max = max(my_max, key);
    if (a.fhist) atomicAdd(&s_hist[log_bin(key - tau)], 1u);
    if (slot < kStage) {
      s_skey[slot] = key;
      s_sidx[slot] = idx;
    } else {
      const uint32_t gp = gbase + (slot - first_over);
      if (gp < a.seg_cap) {
        seg_key[gp] = key;
        seg_idx[gp] = idx;
      }
    }
  };

  for (uint32_t vb = vbeg; vb < vend; vb += vstride) {
    u32x4 cur[U];
    if constexpr (DB) {
#pragma unroll
      for (int u = 0; u < U; ++u) cur[u] = v[u];
      load_step(vb + vstride, th.neutral);
    } else {
      if (vb != vbeg) load_step(vb, th.neutral);
#pragma unroll
      for (int u = 0; u < U; ++u) cur[u] = v[u];
    }
    if (__ballot(tile_any<DT, U>(cur, th)) == 0) continue;
    // Rare path: per-vector survivor masks, one slot reservation per wave,
    // then a short loop over each lane's set bits.
    const TileSparse<DT, U, kFiltBS, LEX> ts(cur, th, vb, vend, tid, a.head);
    uint32_t slot, first_over, gbase;
    reserve(ts.count(), slot, first_over, gbase);
    ts.emit(cur, [&](uint32_t key, uint32_t idx) { store(slot++, first_over, gbase, key, idx); });
  }

  // Elements before the first aligned vector and after the last one.
  if (b == gridDim.x - 1 && tid < kWave) {
    const uint32_t tail0 = a.head + a.nvec * EPV;
    const uint32_t ns = a.head + (a.n - tail0);
    uint32_t idx = 0, key = 0;
    bool ok = false;
    if (lane < ns) {
      idx = lane < a.head ? lane : tail0 + (lane - a.head);
      key = key_of<DT>(load_raw<DT>(a.values, idx));
      ok = LEX ? (key > tau || (key == tau && idx <= th.tie)) : key >= tau;
    }
    (void)EPV;
    if (__ballot(ok)) {
      uint32_t slot, first_over, gbase;
      reserve(ok ? 1u : 0u, slot, first_over, gbase);
      if (ok) store(slot, first_over, gbase, key, idx);
    }
  }

  // Append the staged survivors to the segment: one atomic per block.
  const uint32_t wm = wave_max_u32(my_max);
  if (lane == 0) s_wmax[tid / kWave] = wm;
  __syncthreads();
  const uint32_t n_st = min(s_cnt, kStage);
  if (tid == 0) {
    s_base = n_st ? atomicAdd(seg_counter, n_st) : 0u;
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < kFiltBS / kWave; ++i) m = max(m, s_wmax[i]);
    a.blk_max[b] = m;
  }
  __syncthreads();
  const uint32_t base = s_base;
  for (uint32_t i = tid; i < n_st; i += kFiltBS) {
    const uint32_t gp = base + i;
    if (gp < a.seg_cap) {
      seg_key[gp] = s_skey[i];
      seg_idx[gp] = s_sidx[i];
    }
  }
  // Add the block's non-empty bins to the refinement histogram.
  if (a.fhist && n_st) {
    for (uint32_t i = tid; i < kLogBins; i += kFiltBS) {
      const uint32_t c = s_hist[i];
      if (c) atomicAdd(&a.fhist[i], c);
    }
  }
}

// Filter workgroups one CU holds at once, capped at `want` (the persistent
// grid is sized to what is resident, so no workgroup starts after the
// others have finished).
int filter_blocks_per_cu(int dtype, int want) {
  static int cached[2] = {0, 0};
  const int d = dtype == PROFK_F32 ? 0 : 1;
  if (cached[d] == 0) {
    int n = 0;
    const hipError_t e = d == 0
        ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_filter<0, false, kFiltUSmall, true>, kFiltBS, 0)
        : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_filter<1, false, kFiltUSmall, true>, kFiltBS, 0);
    cached[d] = (e == hipSuccess && n > 0) ? n : kFiltPerCuDense;
  }
  return cached[d] < want ? cached[d] : want;
}

// union_keys null: the filter reads tau from the call state.
template <int DT>
static hipError_t launch_filter_t(const FlatCall& c, CallState* st, const uint32_t* union_keys, bool lex) {
  const FlatLayout& L = c.L;
  constexpr int ES = Elem<DT>::ES, EPV = Elem<DT>::EPV;
  const uintptr_t addr = reinterpret_cast<uintptr_t>(c.values);
  uint32_t head = static_cast<uint32_t>(((16 - (addr & 15)) & 15) / ES);
  if (head > c.n) head = c.n;
  const uint32_t nvec = (c.n - head) / EPV;
  FilterArgs fa{c.values, c.n, head, nvec, L.seg_cap, st,
                union_keys, union_keys ? L.union_n : 0u, static_cast<uint32_t>(c.plan->t),
                at<uint32_t>(c.ws, L.off_segcnt), at<uint32_t>(c.ws, L.off_seg_key),
                at<uint32_t>(c.ws, L.off_seg_idx), at<uint32_t>(c.ws, L.off_blk_max),
                at<uint32_t>(c.ws, L.off_fhist)};
  if (c.ev_before) (void)hipEventRecord(c.ev_before, c.stream);
  // small inputs are never sparse: their steps are always double-buffered
  const bool large = L.filt_u == kFiltULarge, db = L.filt_db;
  const dim3 G(L.G_f), BS(kFiltBS);
  if (lex) {
    if (!large) hipLaunchKernelGGL((k_filter<DT, true, kFiltUSmall, true>), G, BS, 0, c.stream, fa);
    else if (db) hipLaunchKernelGGL((k_filter<DT, true, kFiltULarge, true>), G, BS, 0, c.stream, fa);
    else hipLaunchKernelGGL((k_filter<DT, true, kFiltULarge, false>), G, BS, 0, c.stream, fa);
  } else {
    if (!large) hipLaunchKernelGGL((k_filter<DT, false, kFiltUSmall, true>), G, BS, 0, c.stream, fa);
    else if (db) hipLaunchKernelGGL((k_filter<DT, false, kFiltULarge, true>), G, BS, 0, c.stream, fa);
    else hipLaunchKernelGGL((k_filter<DT, false, kFiltULarge, false>), G, BS, 0, c.stream, fa);
  }
  if (c.ev_after) (void)hipEventRecord(c.ev_after, c.stream);
  return hipGetLastError();
}

hipError_t launch_filter(const FlatCall& c, CallState* st, const uint32_t* union_keys, bool lex) {
  return c.dtype == PROFK_F32 ? launch_filter_t<0>(c, st, union_keys, lex) : launch_filter_t<1>(c, st, union_keys, lex);
}

}  // namespace profk
