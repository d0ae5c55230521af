// Per-row Prof-K (Sec. 3: for batched inputs the procedure runs on each
// batch element).  One workgroup owns one row and runs all four stages in
// LDS:
//   1. draw S indices of the row (Philox counter word 1 = row);
//   2. tau = t-th largest sampled key;
//   3. stream the row once with 16-byte loads, appending survivors to an
//      LDS buffer of capacity M and counting all of them;
//   4. k_req <= count <= M: exact top-k of the buffer; otherwise the exact
//      top-k of the row itself (per-row fallback, no second launch).
// The LDS layout is sized from the plan at launch (dynamic shared memory).
#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"
#include "topk_block.h"

namespace profk {

constexpr int kRowDigit = 11;

struct RowArgs {
  const void* values;
  uint64_t row_stride;  // elements between row starts
  uint32_t D, k, k_req, S, t, M;
  int direct;
  uint64_t seed;
  void* out_vals;
  int64_t* out_idx;
  profk_info_t* info;
  RowLayout L;
};

template <int DT>
__global__ __launch_bounds__(kRowBS) void k_rows(RowArgs a) {
  constexpr int ES = Elem<DT>::ES, EPV = Elem<DT>::EPV, KB = Elem<DT>::KEYBITS;
  constexpr int NW = kRowBS / kWave;
  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* const samp = reinterpret_cast<uint32_t*>(smem + a.L.off_a);  // samples, then buffer keys
  uint32_t* const bkey = samp;
  uint32_t* const bidx = reinterpret_cast<uint32_t*>(smem + a.L.off_b);
  uint32_t* const hist = reinterpret_cast<uint32_t*>(smem + a.L.off_hist);
  uint64_t* const collect = reinterpret_cast<uint64_t*>(smem + a.L.off_collect);
  uint64_t* const exch = reinterpret_cast<uint64_t*>(smem + a.L.off_a);      // after the buffer is done
  __shared__ SelectScratch scr;
  __shared__ uint32_t lists[NW][kWaveTopMax];
  __shared__ uint32_t list_n[NW];
  __shared__ uint32_t s_cnt, s_tau, s_counter, s_wmax[NW];

  const uint32_t r = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const char* row = static_cast<const char*>(a.values) + static_cast<size_t>(r) * a.row_stride * ES;
  void* out_vals = static_cast<char*>(a.out_vals) + static_cast<size_t>(r) * a.k * ES;
  int64_t* out_idx = a.out_idx + static_cast<size_t>(r) * a.k;
  const uint32_t key_max = KB == 32 ? 0xFFFFFFFFu : 0xFFFFu;
  const TopkSmem sm{nullptr, 0, hist, collect, &scr, &s_counter};

  uint32_t status = PROFK_STATUS_DIRECT, count = 0, tau = 0, gmax = 0;
  if (!a.direct) {
    // 1. sample
    for (uint32_t blk = tid; 4 * blk < a.S; blk += kRowBS) {
      const U64x4 rnd = philox4x64_10(blk, r, 0, 0, a.seed, 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t j = 4 * blk + q;
        if (j < a.S) samp[j] = key_of<DT>(load_raw<DT>(row, index_of_word(rnd.w[q], a.D)));
      }
    }
    if (tid == 0) s_cnt = 0;
    __syncthreads();
    // 2. threshold
    if (a.t <= kWaveTopMax && a.S <= kRowWaveSample) {
      constexpr int E = kRowWaveSample / kRowBS;
      uint32_t sk[E];
      uint32_t valid = 0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t i = tid + kRowBS * e;
        sk[e] = i < a.S ? samp[i] : 0u;
        if (i < a.S) valid |= 1u << e;
      }
      uint32_t last = 0;
      const uint32_t got = wave_top_t<E>(sk, valid, a.t, lists[w], last);
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
        if (lane == 0) s_tau = last;
      }
    } else {
      const SelectResult sr = block_select_kth<kRowBS, kRowDigit>(
          [&](auto f) {
            for (uint32_t i = tid; i < a.S; i += kRowBS) f(samp[i]);
          },
          a.t, KB, 0u, hist, scr);
      if (tid == 0) s_tau = sr.kth;
    }
    __syncthreads();
    tau = s_tau;

    // 3. filter the row into the LDS buffer (which reuses the sample space)
    const Thresh<DT> th(tau);
    uint32_t my_max = 0;
    auto reserve = [&](uint32_t cnt) {
      const uint32_t incl = wave_incl_sum(cnt);
      const uint32_t total = __shfl(incl, kWave - 1, kWave);
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&s_cnt, total);
      return __shfl(base, 0, kWave) + incl - cnt;
    };
    auto store = [&](uint32_t slot, uint32_t key, uint32_t idx) {
      my_max = max(my_max, key);
      if (slot < a.M) {
        bkey[slot] = key;
        bidx[slot] = idx;
      }
    };
    const uintptr_t addr = reinterpret_cast<uintptr_t>(row);
    uint32_t head = static_cast<uint32_t>(((16 - (addr & 15)) & 15) / ES);
    if (head > a.D) head = a.D;
    const uint32_t nvec = (a.D - head) / EPV;
    const u32x4* vec = reinterpret_cast<const u32x4*>(row + static_cast<size_t>(head) * ES);
    for (uint32_t vb = 0; vb < nvec; vb += kRowBS * kRowU) {
      u32x4 v[kRowU];
#pragma unroll
      for (int u = 0; u < kRowU; ++u) {
        const uint32_t vi = vb + u * kRowBS + tid;
        if (vi < nvec) v[u] = __builtin_nontemporal_load(vec + vi);
        else v[u] = u32x4{th.neutral, th.neutral, th.neutral, th.neutral};
      }
      if (__ballot(tile_any<DT, kRowU>(v, th)) == 0) continue;
      const TileExact<DT, kRowU, kRowBS> tx{v, th, vb, nvec, tid, head};
      uint32_t slot = reserve(tx.count());
      tx.emit([&](uint32_t key, uint32_t idx) { store(slot++, key, idx); });
    }
    if (tid < kWave) {
      // elements before the first aligned vector and after the last one
      const uint32_t tail0 = head + nvec * EPV;
      const uint32_t ns = head + (a.D - tail0);
      uint32_t idx = 0, key = 0;
      bool ok = false;
      if (lane < ns) {
        idx = lane < head ? lane : tail0 + (lane - head);
        key = key_of<DT>(load_raw<DT>(row, idx));
        ok = key >= tau;
      }
      if (__ballot(ok)) {
        const uint32_t slot = reserve(ok ? 1u : 0u);
        if (ok) store(slot, key, idx);
      }
    }
    const uint32_t wm = wave_max_u32(my_max);
    if (lane == 0) s_wmax[w] = wm;
    __syncthreads();
    count = s_cnt;
#pragma unroll
    for (int i = 0; i < NW; ++i) gmax = max(gmax, s_wmax[i]);
    status = count < a.k_req ? PROFK_STATUS_UNDERFLOW
                             : (count > a.M ? PROFK_STATUS_OVERFLOW : PROFK_STATUS_FILTERED);
  }

  // 4. refinement, or the exact per-row fallback
  uint32_t kk = a.k;
  if (status == PROFK_STATUS_FILTERED) {
    kk = min(a.k, count);
    block_topk<kRowBS, kRowDigit>(LdsSrc{bkey, bidx}, count, kk, tau, max(gmax, tau), KB, sm);
  } else {
    block_topk<kRowBS, kRowDigit>(InputSrc<DT>{row, 0u}, a.D, a.k, 0u, key_max, KB, sm);
  }
  sort_write_any<DT, kRowBS>(collect, kk, a.k, exch, out_vals, out_idx);
  if (a.info && tid == 0) {
    profk_info_t* inf = a.info + r;
    inf->count = count;
    inf->tau_key = tau;
    inf->status = static_cast<int32_t>(status);
    inf->n_valid = kk;
  }
}

// ------------------------------------------------------------- host -------
static inline uint32_t align16(uint32_t x) { return (x + 15u) & ~15u; }

RowLayout row_layout(const profk_plan_t& p) {
  RowLayout L;
  const uint32_t S = static_cast<uint32_t>(p.S), M = static_cast<uint32_t>(p.M);
  const uint32_t k = static_cast<uint32_t>(p.k);
  uint32_t P = 1;
  while (P < (k > static_cast<uint32_t>(kRowBS) ? k : static_cast<uint32_t>(kRowBS))) P <<= 1;
  const uint32_t exch = 2u * P * 8u;
  const uint32_t b_bytes = align16(M * 4u);
  uint32_t a_bytes = align16((S > M ? S : M) * 4u);
  if (a_bytes + b_bytes < exch) a_bytes = exch - b_bytes;
  L.off_a = 0;
  L.off_b = a_bytes;
  L.off_hist = L.off_b + b_bytes;
  L.off_collect = L.off_hist + align16((1u << kRowDigit) * 4u);
  L.bytes = L.off_collect + align16(k * 8u);
  return L;
}

template <int DT>
static hipError_t launch_rows_t(const RowCall& c) {
  const profk_plan_t& p = *c.plan;
  RowArgs ra{c.values, c.row_stride, c.D, c.k, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.S),
             static_cast<uint32_t>(p.t), static_cast<uint32_t>(p.M), p.mode == PROFK_MODE_DIRECT ? 1 : 0,
             c.seed, c.out_vals, c.out_idx, c.info, c.L};
  hipLaunchKernelGGL(k_rows<DT>, dim3(c.B), dim3(kRowBS), c.L.bytes, c.stream, ra);
  return hipGetLastError();
}

hipError_t launch_rows(const RowCall& c) {
  (void)hipGetLastError();  // report only errors of this call's launches
  return c.dtype == PROFK_F32 ? launch_rows_t<0>(c) : launch_rows_t<1>(c);
}

}  // namespace profk
