// Per-row Prof-K (Sec. 3: for batched inputs the procedure runs on each
// batch element).  One workgroup owns one row and runs all four stages in
// LDS:
//   1. draw S indices of the row (Philox counter word 1 = row);
//   2. tau = t-th largest sampled key (radix select in LDS); lexicographic
//      plans also find the index of the threshold pair;
//   3. stream the row once with 16-byte loads, appending survivors to an
//      LDS buffer of capacity M and counting all of them; a buffer that
//      holds them all is then histogrammed by log_bin(key - tau);
//   4. k_req <= count <= M: the survivors at or above the bucket of rank k
//      are ranked within their buckets and written directly (the radix
//      refinement when those buckets are large); otherwise the exact top-k
//      of the row itself (per-row fallback, no second launch).
// The LDS layout is sized from the plan at launch (dynamic shared memory).
#include <type_traits>

#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"
#include "row_common.h"
#include "topk_block.h"

namespace profk {

// tau from the sample held in registers (at most 8 keys per thread): each
// wave's top-t, then the top-t of their union.
__host__ __device__ constexpr bool row_fast_tau(uint32_t S, uint32_t t) {
  return S <= 8u * kRowBS && t >= 1 && t <= kWaveTopMax;
}

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

template <int DT, bool LEX>
__global__ __launch_bounds__(kRowBS) void k_rows(RowArgs a) {
  constexpr int ES = Elem<DT>::ES, EPV = Elem<DT>::EPV, KB = Elem<DT>::KEYBITS;
  constexpr int kSelDigitRow = KB == 16 ? 8 : 11;  // sample select: 2 or 3 passes
  constexpr int kDigit = row_digit<DT>();
  using K = RowKey<DT>;
  constexpr int NW = kRowBS / kWave;
  constexpr uint32_t NB = row_log_bins<DT>();
  constexpr uint32_t RB = NB / kRowBS;              // log bins owned per thread
  static_assert(NB % kRowBS == 0, "log-bin ownership");
  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* const samp = reinterpret_cast<uint32_t*>(smem + a.L.off_a);  // samples, then buffer keys
  K* const bkey = reinterpret_cast<K*>(smem + a.L.off_a);
  uint32_t* const bidx = reinterpret_cast<uint32_t*>(smem + a.L.off_b);
  uint32_t* const hist = reinterpret_cast<uint32_t*>(smem + a.L.off_hist);
  uint64_t* const collect = reinterpret_cast<uint64_t*>(smem + a.L.off_collect);
  uint64_t* const comp = reinterpret_cast<uint64_t*>(smem + a.L.off_comp);
  uint64_t* const exch = reinterpret_cast<uint64_t*>(smem + a.L.off_a);      // after the buffer is done
  __shared__ SelectScratch scr;
  __shared__ uint32_t s_cnt, s_counter, s_tau, s_tie_n, s_wmax[NW];

  const uint32_t r = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const char* row = static_cast<const char*>(a.values) + static_cast<size_t>(r) * a.row_stride * ES;
  void* out_vals = static_cast<char*>(a.out_vals) + static_cast<size_t>(r) * a.k * ES;
  int64_t* out_idx = a.out_idx + static_cast<size_t>(r) * a.k;
  const uint32_t key_max = KB == 32 ? 0xFFFFFFFFu : 0xFFFFu;
  const TopkSmem sm{nullptr, 0, hist, collect, &scr, &s_counter};

  uint32_t status = PROFK_STATUS_DIRECT, count = 0, tau = 0, gmax = 0;
  if (!a.direct) {
    // 1. sample: the Philox words first, then all gathers in flight at once
    const bool fast = row_fast_tau(a.S, a.t);
    uint32_t keys[8], ids[8];
    uint32_t valid = 0;
    for (uint32_t blk0 = 0; 4 * blk0 < a.S; blk0 += 2 * kRowBS) {
      U64x4 rnd[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const uint32_t blk = blk0 + q * kRowBS + tid;
        if (4 * blk < a.S) rnd[q] = philox4x64_10(blk, r, 0, 0, a.seed, 0);
      }
      uint32_t raw[8];
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t j = 4 * (blk0 + q * kRowBS + tid) + x;
          ids[4 * q + x] = j < a.S ? index_of_word(rnd[q].w[x], a.D) : 0u;
          raw[4 * q + x] = j < a.S ? load_raw<DT>(row, ids[4 * q + x]) : 0u;
        }
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const uint32_t j = 4 * (blk0 + q * kRowBS + tid) + x;
          keys[4 * q + x] = key_of<DT>(raw[4 * q + x]);
          if (j < a.S) {
            valid |= 1u << (4 * q + x);
            if (!fast) samp[j] = keys[4 * q + x];
          }
        }
    }
    if (tid == 0) s_cnt = 0;
    // 2. threshold
    if (fast) {
      // every wave's top-t (hist serves as scratch: NW lists of up to
      // kWaveTopMax keys, then their lengths), then the top-t of the union
      uint32_t last = 0;
      const uint32_t got = wave_top_t<8>(keys, valid, a.t, hist + w * kWaveTopMax, last);
      if (lane == 0) hist[NW * kWaveTopMax + w] = got;
      __syncthreads();
      if (w == 0) {
        static_assert(NW * kWaveTopMax == 2 * kWave, "union of the wave lists: two keys per lane");
        uint32_t u[2];
        uint32_t uv = 0;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const uint32_t s = lane + q * kWave, ww = s / kWaveTopMax;
          u[q] = hist[s];
          if (s % kWaveTopMax < hist[NW * kWaveTopMax + ww]) uv |= 1u << q;
        }
        wave_top_t<2>(u, uv, a.t, nullptr, last);
        if (lane == 0) s_tau = last;
      }
      __syncthreads();
      tau = s_tau;
    } else {
      __syncthreads();
      tau = block_select_kth<kRowBS, kSelDigitRow>(
                [&](auto f) {
                  for (uint32_t i = tid; i < a.S; i += kRowBS) f(samp[i]);
                },
                a.t, KB, 0u, hist, scr)
                .kth;
    }
    uint32_t tie = 0xFFFFFFFFu;
    if (LEX && fast) {
      // the draws are still in registers
      auto draws = [&](auto f) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((valid >> e) & 1u) f(keys[e], ids[e]);
      };
      tie = tau_pair_index<kRowBS, kDigit>(draws, tau, a.t, reinterpret_cast<uint32_t*>(smem + a.L.off_a),
                                           a.L.off_b / 4u, hist, scr, &s_tie_n);
    } else if (LEX) {
      // the draws again (Philox words and gathers), for the tied draws' indices
      auto draws = [&](auto f) {
        for (uint32_t jb = tid; 4 * jb < a.S; jb += kRowBS) {
          const U64x4 rr = philox4x64_10(jb, r, 0, 0, a.seed, 0);
          uint32_t raw[4], ix[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const bool in = 4 * jb + q < a.S;
            ix[q] = in ? index_of_word(rr.w[q], a.D) : 0u;
            raw[q] = in ? load_raw<DT>(row, ix[q]) : 0u;
          }
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (4 * jb + q < a.S) f(key_of<DT>(raw[q]), ix[q]);
        }
      };
      tie = tau_pair_index<kRowBS, kDigit>(draws, tau, a.t, reinterpret_cast<uint32_t*>(smem + a.L.off_a),
                                           a.L.off_b / 4u, hist, scr, &s_tie_n);
    }
    for (uint32_t i = tid; i < NB; i += kRowBS) hist[i] = 0;
    __syncthreads();

    // 3. filter the row into the LDS buffer (which reuses the sample space)
    const Thresh<DT> th(tau, tie);
    uint32_t my_max = 0;
    auto reserve = [&](uint32_t cnt) {
      const uint32_t incl = wave_incl_sum(cnt);
      const uint32_t total = __builtin_amdgcn_readlane(incl, kWave - 1);
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&s_cnt, total);
      return __builtin_amdgcn_readlane(base, 0) + incl - cnt;
    };
    auto store = [&](uint32_t slot, uint32_t key, uint32_t idx) {
      my_max = max(my_max, key);
      if (slot < a.M) {
        bkey[slot] = static_cast<K>(key);
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
      const TileSparse<DT, kRowU, kRowBS, LEX> tx(v, th, vb, nvec, tid, head);
      if (__ballot(tx.any()) == 0) continue;
      uint32_t slot = reserve(tx.count());
      tx.emit(v, [&](uint32_t key, uint32_t idx) { store(slot++, key, idx); });
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
        ok = LEX ? (key > tau || (key == tau && idx <= tie)) : key >= tau;
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
    if (status == PROFK_STATUS_FILTERED) {
      // bucket histogram of the buffer (after the pass, so that the
      // streaming loop does no per-survivor histogram atomics)
      for (uint32_t i = tid; i < count; i += kRowBS) atomicAdd(&hist[log_bin(bkey[i] - tau)], 1u);
      __syncthreads();
    }
  }

  // 4. refinement, or the exact per-row fallback
  uint32_t kk = a.k;
  bool done = false;
  if (status == PROFK_STATUS_FILTERED) {
    kk = min(a.k, count);
    // Bucket offsets in descending bucket order, in place: thread t owns
    // buckets [NB - RB(t+1), NB - RB t).
    const uint32_t bb = NB - RB * (tid + 1);
    uint32_t h[RB];
    uint32_t s = 0;
#pragma unroll
    for (uint32_t j = 0; j < RB; ++j) {
      h[j] = hist[bb + j];
      s += h[j];
    }
    uint32_t run = block_excl_sum<kRowBS>(s, scr.wsum, nullptr);
#pragma unroll
    for (int j = static_cast<int>(RB) - 1; j >= 0; --j) {
      hist[bb + j] = run;
      if (run < kk && kk <= run + h[j]) {
        scr.found[0] = bb + j;
        scr.found[1] = run;
        scr.found[2] = h[j];
      }
      run += h[j];
    }
    __syncthreads();
    const uint32_t bstar = scr.found[0], n_sel = scr.found[1] + scr.found[2];
    uint32_t big = 0;
#pragma unroll
    for (uint32_t j = 0; j < RB; ++j)
      if (bb + j >= bstar) big = max(big, h[j]);
    big = block_max<kRowBS>(big, scr.wsum);
    if (n_sel <= a.k + kFastBucket && big <= kFastBucket) {
      // place the buckets >= b*: afterwards hist[b] is the end of bucket b
      // and hist[b + 1] its start
      for (uint32_t i = tid; i < count; i += kRowBS) {
        const uint32_t key = bkey[i];
        const uint32_t bin = log_bin(key - tau);
        if (bin >= bstar) comp[atomicAdd(&hist[bin], 1u)] = composite(key, bidx[i]);
      }
      __syncthreads();
      for (uint32_t p = tid; p < n_sel; p += kRowBS) {
        const uint64_t c = comp[p];
        const uint32_t bin = log_bin(comp_key(c) - tau);
        const uint32_t s0 = bin + 1 < NB ? hist[bin + 1] : 0u, s1 = hist[bin];
        uint32_t rank = 0;
        for (uint32_t q = s0; q < s1; ++q) rank += comp[q] > c ? 1u : 0u;
        const uint32_t dst = s0 + rank;
        if (dst < kk) {
          const uint32_t bits = bits_of_key<DT>(comp_key(c));
          if (DT == 0) static_cast<uint32_t*>(out_vals)[dst] = bits;
          else static_cast<uint16_t*>(out_vals)[dst] = static_cast<uint16_t>(bits);
          out_idx[dst] = comp_idx(c);
        }
      }
      for (uint32_t p = kk + tid; p < a.k; p += kRowBS) {  // relaxed recall: padding
        if (DT == 0) static_cast<uint32_t*>(out_vals)[p] = 0xFF800000u;
        else static_cast<uint16_t*>(out_vals)[p] = 0xFF80u;
        out_idx[p] = -1;
      }
      done = true;
    } else {
      block_topk<kRowBS, kDigit>(LdsSrc<K>{bkey, bidx}, count, kk, tau, max(gmax, tau), KB, sm);
    }
  } else {
    block_topk<kRowBS, kDigit>(InputSrc<DT>{row, 0u}, a.D, a.k, 0u, key_max, KB, sm);
  }
  if (!done) sort_write_any<DT, kRowBS>(collect, kk, a.k, exch, out_vals, out_idx);
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

RowLayout row_layout(const profk_plan_t& p, int dtype) {
  RowLayout L;
  const uint32_t S = static_cast<uint32_t>(p.S), M = static_cast<uint32_t>(p.M);
  const uint32_t k = static_cast<uint32_t>(p.k), t = static_cast<uint32_t>(p.t);
  const bool f32 = dtype == PROFK_F32;
  uint32_t P = 1;
  while (P < (k > static_cast<uint32_t>(kRowBS) ? k : static_cast<uint32_t>(kRowBS))) P <<= 1;
  const uint32_t exch = 2u * P * 8u;
  const uint32_t b_bytes = align16(M * 4u);
  const uint32_t samp_bytes = row_fast_tau(S, t) ? 0u : S * 4u;   // samples kept in LDS
  const uint32_t key_bytes = M * (f32 ? 4u : 2u);
  uint32_t a_bytes = align16(samp_bytes > key_bytes ? samp_bytes : key_bytes);
  if (a_bytes + b_bytes < exch) a_bytes = exch - b_bytes;
  const uint32_t nb = f32 ? row_log_bins<0>() : row_log_bins<1>();
  const uint32_t radix = 1u << (f32 ? row_digit<0>() : row_digit<1>());
  uint32_t hist_words = radix > nb ? radix : nb;
  if (hist_words < static_cast<uint32_t>(kRowBS / kWave) * (kWaveTopMax + 1))
    hist_words = static_cast<uint32_t>(kRowBS / kWave) * (kWaveTopMax + 1);
  L.off_a = 0;
  L.off_b = a_bytes;
  L.off_hist = L.off_b + b_bytes;
  L.off_collect = L.off_hist + align16(hist_words * 4u);
  L.off_comp = L.off_collect + align16(k * 8u);
  L.bytes = L.off_comp + align16((k + kFastBucket) * 8u);
  return L;
}

template <int DT>
static hipError_t launch_rows_t(const RowCall& c) {
  const profk_plan_t& p = *c.plan;
  RowArgs ra{c.values, c.row_stride, c.D, c.k, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.S),
             static_cast<uint32_t>(p.t), static_cast<uint32_t>(p.M), p.mode == PROFK_MODE_DIRECT ? 1 : 0,
             c.seed, c.out_vals, c.out_idx, c.info, c.L};
  if (p.lexicographic) hipLaunchKernelGGL((k_rows<DT, true>), dim3(c.B), dim3(kRowBS), c.L.bytes, c.stream, ra);
  else hipLaunchKernelGGL((k_rows<DT, false>), dim3(c.B), dim3(kRowBS), c.L.bytes, c.stream, ra);
  return hipGetLastError();
}

hipError_t launch_rows(const RowCall& c) {
  (void)hipGetLastError();  // report only errors of this call's launches
  return c.dtype == PROFK_F32 ? launch_rows_t<0>(c) : launch_rows_t<1>(c);
}

}  // namespace profk
