// The BatchTopK SAE layer with Prof-K in the encoder's epilogue (Sec. 5,
// "Application: BatchTopK Sparse Autoencoders": the K = B*k largest of the
// B x d_dict post-ReLU latents, flattened).
//
//   z[b, j] = relu(sum_m x[b, m] W_enc[j, m] + b_enc[j])     (bf16 inputs,
//                                                             fp32 sums)
//
// The latent matrix is never written to HBM:
//   k_sae_sample   stage 1: the S sampled latents, each computed with the same
//                  MFMA sequence as the GEMM (so its value is the GEMM's, bit
//                  for bit), and each sample workgroup's top-t of them;
//   k_select_tau   stage 2 (shared with the vector path);
//   k_sae_thresholds  each column's accumulator threshold for tau;
//   k_sae_filter   the GEMM with stage 3 in its epilogue: survivors are
//                  compacted exactly as the vector filter does it, so the
//                  vector path's refinement (stage 4) runs unchanged;
//   k_sae_dense    the GEMM with a dense epilogue: for the exact fallback only
//                  (it returns at once when the filter's count is in range),
//                  and as an inspection entry point.
// Sparse decode (k_dec_*): x_hat[b, :] = sum over b's selected latents of
// z W_dec[j, :] + b_dec, grouped by row and summed in ascending j, so the
// result does not depend on the order the selection lists them in.
//
// One 32x32x16 MFMA step rounds once: the accumulator and its 16 products
// are summed together before rounding to fp32.
#include "device_common.h"
#include "launch.h"
#include "sample_union.h"

namespace profk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

// GEMM tiling: a workgroup of 8 waves computes a 256 x 128 tile of z (waves
// in a 4 x 2 grid, 64 x 64 each as 2 x 2 32x32 MFMA accumulators); d_model
// is consumed in chunks of 64, double-buffered in LDS (rows padded to 144 B)
// with one barrier per chunk: the next chunk's global loads are in flight,
// and then written to the other buffer, while this chunk's MFMAs run.
constexpr int kSaeBS = 512;
constexpr uint32_t kSaeBM = 256, kSaeBN = 128, kSaeBK = 64;
constexpr uint32_t kSaeLd = kSaeBK + 8;  // LDS row stride in bf16 elements
constexpr uint32_t kSaeMaxBlocks = 1024;
constexpr int kSaeApieces = kSaeBM * kSaeBK / 8 / kSaeBS;  // 16-byte pieces per thread and chunk
constexpr int kSaeBpieces = kSaeBN * kSaeBK / 8 / kSaeBS;
static_assert(kSaeBS / kWave == (kSaeBM / 64) * (kSaeBN / 64), "one wave per 64 x 64 block");

struct SaeGemm {
  const uint16_t* x;  // [B, d_model] bf16 bits, 16-byte aligned rows
  const uint16_t* w;  // [d_dict, d_model]
  const float* bias;  // [d_dict]
  uint32_t B, d_model, d_dict;
};

struct alignas(16) SaeTileLds {
  uint16_t a[2][kSaeBM * kSaeLd];
  uint16_t b[2][kSaeBN * kSaeLd];
};

__device__ __forceinline__ float sae_relu(float pre) { return pre > 0.0f ? pre : 0.0f; }

// acc[i][j] = this wave's 64x64 part of the product for the tile at (m0, n0).
// Ends with a barrier, after which the tile buffers are free.
__device__ __forceinline__ void sae_tile_mma(const SaeGemm& g, uint32_t m0, uint32_t n0, SaeTileLds& sh,
                                             f32x16 (&acc)[2][2]) {
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const uint32_t wm = w >> 1, wn = w & 1;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  const uint32_t nchunk = g.d_model / kSaeBK;
  // piece id = q * kSaeBS + tid is row id / 8, 16-byte segment id % 8 of the
  // chunk.  Two register sets hold the chunks in flight: chunk c + 2 is
  // loaded while chunk c is computed and stored to LDS after chunk c + 1 is.
  // Rows past B and columns past d_dict load the last row or column instead
  // (no branch around a load, so the loads' waits stay exact): they only
  // feed accumulators of rows and columns the epilogues skip.
  u32x4v ra[2][kSaeApieces], rb[2][kSaeBpieces];
  auto gload = [&](uint32_t kc, u32x4v (&xa)[kSaeApieces], u32x4v (&xb)[kSaeBpieces]) {
    const size_t col = static_cast<size_t>(kc) * kSaeBK;
#pragma unroll
    for (int q = 0; q < kSaeApieces; ++q) {
      const uint32_t id = q * kSaeBS + tid, gm = min(m0 + (id >> 3), g.B - 1);
      xa[q] = *reinterpret_cast<const u32x4v*>(g.x + static_cast<size_t>(gm) * g.d_model + col + (id & 7) * 8);
    }
#pragma unroll
    for (int q = 0; q < kSaeBpieces; ++q) {
      const uint32_t id = q * kSaeBS + tid, gn = min(n0 + (id >> 3), g.d_dict - 1);
      xb[q] = *reinterpret_cast<const u32x4v*>(g.w + static_cast<size_t>(gn) * g.d_model + col + (id & 7) * 8);
    }
  };
  auto lstore = [&](uint32_t buf, const u32x4v (&xa)[kSaeApieces], const u32x4v (&xb)[kSaeBpieces]) {
#pragma unroll
    for (int q = 0; q < kSaeApieces; ++q) {
      const uint32_t id = q * kSaeBS + tid;
      *reinterpret_cast<u32x4v*>(&sh.a[buf][(id >> 3) * kSaeLd + (id & 7) * 8]) = xa[q];
    }
#pragma unroll
    for (int q = 0; q < kSaeBpieces; ++q) {
      const uint32_t id = q * kSaeBS + tid;
      *reinterpret_cast<u32x4v*>(&sh.b[buf][(id >> 3) * kSaeLd + (id & 7) * 8]) = xb[q];
    }
  };
  auto compute = [&](uint32_t buf) {
#pragma unroll
    for (uint32_t ks = 0; ks < kSaeBK / 16; ++ks) {
      const uint32_t kofs = ks * 16 + 8 * (lane >> 5);
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = *reinterpret_cast<const bf16x8*>(&sh.a[buf][(wm * 64 + i * 32 + (lane & 31)) * kSaeLd + kofs]);
        fb[i] = *reinterpret_cast<const bf16x8*>(&sh.b[buf][(wn * 64 + i * 32 + (lane & 31)) * kSaeLd + kofs]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  };
  __syncthreads();  // the previous tile's epilogue is done with the buffers
  gload(0, ra[0], rb[0]);
  lstore(0, ra[0], rb[0]);
  if (nchunk > 1) gload(1, ra[1], rb[1]);
  __syncthreads();
  // Chunk c is in LDS buffer c % 2 and register set c % 2.  The steady loop
  // has no branch around its loads, so the compiler's waits before each LDS
  // store cover that set's loads only and chunk c + 2 stays in flight; the
  // last one to three chunks are peeled off.
  // (sched_barrier keeps the compiler from sinking the loads below the
  // MFMAs, which would shorten their lead to under one chunk.)
  uint32_t kc = 0;
  for (; kc + 3 < nchunk; kc += 2) {
    gload(kc + 2, ra[0], rb[0]);
    __builtin_amdgcn_sched_barrier(0);
    compute(0);
    lstore(1, ra[1], rb[1]);  // buffer 1 was last read before the previous barrier
    __syncthreads();
    gload(kc + 3, ra[1], rb[1]);
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    lstore(0, ra[0], rb[0]);  // buffer 0 was read before the barrier above
    __syncthreads();
  }
  if (kc + 2 < nchunk) {  // chunks kc, kc + 1, kc + 2
    gload(kc + 2, ra[0], rb[0]);
    __builtin_amdgcn_sched_barrier(0);
    compute(0);
    lstore(1, ra[1], rb[1]);
    __syncthreads();
    compute(1);
    lstore(0, ra[0], rb[0]);
    __syncthreads();
    compute(0);
  } else if (kc + 1 < nchunk) {  // chunks kc, kc + 1
    compute(0);
    lstore(1, ra[1], rb[1]);
    __syncthreads();
    compute(1);
  } else {  // chunk kc
    compute(0);
  }
  __syncthreads();
}

// XCD-aware tile order.  Workgroups are dispatched to the 8 XCDs round-robin
// (workgroup b runs on XCD b % 8), each XCD with its own L2.  The grid is a
// multiple of V = min(8, grid) workgroups; group x = b % V owns the column
// tiles [nlo, nlo + nx) -- a slice of W_enc that stays in its XCD's L2 --
// and walks all row tiles; its workgroups (b / V = 0, 1, ...) take the
// group's tiles in row-major order with stride grid / V, so consecutive tiles
// of an XCD share their row block of x.  Every column tile has one owner.
constexpr uint32_t kXcds = 8;

struct XcdTiles {
  uint32_t nlo, nx, count;  // the group's column tiles [nlo, nlo + nx), tiles in all
  uint32_t first, stride;   // this workgroup's first tile of the group, and the step
  __device__ __forceinline__ XcdTiles(uint32_t tiles_m, uint32_t tiles_n) {
    const uint32_t V = gridDim.x < kXcds ? gridDim.x : kXcds;
    const uint32_t x = blockIdx.x % V;
    nlo = tiles_n * x / V;
    nx = tiles_n * (x + 1) / V - nlo;
    count = tiles_m * nx;
    first = blockIdx.x / V;
    stride = gridDim.x / V;
  }
  __device__ __forceinline__ void tile(uint32_t t, uint32_t& m0, uint32_t& n0) const {
    m0 = (t / nx) * kSaeBM;
    n0 = (nlo + t % nx) * kSaeBN;
  }
};

// Tile-local row and column of accumulator element v of block (i, j).
__device__ __forceinline__ uint32_t sae_row(uint32_t lane, uint32_t w, int i, int v) {
  return (w >> 1) * 64 + i * 32 + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
}
__device__ __forceinline__ uint32_t sae_col(uint32_t lane, uint32_t w, int j) {
  return (w & 1) * 64 + j * 32 + (lane & 31);
}

// ------------------------------------------------------------ stage 1 -----
// k_sae_sample: every draw's latent key, into skeys[S].  k_sae_union: each
// workgroup of 1024 threads takes 4096 of them and keeps its top-t (the
// union stays small enough for one workgroup to select tau from in LDS even
// when t is in the hundreds).
constexpr int kSaeUnionBS = 1024;
constexpr uint32_t kSaeUnionPer = 4 * kSaeUnionBS;

struct SaeSampleArgs {
  SaeGemm g;
  uint64_t seed;
  uint32_t S;
  uint32_t* skeys;
  CallState* st;
  uint32_t* seg_cnt;
  uint32_t* fhist;
};

// Draw j is word j%4 of Philox block j/4 (row 0) over the N = B*d_dict
// flattened latents.  Each wave takes 32 draws: lanes L and L+32 feed draw
// L%32's input row and weight row to the MFMA, and the draw's latent is the
// diagonal element (L%32, L%32) of the 32x32 result -- the same sums, in the
// same order, as the GEMM computes for that element.  The 32 rows are staged
// through the wave's own LDS one 64-wide chunk at a time, 8 lanes per
// 128-byte row piece, so the loads are coalesced rather than one 16-byte
// line per lane.
__global__ __launch_bounds__(kSampBS) void k_sae_sample(SaeSampleArgs a) {
  constexpr int NW = kSampBS / kWave;
  __shared__ __align__(16) uint16_t s_x[NW][32 * kSaeLd];
  __shared__ __align__(16) uint16_t s_w[NW][32 * kSaeLd];
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  if (blockIdx.x == 0) reset_state(a.st, a.seg_cnt, a.fhist);
  const uint32_t j = (blockIdx.x * NW + w) * 32 + (lane & 31);
  const bool in = j < a.S;
  uint32_t r = 0, c = 0;
  if (in) {
    const U64x4 p = philox4x64_10(j >> 2, 0, 0, 0, a.seed, 0);
    const uint64_t flat = index_of_word(p.w[j & 3], static_cast<uint64_t>(a.g.B) * a.g.d_dict);
    r = static_cast<uint32_t>(flat / a.g.d_dict);
    c = static_cast<uint32_t>(flat % a.g.d_dict);
  }
  // piece s*64 + lane of a chunk: row (s*64 + lane) / 8, 16-byte segment lane % 8
  uint32_t pr[4], pc[4];
  bool pin[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int row = (s * kWave + static_cast<int>(lane)) >> 3;
    pr[s] = __shfl(r, row, kWave);
    pc[s] = __shfl(c, row, kWave);
    pin[s] = __shfl(in ? 1 : 0, row, kWave) != 0;
  }
  const uint32_t seg = lane & 7;
  f32x16 acc{};
  for (uint32_t k0 = 0; k0 < a.g.d_model; k0 += kSaeBK) {
    u32x4v vx[4], vw[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      vx[s] = pin[s] ? *reinterpret_cast<const u32x4v*>(a.g.x + static_cast<size_t>(pr[s]) * a.g.d_model + k0 + seg * 8)
                     : u32x4v{0u, 0u, 0u, 0u};
      vw[s] = pin[s] ? *reinterpret_cast<const u32x4v*>(a.g.w + static_cast<size_t>(pc[s]) * a.g.d_model + k0 + seg * 8)
                     : u32x4v{0u, 0u, 0u, 0u};
    }
    // (the wave's previous chunk was read by this wave's own earlier LDS
    // reads, which complete in order before these writes)
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t row = (s * kWave + lane) >> 3;
      *reinterpret_cast<u32x4v*>(&s_x[w][row * kSaeLd + seg * 8]) = vx[s];
      *reinterpret_cast<u32x4v*>(&s_w[w][row * kSaeLd + seg * 8]) = vw[s];
    }
#pragma unroll
    for (uint32_t ks = 0; ks < kSaeBK / 16; ++ks) {
      const uint32_t kofs = ks * 16 + 8 * (lane >> 5);
      const bf16x8 fa = *reinterpret_cast<const bf16x8*>(&s_x[w][(lane & 31) * kSaeLd + kofs]);
      const bf16x8 fb = *reinterpret_cast<const bf16x8*>(&s_w[w][(lane & 31) * kSaeLd + kofs]);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, acc, 0, 0, 0);
    }
  }
  // element (i, i), i = lane % 32, is held by lane i + 32*((i>>2)&1) as
  // accumulator 4*(i>>3) + (i&3)
  const uint32_t i = lane & 31, v = 4 * (i >> 3) + (i & 3);
  float d = acc[0];
#pragma unroll
  for (int q = 1; q < 16; ++q) d = v == static_cast<uint32_t>(q) ? acc[q] : d;
  if (in && (lane >> 5) == ((i >> 2) & 1)) a.skeys[j] = key_f32(__float_as_uint(sae_relu(d + a.g.bias[c])));
}

struct SaeUnionArgs {
  const uint32_t* skeys;
  uint32_t S, t, tcap;
  uint32_t* union_keys;
};

__global__ __launch_bounds__(kSaeUnionBS) void k_sae_union(SaeUnionArgs a) {
  __shared__ SampleUnionShared<kSaeUnionBS> sh;
  const uint32_t b = blockIdx.x, tid = threadIdx.x;
  const uint32_t j0 = b * kSaeUnionPer;
  const uint32_t nb = min(kSaeUnionPer, a.S - j0);
  uint32_t kv[4];
  uint32_t valid = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t j = 4 * tid + q;
    kv[q] = j < nb ? a.skeys[j0 + j] : 0u;
    if (j < nb) valid |= 1u << q;
  }
  sample_block_top<kSaeUnionBS, 32>(kv, valid, nb, a.t, a.union_keys + static_cast<size_t>(b) * a.tcap, sh);
}

// ------------------------------------------------------- thresholds ------
// A latent relu(acc + b_enc[j]) survives iff its key is >= tau.  With tau
// above the key of +0 that is fl(acc + b_enc[j]) >= tau as floats (relu
// lifts nothing to a positive value), and since fl(acc + b) does not decrease
// as acc grows, it is acc >= thr[j] for the smallest float thr[j] that passes
// (NaN when none does): one compare per latent in the filter's epilogue.
// thr[j] is found by bisection over the floats in key order (-0 and +0 pass
// alike, so the float compare agrees with the key order).
__device__ __forceinline__ bool sae_passes(uint32_t akey, float b, float tf) {
  return __uint_as_float(bits_from_key_f32(akey)) + b >= tf;
}

__global__ void k_sae_thresholds(const CallState* st, const float* bias, uint32_t d_dict, float* thr) {
  const uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= d_dict) return;
  const float tf = __uint_as_float(bits_from_key_f32(st->tau_key));
  const float b = bias[j];
  uint32_t lo = key_f32(0xFF800000u), hi = key_f32(0x7F800000u);  // -inf, +inf
  if (!sae_passes(hi, b, tf)) {
    thr[j] = __uint_as_float(0x7FC00000u);
    return;
  }
  while (lo < hi) {  // the smallest passing key in [lo, hi]
    const uint32_t mid = lo + (hi - lo) / 2;
    if (sae_passes(mid, b, tf)) hi = mid; else lo = mid + 1;
  }
  thr[j] = __uint_as_float(bits_from_key_f32(lo));
}

// ------------------------------------------------------------ stage 3 -----
struct SaeFilterArgs {
  SaeGemm g;
  uint32_t tiles_m, tiles_n;
  CallState* st;
  uint32_t seg_cap;
  uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  uint32_t* fhist;   // refinement histogram, zero on entry
  const float* thr;  // [d_dict] from k_sae_thresholds
};

constexpr uint32_t kSaeSlice = kStage / (kSaeBS / kWave);  // survivors a wave stages in LDS



// Persistent: workgroup b takes its XCD group's tiles (XcdTiles).  Each
// wave stages survivors (key, index) in its own slice of the workgroup stage
// with a wave-uniform fill count, so the common path takes no atomics; a
// slice is appended to the workgroup's candidate segment (one atomic) when it
// is half full at a tile's start, and at the end.  The log-bin counts and the
// maximum key are taken from the slice as it is appended.
//
// Per latent of a full tile, the fast epilogue costs one compare against the
// column threshold and a wave-uniform branch; the body runs only for
// accumulator elements with a survivor in the wave.  A tile whose survivors
// do not fit the slice, a tile cut by the last row, and every tile when tau
// is at most key(+0) (all latents survive) go through the general epilogue: the accumulators pass through LDS and each
// element's survivors are appended to the segment directly.
__global__ __launch_bounds__(kSaeBS) void k_sae_filter(SaeFilterArgs a) {
  __shared__ SaeTileLds tl;
  __shared__ uint32_t s_skey[kStage], s_sidx[kStage];
  __shared__ uint32_t s_hist[kLogBins];
  __shared__ uint32_t s_wmax[kSaeBS / kWave];
  const uint32_t b = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const uint32_t seg = b & (kSegs - 1);
  const uint32_t tau = a.st->tau_key;
  const bool all = tau <= 0x80000000u;  // tau <= key(+0): every latent survives
  for (uint32_t i = tid; i < kLogBins; i += kSaeBS) s_hist[i] = 0;  // visible after the first tile's barrier
  uint32_t* const seg_counter = a.seg_cnt + seg * kSegStride;
  uint32_t* const seg_key = a.seg_key + static_cast<size_t>(seg) * a.seg_cap;
  uint32_t* const seg_idx = a.seg_idx + static_cast<size_t>(seg) * a.seg_cap;
  uint32_t* const wkey = s_skey + w * kSaeSlice;
  uint32_t* const widx = s_sidx + w * kSaeSlice;
  uint32_t wcnt = 0;  // wave-uniform fill of the wave's slice
  uint32_t my_max = 0;
  // one survivor's log-bin count and maximum
  auto note = [&](uint32_t key) {
    atomicAdd(&s_hist[log_bin(key - tau)], 1u);
    my_max = max(my_max, key);
  };
  // the wave's n staged survivors to the segment (a wave's LDS operations
  // execute in program order, so the slice reads see its writes)
  auto flush = [&](uint32_t n) {
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(seg_counter, n);
    base = __shfl(base, 0, kWave);
    for (uint32_t q = lane; q < n; q += kWave) {
      const uint32_t key = wkey[q], gp = base + q;
      note(key);
      if (gp < a.seg_cap) {
        seg_key[gp] = key;
        seg_idx[gp] = widx[q];
      }
    }
  };
  float* const stage = reinterpret_cast<float*>(&tl) + w * (32 * kWave);
  static_assert(kSaeBS / kWave * 32 * kWave * 4 <= sizeof(SaeTileLds), "epilogue stage");
  const XcdTiles xt(a.tiles_m, a.tiles_n);
  for (uint32_t tl_i = xt.first; tl_i < xt.count; tl_i += xt.stride) {
    uint32_t m0, n0;
    xt.tile(tl_i, m0, n0);
    // the lane's two columns: threshold, bias (loaded ahead of the MFMAs)
    float thr[2], bias[2];
    bool pass_all[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t c = n0 + sae_col(lane, w, j), cc = min(c, a.g.d_dict - 1);
      const bool colok = c < a.g.d_dict;
      const float th = a.thr[cc], bi = a.g.bias[cc];  // unconditional loads, then the column check
      thr[j] = colok ? th : __uint_as_float(0x7FC00000u);
      bias[j] = colok ? bi : 0.0f;
      pass_all[j] = all && colok;
    }
    if (wcnt > kSaeSlice / 2) {
      flush(wcnt);
      wcnt = 0;
    }
    f32x16 acc[2][2];
    sae_tile_mma(a.g, m0, n0, tl, acc);
    const uint32_t wcnt0 = wcnt;
    if (!all && m0 + kSaeBM <= a.g.B) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float av = acc[i][j][v];
            const bool ok = av >= thr[j];
            const uint64_t s = __ballot(ok);
            if (s == 0) continue;
            if (ok) {
              const uint32_t pos =
                  wcnt + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(s >> 32),
                                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(s), 0u));
              if (pos < kSaeSlice) {
                wkey[pos] = key_f32(__float_as_uint(sae_relu(av + bias[j])));
                widx[pos] = (m0 + sae_row(lane, w, i, v)) * a.g.d_dict + n0 + sae_col(lane, w, j);
              }
            }
            wcnt += static_cast<uint32_t>(__popcll(s));
          }
      if (wcnt <= kSaeSlice) continue;
      wcnt = wcnt0;  // the slice overflowed: drop this tile's entries, redo it below
    }
    // General epilogue, per half i: the lane's 32 accumulators through the
    // wave's 8 KB of the (idle) tile buffers; element e = 16 j + v.
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const f32x16& src = acc[i][q >> 2];
        const int v0 = 4 * (q & 3);
        *reinterpret_cast<float4*>(&stage[lane * 32 + 4 * q]) =
            make_float4(src[v0], src[v0 + 1], src[v0 + 2], src[v0 + 3]);
      }
      for (uint32_t e = 0; e < 32; ++e) {
        const uint32_t j = e >> 4, v = e & 15;
        const float av = stage[lane * 32 + e];
        const uint32_t r = m0 + (w >> 1) * 64 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const bool ok = (j ? pass_all[1] || av >= thr[1] : pass_all[0] || av >= thr[0]) && r < a.g.B;
        const uint64_t s = __ballot(ok);
        if (s == 0) continue;
        uint32_t base = 0;
        if (lane == 0) base = atomicAdd(seg_counter, static_cast<uint32_t>(__popcll(s)));
        base = __shfl(base, 0, kWave);
        if (ok) {
          const uint32_t gp = base + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(s >> 32),
                                                               __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(s), 0u));
          const uint32_t key = key_f32(__float_as_uint(sae_relu(av + (j ? bias[1] : bias[0]))));
          note(key);
          if (gp < a.seg_cap) {
            seg_key[gp] = key;
            seg_idx[gp] = r * a.g.d_dict + n0 + (w & 1) * 64 + j * 32 + (lane & 31);
          }
        }
      }
    }
  }
  if (wcnt) flush(wcnt);
  const uint32_t wm = wave_max_u32(my_max);
  if (lane == 0) s_wmax[w] = wm;
  __syncthreads();
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < kSaeBS / kWave; ++i) m = max(m, s_wmax[i]);
  if (tid == 0) a.blk_max[b] = m;
  if (m) {  // survivors' keys are >= key(+0) > 0
    for (uint32_t i = tid; i < kLogBins; i += kSaeBS) {
      const uint32_t c = s_hist[i];
      if (c) atomicAdd(&a.fhist[i], c);
    }
  }
}

// ------------------------------------------------------------- dense ------
struct SaeDenseArgs {
  SaeGemm g;
  uint32_t tiles_m, tiles_n;
  float* out;               // [B, d_dict]
  const uint32_t* seg_cnt;  // null: always write; else only when the count is outside [k_req, M]
  uint32_t k_req, M;
};

__global__ __launch_bounds__(kSaeBS) void k_sae_dense(SaeDenseArgs a) {
  __shared__ SaeTileLds tl;
  if (a.seg_cnt) {
    uint32_t total = 0;
#pragma unroll
    for (int x = 0; x < kSegs; ++x) total += a.seg_cnt[x * kSegStride];
    if (total >= a.k_req && total <= a.M) return;  // filtered: the candidates suffice
  }
  const uint32_t lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const XcdTiles xt(a.tiles_m, a.tiles_n);
  for (uint32_t tl_i = xt.first; tl_i < xt.count; tl_i += xt.stride) {
    uint32_t m0, n0;
    xt.tile(tl_i, m0, n0);
    float bias[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) bias[j] = a.g.bias[min(n0 + sae_col(lane, w, j), a.g.d_dict - 1)];
    f32x16 acc[2][2];
    sae_tile_mma(a.g, m0, n0, tl, acc);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t c = n0 + sae_col(lane, w, j);
      if (c >= a.g.d_dict) continue;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t r = m0 + sae_row(lane, w, i, v);
          if (r < a.g.B) a.out[static_cast<size_t>(r) * a.g.d_dict + c] = sae_relu(acc[i][j][v] + bias[j]);
        }
    }
  }
}

// ------------------------------------------------------------ decode ------
// Selected latents grouped by row: counts, offsets, a scatter, then one
// workgroup per row places its entries by latent index in LDS and sums them
// in ascending index order.
constexpr uint32_t kDecMaxDict = 16384;  // LDS per row: one float and one flag per latent
constexpr int kDecBS = 256;

struct DecArgs {
  const float* vals;
  const int64_t* idx;  // flat b*d_dict + j; -1 (padding) and out-of-range entries are skipped
  uint32_t K, B, d_model, d_dict;
  const uint16_t* w;   // W_dec [d_dict, d_model] bf16 bits
  const float* bias;   // b_dec [d_model]
  float* out;          // [B, d_model]
  uint32_t* row_cnt;   // [B + 1]
  uint32_t* row_off;   // [B + 1]
  uint32_t* row_fill;  // [B]
  uint32_t* grouped;   // [K] positions into vals/idx
};

__global__ void k_dec_clear(DecArgs a) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i <= a.B; i += gridDim.x * blockDim.x) {
    a.row_cnt[i] = 0;
    if (i < a.B) a.row_fill[i] = 0;
  }
}

__global__ void k_dec_count(DecArgs a) {
  const uint32_t e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= a.K) return;
  const int64_t f = a.idx[e];
  if (f >= 0 && static_cast<uint64_t>(f) < static_cast<uint64_t>(a.B) * a.d_dict)
    atomicAdd(&a.row_cnt[static_cast<uint64_t>(f) / a.d_dict], 1u);
}

__global__ __launch_bounds__(1024) void k_dec_scan(DecArgs a) {
  __shared__ uint32_t wsum[20];
  __shared__ uint32_t s_carry;
  if (threadIdx.x == 0) s_carry = 0;
  __syncthreads();
  for (uint32_t base = 0; base < a.B; base += 1024) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < a.B ? a.row_cnt[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_sum<1024>(v, wsum, &tot);
    if (i < a.B) a.row_off[i] = s_carry + ex;
    __syncthreads();
    if (threadIdx.x == 0) s_carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) a.row_off[a.B] = s_carry;
}

__global__ void k_dec_scatter(DecArgs a) {
  const uint32_t e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= a.K) return;
  const int64_t f = a.idx[e];
  if (f < 0 || static_cast<uint64_t>(f) >= static_cast<uint64_t>(a.B) * a.d_dict) return;  // padding or out of range
  const uint32_t r = static_cast<uint32_t>(static_cast<uint64_t>(f) / a.d_dict);
  a.grouped[a.row_off[r] + atomicAdd(&a.row_fill[r], 1u)] = e;
}

__global__ __launch_bounds__(kDecBS) void k_dec_rows(DecArgs a) {
  __shared__ float s_val[kDecMaxDict];
  __shared__ uint32_t s_has[kDecMaxDict / 32];
  __shared__ uint32_t s_list[kDecMaxDict];
  __shared__ uint32_t wsum[20];
  const uint32_t r = blockIdx.x, tid = threadIdx.x;
  const uint32_t nw = (a.d_dict + 31) / 32;
  for (uint32_t i = tid; i < nw; i += kDecBS) s_has[i] = 0;
  __syncthreads();
  const uint32_t e0 = a.row_off[r], e1 = a.row_off[r + 1];
  for (uint32_t p = e0 + tid; p < e1; p += kDecBS) {
    const uint32_t e = a.grouped[p];
    const uint32_t j = static_cast<uint32_t>(static_cast<uint64_t>(a.idx[e]) % a.d_dict);
    s_val[j] = a.vals[e];
    atomicOr(&s_has[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  // the row's latent indices, ascending: a prefix sum over the flag words
  uint32_t n_list = 0;
  for (uint32_t base = 0; base < nw; base += kDecBS) {
    const uint32_t i = base + tid;
    const uint32_t word = i < nw ? s_has[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_sum<kDecBS>(__popc(word), wsum, &tot);
    uint32_t pos = n_list + ex, rest = word;
    while (rest) {
      const uint32_t bit = __builtin_ctz(rest);
      rest &= rest - 1;
      s_list[pos++] = i * 32 + bit;
    }
    n_list += tot;
    __syncthreads();
  }
  for (uint32_t d = tid; d < a.d_model; d += kDecBS) {
    float acc = 0.0f;
    for (uint32_t q = 0; q < n_list; ++q) {
      const uint32_t j = s_list[q];
      const uint32_t bits = static_cast<uint32_t>(a.w[static_cast<size_t>(j) * a.d_model + d]) << 16;
      acc = fmaf(s_val[j], __uint_as_float(bits), acc);
    }
    a.out[static_cast<size_t>(r) * a.d_model + d] = acc + a.bias[d];
  }
}

// ------------------------------------------------------------- host -------
static uint32_t cdiv_s(uint64_t a, uint64_t b) { return static_cast<uint32_t>((a + b - 1) / b); }

// Persistent GEMM grid: one workgroup per CU (the LDS of a 256 x 128 tile,
// double-buffered, allows one), a multiple of the XCD count when there are
// enough tiles.
static uint32_t sae_grid(uint32_t tiles) {
  const uint32_t cus = static_cast<uint32_t>(device_cu_count());
  uint32_t g = cus < kSaeMaxBlocks ? cus : kSaeMaxBlocks;
  if (tiles < g) g = tiles;
  return g >= kXcds ? g / kXcds * kXcds : g;
}

SaeLayout sae_layout(const profk_plan_t& plan, uint32_t B, uint32_t d_dict, int num_cus) {
  SaeLayout S;
  S.flat = flat_layout(plan, PROFK_F32, num_cus);
  S.G = sae_grid(cdiv_s(B, kSaeBM) * cdiv_s(d_dict, kSaeBN));
  if (S.G > S.flat.G_f) S.G = S.flat.G_f >= kXcds ? S.flat.G_f / kXcds * kXcds : S.flat.G_f;  // blk_max: G_f entries
  const uint32_t Sn = static_cast<uint32_t>(plan.S), t = static_cast<uint32_t>(plan.t);
  S.G_u = cdiv_s(Sn, kSaeUnionPer);
  S.tcap_u = t < kSaeUnionPer ? t : kSaeUnionPer;
  const uint32_t last_nb = Sn - (S.G_u - 1) * kSaeUnionPer;
  S.union_n_u = (S.G_u - 1) * S.tcap_u + (t < last_nb ? t : last_nb);  // fits the vector path's union area
  S.off_skeys = (S.flat.bytes + 255) & ~static_cast<size_t>(255);
  S.off_thr = (S.off_skeys + static_cast<size_t>(Sn) * 4 + 255) & ~static_cast<size_t>(255);
  S.off_dense = (S.off_thr + static_cast<size_t>(d_dict) * 4 + 255) & ~static_cast<size_t>(255);
  S.bytes = S.off_dense + static_cast<size_t>(B) * d_dict * 4;
  return S;
}

static SaeGemm gemm_of(const SaeCall& c) {
  return SaeGemm{static_cast<const uint16_t*>(c.x), static_cast<const uint16_t*>(c.w), c.bias, c.B, c.d_model,
                 c.d_dict};
}

hipError_t launch_sae_dense(const SaeCall& c, float* out) {
  (void)hipGetLastError();
  const uint32_t tm = cdiv_s(c.B, kSaeBM), tn = cdiv_s(c.d_dict, kSaeBN);
  SaeDenseArgs da{gemm_of(c), tm, tn, out, nullptr, 0, 0};
  hipLaunchKernelGGL(k_sae_dense, dim3(sae_grid(tm * tn)), dim3(kSaeBS), 0, c.stream, da);
  return hipGetLastError();
}

hipError_t launch_sae_topk(const SaeCall& c) {
  (void)hipGetLastError();
  const profk_plan_t& p = *c.plan;
  const FlatLayout& L = c.L.flat;
  uint8_t* ws = c.ws;
  float* dense = reinterpret_cast<float*>(ws + c.L.off_dense);
  const uint32_t N = c.B * c.d_dict;
  FlatCall fc{};
  fc.plan = c.plan;
  fc.dtype = PROFK_F32;
  fc.values = dense;
  fc.n = N;
  fc.k = c.K;
  fc.seed = c.seed;
  fc.row = 0;
  fc.out_vals = c.out_vals;
  fc.out_idx = c.out_idx;
  fc.ws = ws;
  fc.L = L;
  fc.stream = c.stream;
  fc.info = c.info;
  if (p.mode == PROFK_MODE_DIRECT) {
    // no sampling pays off: the dense latents, then the exact selection
    hipError_t e = launch_sae_dense(c, dense);
    if (e != hipSuccess) return e;
    return launch_flat(fc);
  }
  CallState* st = reinterpret_cast<CallState*>(ws + L.off_state);
  uint32_t* seg_cnt = reinterpret_cast<uint32_t*>(ws + L.off_segcnt);
  uint32_t* fhist = reinterpret_cast<uint32_t*>(ws + L.off_fhist);
  uint32_t* uk = reinterpret_cast<uint32_t*>(ws + L.off_union);
  const SaeGemm g = gemm_of(c);
  hipError_t e = launch_sae_sample(c);
  if (e != hipSuccess) return e;
  SaeUnionArgs ua{reinterpret_cast<const uint32_t*>(ws + c.L.off_skeys), static_cast<uint32_t>(p.S),
                  static_cast<uint32_t>(p.t), c.L.tcap_u, uk};
  hipLaunchKernelGGL(k_sae_union, dim3(c.L.G_u), dim3(kSaeUnionBS), 0, c.stream, ua);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = launch_select_tau(uk, c.L.union_n_u, static_cast<uint32_t>(p.t), 32, st, c.stream)) != hipSuccess)
    return e;
  float* thr = reinterpret_cast<float*>(ws + c.L.off_thr);
  hipLaunchKernelGGL(k_sae_thresholds, dim3(cdiv_s(c.d_dict, 256)), dim3(256), 0, c.stream, st, c.bias, c.d_dict,
                     thr);
  const uint32_t tm = cdiv_s(c.B, kSaeBM), tn = cdiv_s(c.d_dict, kSaeBN);
  SaeFilterArgs fa{g, tm, tn, st, L.seg_cap, seg_cnt,
                   reinterpret_cast<uint32_t*>(ws + L.off_seg_key), reinterpret_cast<uint32_t*>(ws + L.off_seg_idx),
                   reinterpret_cast<uint32_t*>(ws + L.off_blk_max), fhist, thr};
  if (c.ev_before) (void)hipEventRecord(c.ev_before, c.stream);
  hipLaunchKernelGGL(k_sae_filter, dim3(c.L.G), dim3(kSaeBS), 0, c.stream, fa);
  if (c.ev_after) (void)hipEventRecord(c.ev_after, c.stream);
  // the dense latents only when the candidates do not suffice (exact fallback)
  SaeDenseArgs da{g, tm, tn, dense, seg_cnt, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.M)};
  hipLaunchKernelGGL(k_sae_dense, dim3(sae_grid(tm * tn)), dim3(kSaeBS), 0, c.stream, da);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_refine(fc, c.L.G);
}

hipError_t launch_sae_sample(const SaeCall& c) {
  (void)hipGetLastError();
  const FlatLayout& L = c.L.flat;
  uint32_t* skeys = c.sample_keys ? c.sample_keys : reinterpret_cast<uint32_t*>(c.ws + c.L.off_skeys);
  const uint32_t S = static_cast<uint32_t>(c.plan->S);
  SaeSampleArgs sa{gemm_of(c), c.seed, S, skeys, reinterpret_cast<CallState*>(c.ws + L.off_state),
                   reinterpret_cast<uint32_t*>(c.ws + L.off_segcnt), reinterpret_cast<uint32_t*>(c.ws + L.off_fhist)};
  hipLaunchKernelGGL(k_sae_sample, dim3(cdiv_s(S, 32 * (kSampBS / kWave))), dim3(kSampBS), 0, c.stream, sa);
  return hipGetLastError();
}

size_t sae_decode_workspace(uint32_t B, uint32_t K) {
  return (static_cast<size_t>(B) * 3 + 2 + K) * 4 + 256;
}

hipError_t launch_sae_decode(const SaeDecodeCall& c) {
  (void)hipGetLastError();
  uint32_t* ws = static_cast<uint32_t*>(c.ws);
  DecArgs a{c.vals, c.idx, c.K, c.B, c.d_model, c.d_dict, static_cast<const uint16_t*>(c.w), c.bias, c.out,
            ws, ws + (c.B + 1), ws + 2 * (c.B + 1), ws + 2 * (c.B + 1) + c.B};
  const uint32_t gk = cdiv_s(c.K, 256);
  hipLaunchKernelGGL(k_dec_clear, dim3(cdiv_s(c.B + 1, 256)), dim3(256), 0, c.stream, a);
  if (gk) hipLaunchKernelGGL(k_dec_count, dim3(gk), dim3(256), 0, c.stream, a);
  hipLaunchKernelGGL(k_dec_scan, dim3(1), dim3(1024), 0, c.stream, a);
  if (gk) hipLaunchKernelGGL(k_dec_scatter, dim3(gk), dim3(256), 0, c.stream, a);
  hipLaunchKernelGGL(k_dec_rows, dim3(c.B), dim3(kDecBS), 0, c.stream, a);
  return hipGetLastError();
}

uint32_t sae_decode_max_dict() { return kDecMaxDict; }

}  // namespace profk
