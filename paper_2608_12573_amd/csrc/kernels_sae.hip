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
//                  for bit);
//   k_key_union,   stage 2 (shared with the vector path): per-block top-t
//   k_select_tau   lists of the S keys, then one block over their union;
//   k_sae_thresholds  each column's accumulator threshold for tau, with its
//                  bias;
//   k_sae_filter   the GEMM with stage 3 in its epilogue: survivors are
//                  compacted as the vector filter does it, so the vector
//                  path's refinement (stage 4) runs unchanged;
//   k_sae_dense    the same GEMM with a dense epilogue: for the exact
//                  fallback (it returns at once when the filter's count is in
//                  range), for plans without sampling, and as an inspection
//                  entry point.
// Sparse decode (k_dec_*): x_hat[b, :] = sum over b's selected latents of
// z W_dec[j, :] + b_dec, grouped by row and summed in ascending j, so the
// result does not depend on the order the selection lists them in.
//
// One 32x32x16 MFMA step rounds once: the accumulator and its 16 products
// are summed together before rounding to fp32.
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "sample_union.h"

namespace profk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

constexpr int kSaeBS = 512;              // threads of a GEMM workgroup (8 waves)
constexpr uint32_t kSaeBK = 64;           // d_model chunk of the sample kernel
constexpr uint32_t kSaeLd = kSaeBK + 8;   // its LDS row stride in bf16 elements
constexpr uint32_t kSaeMaxBlocks = 1024;

struct SaeGemm {
  const uint16_t* x;  // [B, d_model] bf16 bits, 16-byte aligned rows
  const uint16_t* w;  // [d_dict, d_model]
  const float* bias;  // [d_dict]
  uint32_t B, d_model, d_dict;
};

__device__ __forceinline__ float sae_relu(float pre) { return pre > 0.0f ? pre : 0.0f; }


// XCD-aware tile order.  Workgroups are dispatched to the 8 XCDs round-robin
// (workgroup b runs on XCD b % 8), each XCD with its own L2.  The grid is a
// multiple of V = min(8, grid) workgroups; group x = b % V owns the column
// tiles [nlo, nlo + nx) -- a slice of W_enc that stays in its XCD's L2 --
// and walks all row tiles; its workgroups (b / V = 0, 1, ...) take the
// group's tiles in row-major order with stride grid / V, so consecutive tiles
// of an XCD share their row block of x.  Every column tile has one owner.

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
};


// ------------------------------------------------------------ stage 1 -----
// k_sae_sample: every draw's latent key, into skeys[S]; k_key_union and
// k_select_tau then take the t-th largest of them.

struct SaeSampleArgs {
  SaeGemm g;
  uint64_t seed;
  uint32_t S;
  uint32_t* skeys;
  CallState* st;
  uint32_t* seg_cnt;
  uint32_t* fhist;
  uint32_t* bcur;   // null unless the call takes the large-k path
  uint32_t* ghist;  // null unless the call takes the large-k path
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
  if (blockIdx.x == 0) reset_state(a.st, a.seg_cnt, a.fhist, a.bcur, a.ghist);
  const uint32_t j = (blockIdx.x * NW + w) * 32 + (lane & 31);
  const bool in = j < a.S;
  uint32_t r = 0, c = 0;
  if (in) {
    const U64x4 p = philox4x64_10(j >> 2, 0, 0, 0, a.seed, 0);
    // word j % 4, chosen in registers (indexing p.w by a lane-varying value
    // would place it in scratch memory)
    const uint32_t q = j & 3;
    const uint64_t word = q == 0 ? p.w[0] : q == 1 ? p.w[1] : q == 2 ? p.w[2] : p.w[3];
    const uint64_t flat = index_of_word(word, static_cast<uint64_t>(a.g.B) * a.g.d_dict);
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
  // chunk k0 of the wave's 32 rows of x and of W_enc, into registers
  auto load_chunk = [&](uint32_t k0, u32x4v (&vx)[4], u32x4v (&vw)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      vx[s] = pin[s] ? *reinterpret_cast<const u32x4v*>(a.g.x + static_cast<size_t>(pr[s]) * a.g.d_model + k0 + seg * 8)
                     : u32x4v{0u, 0u, 0u, 0u};
      vw[s] = pin[s] ? *reinterpret_cast<const u32x4v*>(a.g.w + static_cast<size_t>(pc[s]) * a.g.d_model + k0 + seg * 8)
                     : u32x4v{0u, 0u, 0u, 0u};
    }
  };
  // the next chunk's loads are in flight while this chunk's MFMAs run
  u32x4v nx[4], nw[4];
  load_chunk(0, nx, nw);
  for (uint32_t k0 = 0; k0 < a.g.d_model; k0 += kSaeBK) {
    u32x4v vx[4], vw[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      vx[s] = nx[s];
      vw[s] = nw[s];
    }
    if (k0 + kSaeBK < a.g.d_model) load_chunk(k0 + kSaeBK, nx, nw);
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

// col[j] = {thr[j], b_enc[j]} for j < d_dict, and {NaN, 0} up to the
// padded length (a multiple of kSaeFBN), so that the filter copies a tile's
// columns whole.  When tau is at most key(+0) every latent survives (relu
// maps each to +0 or above) and thr[j] is -inf.
__global__ void k_sae_thresholds(const CallState* st, const float* bias, uint32_t d_dict, uint32_t d_pad,
                                 float2* col) {
  const uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= d_pad) return;
  if (j >= d_dict) {
    col[j] = float2{__uint_as_float(0x7FC00000u), 0.0f};
    return;
  }
  const uint32_t tau = st->tau_key;
  const float tf = __uint_as_float(bits_from_key_f32(tau));
  const float b = bias[j];
  if (tau <= 0x80000000u) {
    col[j] = float2{-__builtin_inff(), b};
    return;
  }
  uint32_t lo = key_f32(0xFF800000u), hi = key_f32(0x7F800000u);  // -inf, +inf
  if (!sae_passes(hi, b, tf)) {
    col[j] = float2{__uint_as_float(0x7FC00000u), b};
    return;
  }
  while (lo < hi) {  // the smallest passing key in [lo, hi]
    const uint32_t mid = lo + (hi - lo) / 2;
    if (sae_passes(mid, b, tf)) hi = mid; else lo = mid + 1;
  }
  col[j] = float2{__uint_as_float(bits_from_key_f32(lo)), b};
}

// ------------------------------------------------------------ stage 3 -----
struct SaeFilterArgs {
  SaeGemm g;
  uint32_t tiles_m, tiles_n;
  CallState* st;
  uint32_t seg_cap;
  uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  uint32_t* fhist;   // refinement histogram, zero on entry
  const float2* col;  // {threshold, bias} per column, padded to whole tiles (k_sae_thresholds)
};

constexpr uint32_t kSaeSlice = kStage / (kSaeBS / kWave);  // survivors a wave stages in LDS

// The filter's GEMM: 256 x 256 tiles (waves in a 4 x 2 grid, 64 x 128 each
// as 2 x 4 32x32 accumulators), twice the arithmetic per loaded byte and per
// LDS fragment read of 256 x 128 tiles with 64 x 64 wave blocks.  d_model is consumed in
// chunks of kSaeFK, in two LDS stages that direct-to-LDS loads fill
// (global_load_lds, 16 bytes per lane: lane L of a wave's instruction fills
// the granule at the instruction's base + L), so no registers stage them.
// Fragments are double-buffered in registers: the reads of a k-step are in
// flight during the previous k-step's MFMAs, and a chunk's last MFMAs are in
// flight during the wait and barrier for the next chunk.  The k-steps are the
// same 32x32x16 MFMAs in the same ascending order as k_sae_sample's, so every
// latent is bit-identical to the sample's and the dense kernel's.
constexpr uint32_t kSaeFBM = 256, kSaeFBN = 256, kSaeFK = 64;
constexpr uint32_t kSaeFSeg = kSaeFK / 8;              // 16-byte granules of a row in a chunk
constexpr uint32_t kSaeFGran = kSaeFBM * kSaeFSeg;     // granules of one operand stage
constexpr int kSaeFQ = kSaeFGran / kSaeBS;             // loads per lane, operand and chunk
constexpr int kSaeFKS = kSaeFK / 16;                   // k-steps per chunk
static_assert(kSaeFBN == kSaeFBM && kSaeFGran % kSaeBS == 0 && kSaeFKS % 2 == 0, "filter tile shape");
static_assert(kSaeBS / kWave == 8, "waves of the filter tile");

// s_waitcnt vmcnt(0) lgkmcnt(0), leaving expcnt alone (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt in 6:4, lgkmcnt in 11:8).
__device__ __forceinline__ void wait_loads_lds() { __builtin_amdgcn_s_waitcnt(0x7 << 4); }
// vmcnt(N) lgkmcnt(0)
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
}

// Granule of row `row`, 16-byte k segment `seg` in a stage: the XOR puts the
// eight rows that eight neighbouring lanes read together into eight
// different 16-byte bank groups.  Its inverse is itself.
__device__ __forceinline__ uint32_t sae_swz(uint32_t row, uint32_t seg) { return row * kSaeFSeg + (seg ^ (row & 7)); }

// Tile-local row and column of element v of accumulator (i, j) in the filter
// tile.
__device__ __forceinline__ uint32_t sae_frow(uint32_t lane, uint32_t w, int i, int v) {
  return (w >> 1) * 64 + i * 32 + 8 * (v / 4) + 4 * (lane >> 5) + (v % 4);
}
__device__ __forceinline__ uint32_t sae_fcol(uint32_t lane, uint32_t w, int j) {
  return (w & 1) * 128 + j * 32 + (lane & 31);
}

// Persistent: workgroup b takes its XCD group's tiles (XcdTiles).  A wave
// writes a tile's survivors to its own slice of LDS at their ranks (a
// wave-uniform fill count, no atomics); during the next tile's MFMAs they are
// converted to (key, flat index) and appended to the workgroup's candidate
// segment with one atomic, and their log-bin counts and maximum key taken.
//
// Epilogue: per accumulator element one compare against the column's
// threshold, ballots taken eight at a time, and a wave-uniform branch to the
// out-of-line body, taken only for elements with a survivor in the wave.
// Columns past d_dict have a NaN threshold, rows past B NaN accumulators (see
// issue), so neither passes; when tau is at most key(+0) every latent
// survives and in-range columns have the threshold -inf.
//
// CROSS (the chunks of a tile are even in number, so chunk c of every tile
// is in stage c % 2): the next tile's first chunk is awaited, and its second
// issued, before this tile's epilogue, so that they load meanwhile.
// Otherwise each tile starts its own loads behind a barrier.
//
// Waits: with two stages the chunk awaited is the newest one issued, so each
// wait is vmcnt(0) (with lgkmcnt(0), which also completes this wave's
// fragment reads of the stage refilled after the barrier); the barrier then
// covers the other waves' loads and reads.
// The dense variant (DENSE) runs the same GEMM and writes every latent
// relu(acc + b_enc[j]) to d.out instead of filtering; given d.chk it first
// returns when the candidate count there is within [k_req, M] (the exact
// fallback's case only).
struct SaeDenseOut {
  float* out;               // [B, d_dict]
  const uint32_t* chk;      // null: always write; else the filter's segment counters
  uint32_t k_req, M;
};

template <bool CROSS, bool DENSE>
__device__ __forceinline__ void sae_gemm_body(const SaeFilterArgs& a, const SaeDenseOut& d) {
  if (DENSE && d.chk) {
    uint32_t total = 0;
#pragma unroll
    for (int x = 0; x < kSegs; ++x) total += d.chk[x * kSegStride];
    if (total >= d.k_req && total <= d.M) return;  // filtered: the candidates suffice
  }
  // distinct arrays per stage, so that the compiler can tell the stage being
  // read from the one being filled
  __shared__ __align__(16) uint4 sA0[kSaeFGran], sA1[kSaeFGran], sB0[kSaeFGran], sB1[kSaeFGran];
  __shared__ uint2 s_slice[kStage];  // per wave kSaeSlice (accumulator bits, element id) pairs
  __shared__ uint32_t s_hist[kLogBins];
  __shared__ uint32_t s_wmax[kSaeBS / kWave];
  __shared__ __align__(16) float2 s_col[2][kSaeFBN];  // a tile's {threshold, bias}, by tile parity
  // the wave index is wave-uniform: read from lane 0 it is a scalar, and so
  // are the LDS bases derived from it
  const uint32_t b = blockIdx.x, tid = threadIdx.x, lane = tid & (kWave - 1);
  const uint32_t w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const uint32_t wm = w >> 1, wn = w & 1;
  const uint32_t seg = b & (kSegs - 1);
  const uint32_t tau = DENSE ? 0u : a.st->tau_key;
  if (!DENSE)
    for (uint32_t i = tid; i < kLogBins; i += kSaeBS) s_hist[i] = 0;  // complete before the first barrier
  uint32_t* const seg_counter = a.seg_cnt + seg * kSegStride;
  uint32_t* const seg_key = a.seg_key + static_cast<size_t>(seg) * a.seg_cap;
  uint32_t* const seg_idx = a.seg_idx + static_cast<size_t>(seg) * a.seg_cap;
  // the wave's slice: a tile's survivors as (accumulator bits, element id);
  // its last entry is a spare that takes every rank past the others
  uint2* const wslice = s_slice + w * kSaeSlice;
  constexpr uint32_t kHot = kSaeSlice - 1;
  uint32_t my_max = 0;
  const uint32_t nchunk = a.g.d_model / kSaeFK;
  const uint32_t B = a.g.B, dd = a.g.d_dict, dm = a.g.d_model;

  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  // Load q (of kSaeFQ) of an operand fills granules (kSaeFQ w + q) 64 + lane
  // of a stage; granule P holds row P / 8, segment (P % 8) ^ (row % 8), so
  // lane L loads row 32 w + 8 q + L / 8 of the tile, segment
  // (L % 8) ^ (L / 8 % 8): a wave-uniform row base plus a lane offset that is
  // the same for every load (the loads take a scalar base and a 32-bit
  // offset).
  const uint32_t loff = ((lane / 8) * dm + (((lane & 7) ^ ((lane >> 3) & 7)) * 8)) * 2;  // bytes
  // chunk kc of tile (m0, n0) into stage S.  In a tile that passes B or
  // d_dict, lanes of rows out of range write their granule instead: NaN for x
  // (such rows' accumulators are NaN and pass no compare), zero for W_enc
  // (such columns have a NaN threshold).
  auto issue = [&](auto S, uint32_t m0, uint32_t n0, uint32_t kc) {
    uint4* const A = decltype(S)::value == 0 ? sA0 : sA1;
    uint4* const W = decltype(S)::value == 0 ? sB0 : sB1;
    // a wave-uniform base (row, chunk) and the lane's byte offset
    const char* const xc = reinterpret_cast<const char*>(a.g.x) + static_cast<size_t>(kc) * kSaeFK * 2 + loff;
    const char* const wc = reinterpret_cast<const char*>(a.g.w) + static_cast<size_t>(kc) * kSaeFK * 2 + loff;
    const size_t rb = static_cast<size_t>(dm) * 2;  // bytes per row
#define SAE_SRC(base, row) reinterpret_cast<const uint16_t*>((base) + static_cast<size_t>(row) * rb)
    if (m0 + kSaeFBM <= B && n0 + kSaeFBN <= dd) {
#pragma unroll
      for (int q = 0; q < kSaeFQ; ++q)
        __builtin_amdgcn_global_load_lds(SAE_SRC(xc, m0 + 32 * w + 8 * q), A + (kSaeFQ * w + q) * kWave, 16, 0, 0);
#pragma unroll
      for (int q = 0; q < kSaeFQ; ++q)
        __builtin_amdgcn_global_load_lds(SAE_SRC(wc, n0 + 32 * w + 8 * q), W + (kSaeFQ * w + q) * kWave, 16, 0, 0);
    } else {
#pragma unroll
      for (int q = 0; q < kSaeFQ; ++q) {
        const uint32_t r = m0 + 32 * w + 8 * q;
        uint4* const slot = A + (kSaeFQ * w + q) * kWave;
        if (r + lane / 8 < B) __builtin_amdgcn_global_load_lds(SAE_SRC(xc, r), slot, 16, 0, 0);
        else slot[lane] = uint4{0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u, 0x7FC07FC0u};
      }
#pragma unroll
      for (int q = 0; q < kSaeFQ; ++q) {
        const uint32_t r = n0 + 32 * w + 8 * q;
        uint4* const slot = W + (kSaeFQ * w + q) * kWave;
        if (r + lane / 8 < dd) __builtin_amdgcn_global_load_lds(SAE_SRC(wc, r), slot, 16, 0, 0);
        else slot[lane] = uint4{0u, 0u, 0u, 0u};
      }
    }
#undef SAE_SRC
  };
  struct Frag {
    bf16x8 a[2], b[4];
  };
  auto rd = [&](auto S, uint32_t ks, Frag& f) {
    const uint4* const A = decltype(S)::value == 0 ? sA0 : sA1;
    const uint4* const W = decltype(S)::value == 0 ? sB0 : sB1;
    const uint32_t sg = 2 * ks + (lane >> 5);
#pragma unroll
    for (int i = 0; i < 2; ++i) f.a[i] = __builtin_bit_cast(bf16x8, A[sae_swz(wm * 64 + i * 32 + (lane & 31), sg)]);
#pragma unroll
    for (int j = 0; j < 4; ++j) f.b[j] = __builtin_bit_cast(bf16x8, W[sae_swz(wn * 128 + j * 32 + (lane & 31), sg)]);
  };
  f32x16 acc[2][4];
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  };

  // one survivor's log-bin count and maximum
  auto note = [&](uint32_t key) {
    atomicAdd(&s_hist[log_bin(key - tau)], 1u);
    my_max = max(my_max, key);
  };
  // the wave's n staged survivors to the segment (a wave's LDS operations
  // execute in program order, so the slice reads see its writes)
  // one survivor to the segment (lanes of `ok`; the whole wave calls it)
  auto append_direct = [&](bool ok, uint32_t key, uint32_t idx) {
    const uint64_t s = __ballot(ok);
    if (s == 0) return;
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(seg_counter, static_cast<uint32_t>(__popcll(s)));
    base = __builtin_amdgcn_readfirstlane(base);  // the whole wave is active here: lane 0's
    if (ok) {
      const uint32_t gp = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(s >> 32),
                                                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(s), base));
      note(key);
      if (gp < a.seg_cap) {
        seg_key[gp] = key;
        seg_idx[gp] = idx;
      }
    }
  };
  // key and flat index of element e = 32 (2 j + i) + ... (see epilogue) of a
  // lane, from its accumulator value and the tile's column table
  auto survivor = [&](float av, uint32_t e, uint32_t l, const float2* cols, uint32_t m0, uint32_t n0, uint32_t& key,
                      uint32_t& idx) {
    const uint32_t j = e >> 5, i = (e >> 4) & 1, v = e & 15;
    const uint32_t row = m0 + wm * 64 + i * 32 + 8 * (v / 4) + 4 * (l >> 5) + (v % 4);
    const uint32_t cl = wn * 128 + j * 32 + (l & 31);
    key = key_f32(__float_as_uint(sae_relu(av + cols[cl].y)));
    idx = row * dd + n0 + cl;
  };
  // A tile's slice is appended to the segment while the next tile's MFMAs
  // run: the position (one atomic per wave) is requested at that tile's
  // start and used after its first chunk, whose wait covers it.
  uint32_t pend = 0, pm0 = 0, pn0 = 0, ppar = 0;  // the slice's survivors and their tile
  uint32_t pbase = 0;                             // lane 0: the segment position for them
  auto request_pending = [&]() {
    if (!DENSE && pend && lane == 0) pbase = atomicAdd(seg_counter, pend);
  };
  auto flush_pending = [&]() {
    if (DENSE || pend == 0) return;
    const uint32_t base = __builtin_amdgcn_readfirstlane(pbase);  // the whole wave is active here
    for (uint32_t q = lane; q < pend; q += kWave) {
      const uint2 en = wslice[q];
      const uint32_t gp = base + q;
      uint32_t key, idx;
      survivor(__uint_as_float(en.x), en.y >> 6, en.y & 63, s_col[ppar], pm0, pn0, key, idx);
      note(key);
      if (gp < a.seg_cap) {
        seg_key[gp] = key;
        seg_idx[gp] = idx;
      }
    }
    pend = 0;
  };
  // the dense variant's epilogue: every latent of the tile that is in range
  auto write_dense = [&](uint32_t m0, uint32_t n0) {
    const uint32_t r0 = m0 + wm * 64 + 4 * (lane >> 5);
    const bool full = m0 + kSaeFBM <= B;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t c = n0 + sae_fcol(lane, w, j);
      if (c >= dd) continue;
      const float bias = a.g.bias[c];
      float* const o = d.out + static_cast<size_t>(r0) * dd + c;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t ro = i * 32 + 8 * (v / 4) + (v % 4);
          if (full || r0 + ro < B) o[static_cast<size_t>(ro) * dd] = sae_relu(acc[i][j][v] + bias);
        }
    }
  };
  // Epilogue of one tile.  Hot pass, straight-line: per element a compare,
  // a ballot, and the survivors' (accumulator bits, element id) written to
  // the wave's slice at their ranks (lanes without a survivor are masked
  // off).  The slice is converted and appended later (flush_pending).  A
  // tile whose survivors do not fit the slice is done again by the cold
  // pass, which appends each element's survivors to the segment directly.
  auto epilogue = [&](const float2* cols, uint32_t m0, uint32_t n0) {
    uint32_t fill = 0;  // survivors of the tile so far (may pass kHot)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float thr = cols[sae_fcol(lane, w, j)].x;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        // the ballots of 8 elements first, so that each branch finds its
        // mask computed
        uint64_t sm[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) sm[u] = __ballot(acc[g >> 1][j][(g & 1) * 8 + u] >= thr);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = g >> 1, v = (g & 1) * 8 + u;
          const uint32_t e = (2 * j + i) * 16 + v;
          const uint64_t s = sm[u];
          // most elements have no survivor: that case falls through
          if (__builtin_expect(s == 0, 1)) continue;
          const float av = acc[i][j][v];
          if (av >= thr) {
            // the empty asm keeps the id inside the branch: it does not
            // depend on the tile, and hoisted out of the tile loop for
            // every element it would hold 128 registers
            uint32_t ln = lane;
            asm volatile("" : "+v"(ln));
            const uint32_t pos = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(s >> 32),
                                                           __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(s), fill));
            wslice[min(pos, kHot)] = uint2{__float_as_uint(av), (e << 6) | ln};
          }
          fill += static_cast<uint32_t>(__popcll(s));
        }
      }
    }
    if (fill <= kHot) {
      pend = fill;  // appended during the next tile's first chunks (flush_pending)
      return;
    }
    // cold pass: every element again, straight to the segment
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float thr = cols[sae_fcol(lane, w, j)].x;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t e = (2 * j + i) * 16 + v;
          const float av = acc[i][j][v];
          const bool ok = av >= thr;
          uint32_t key = 0, idx = 0;
          if (ok) survivor(av, e, lane, cols, m0, n0, key, idx);
          append_direct(ok, key, idx);
        }
    }
  };

  const XcdTiles xt(a.tiles_m, a.tiles_n);
  auto tile_of = [&](uint32_t t, uint32_t& m0, uint32_t& n0) {
    m0 = (t / xt.nx) * kSaeFBM;
    n0 = (xt.nlo + t % xt.nx) * kSaeFBN;
  };
  Frag F0, F1;
  bool primed = false;  // the tile's chunk 0 is in stage 0, awaited behind a barrier
  uint32_t par = 0;     // parity of the tile in this workgroup's sequence
  for (uint32_t t = xt.first; t < xt.count; t += xt.stride, par ^= 1) {
    uint32_t m0, n0, nm0 = 0, nn0 = 0;
    tile_of(t, m0, n0);
    const bool has_next = t + xt.stride < xt.count;
    if (has_next) tile_of(t + xt.stride, nm0, nn0);
    // the tile's {threshold, bias} into s_col[par] (2 KB, wave 0).  A wait
    // and barrier of this tile before its epilogue cover it; its last
    // readers, two tiles back (the epilogue, and the slice's append in the
    // next tile) are behind a barrier: the one that ends chunk 1 of the tile
    // before this one when the tile is primed, else the prologue's first.
    auto load_cols = [&]() {
      if (!DENSE && w == 0) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
          __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4*>(a.col + n0) + q * kWave + lane,
                                           reinterpret_cast<uint4*>(s_col[par]) + q * kWave, 16, 0, 0);
      }
    };
    request_pending();
    if (!primed) {
      // this tile's first two chunks; a barrier first, after which no wave
      // still reads the stages (the previous tile's fragment reads)
      wait_loads_lds();
      __builtin_amdgcn_s_barrier();
      load_cols();
      issue(I0{}, m0, n0, 0);
      if (nchunk > 1) issue(I1{}, m0, n0, 1);
      // all loads (a masked-off load instruction is not counted)
      wait_loads_lds();
      __builtin_amdgcn_s_barrier();
    } else {
      load_cols();
    }
    rd(I0{}, 0, F0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
    const bool cross = CROSS && has_next;
    // chunk c in stage S, its first fragments in F0
    auto chunk = [&](auto S, uint32_t c) {
      constexpr int st = decltype(S)::value;
#pragma unroll
      for (int ks = 0; ks + 1 < kSaeFKS; ++ks) {
        if (ks % 2 == 0) rd(S, ks + 1, F1);
        else rd(S, ks + 1, F0);
        __builtin_amdgcn_sched_barrier(0);
        if (ks % 2 == 0) mma(F0);
        else mma(F1);
        __builtin_amdgcn_sched_barrier(0);
        // the previous tile's slice, while these MFMAs run: in chunk 1,
        // after the wait that ends chunk 0 (chunk 0 when there is no other)
        if (ks == 0 && c == (nchunk > 1 ? 1u : 0u)) flush_pending();
        __builtin_amdgcn_sched_barrier(0);
      }
      mma(F1);  // the last k-step (kSaeFKS is even)
      __builtin_amdgcn_sched_barrier(0);
      // the next chunk: c + 1 here, or chunk 0 of the next tile (CROSS)
      const bool here = c + 1 < nchunk;
      if (here || cross) {
        wait_loads_lds();
        __builtin_amdgcn_s_barrier();
        // stage st is free: the chunk after the next one
        if (c + 2 < nchunk) issue(S, m0, n0, c + 2);
        else if (cross && c + 2 - nchunk < nchunk) issue(S, nm0, nn0, c + 2 - nchunk);
        // the next tile's first fragments are read after the epilogue, so
        // that they do not hold registers through it
        if (here) rd(std::integral_constant<int, 1 - st>{}, 0, F0);
      }
    };
    for (uint32_t c = 0; c < nchunk; c += 2) {
      chunk(I0{}, c);
      if (c + 1 < nchunk) chunk(I1{}, c + 1);
    }
    primed = cross;
    if constexpr (DENSE) write_dense(m0, n0);
    else epilogue(s_col[par], m0, n0);
    pm0 = m0;
    pn0 = n0;
    ppar = par;
  }
  if constexpr (DENSE) return;
  request_pending();
  flush_pending();
  const uint32_t wmx = wave_max_u32(my_max);
  if (lane == 0) s_wmax[w] = wmx;
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

template <bool CROSS>
__global__ __launch_bounds__(kSaeBS) void k_sae_filter(SaeFilterArgs a) {
  sae_gemm_body<CROSS, false>(a, SaeDenseOut{});
}

template <bool CROSS>
__global__ __launch_bounds__(kSaeBS) void k_sae_dense(SaeFilterArgs a, SaeDenseOut d) {
  sae_gemm_body<CROSS, true>(a, d);
}

// ------------------------------------------------------------- dense ------

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
  S.G = sae_grid(cdiv_s(B, kSaeFBM) * cdiv_s(d_dict, kSaeFBN));
  if (S.G > S.flat.G_f) S.G = S.flat.G_f >= kXcds ? S.flat.G_f / kXcds * kXcds : S.flat.G_f;  // blk_max: G_f entries
  const uint32_t Sn = static_cast<uint32_t>(plan.S);
  S.off_skeys = (S.flat.bytes + 255) & ~static_cast<size_t>(255);
  S.off_thr = (S.off_skeys + static_cast<size_t>(Sn) * 4 + 255) & ~static_cast<size_t>(255);
  S.off_dense = (S.off_thr + static_cast<size_t>(cdiv_s(d_dict, kSaeFBN)) * kSaeFBN * 8 + 255) & ~static_cast<size_t>(255);
  S.bytes = S.off_dense + static_cast<size_t>(B) * d_dict * 4;
  return S;
}

static SaeGemm gemm_of(const SaeCall& c) {
  return SaeGemm{static_cast<const uint16_t*>(c.x), static_cast<const uint16_t*>(c.w), c.bias, c.B, c.d_model,
                 c.d_dict};
}

// Filter-tile arguments for the dense variant: only the GEMM and the tiles.
static SaeFilterArgs dense_args(const SaeCall& c) {
  SaeFilterArgs fa{};
  fa.g = gemm_of(c);
  fa.tiles_m = cdiv_s(c.B, kSaeFBM);
  fa.tiles_n = cdiv_s(c.d_dict, kSaeFBN);
  return fa;
}

// The dense variant on the filter's tiles; chk as in SaeDenseOut.
static void launch_dense_tiles(const SaeCall& c, float* out, const uint32_t* chk, uint32_t k_req, uint32_t M) {
  const SaeFilterArgs fa = dense_args(c);
  const SaeDenseOut d{out, chk, k_req, M};
  const dim3 grid(sae_grid(fa.tiles_m * fa.tiles_n));
  if ((c.d_model / kSaeFK) % 2 == 0) hipLaunchKernelGGL(k_sae_dense<true>, grid, dim3(kSaeBS), 0, c.stream, fa, d);
  else hipLaunchKernelGGL(k_sae_dense<false>, grid, dim3(kSaeBS), 0, c.stream, fa, d);
}

hipError_t launch_sae_dense(const SaeCall& c, float* out) {
  (void)hipGetLastError();
  launch_dense_tiles(c, out, nullptr, 0, 0);
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
  const SaeGemm g = gemm_of(c);
  hipError_t e = launch_sae_sample(c);
  if (e != hipSuccess) return e;
  // tau: the t-th largest of the S sampled keys (per-block top-t lists in
  // the vector path's union space, then one block)
  if ((e = launch_select_tau_keys(reinterpret_cast<const uint32_t*>(ws + c.L.off_skeys), static_cast<uint32_t>(p.S),
                                  static_cast<uint32_t>(p.t), reinterpret_cast<uint32_t*>(ws + L.off_union),
                                  static_cast<size_t>(L.G_s) * L.tcap, st, c.stream)) != hipSuccess)
    return e;
  float2* col = reinterpret_cast<float2*>(ws + c.L.off_thr);
  const uint32_t d_pad = cdiv_s(c.d_dict, kSaeFBN) * kSaeFBN;
  hipLaunchKernelGGL(k_sae_thresholds, dim3(d_pad / 256), dim3(256), 0, c.stream, st, c.bias, c.d_dict, d_pad, col);
  const uint32_t ftm = cdiv_s(c.B, kSaeFBM), ftn = cdiv_s(c.d_dict, kSaeFBN);
  SaeFilterArgs fa{g, ftm, ftn, st, L.seg_cap, seg_cnt,
                   reinterpret_cast<uint32_t*>(ws + L.off_seg_key), reinterpret_cast<uint32_t*>(ws + L.off_seg_idx),
                   reinterpret_cast<uint32_t*>(ws + L.off_blk_max), fhist, col};
  if (c.ev_before) (void)hipEventRecord(c.ev_before, c.stream);
  // the next tile's loads overlap the epilogue when the chunks of a tile
  // are even in number (chunk c is then in stage c % 2 in every tile)
  if ((c.d_model / kSaeFK) % 2 == 0) hipLaunchKernelGGL(k_sae_filter<true>, dim3(c.L.G), dim3(kSaeBS), 0, c.stream, fa);
  else hipLaunchKernelGGL(k_sae_filter<false>, dim3(c.L.G), dim3(kSaeBS), 0, c.stream, fa);
  if (c.ev_after) (void)hipEventRecord(c.ev_after, c.stream);
  // the dense latents only when the candidates do not suffice (exact fallback)
  launch_dense_tiles(c, dense, seg_cnt, static_cast<uint32_t>(p.k_req), static_cast<uint32_t>(p.M));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_refine(fc, c.L.G);
}

hipError_t launch_sae_sample(const SaeCall& c) {
  (void)hipGetLastError();
  const FlatLayout& L = c.L.flat;
  uint32_t* skeys = c.sample_keys ? c.sample_keys : reinterpret_cast<uint32_t*>(c.ws + c.L.off_skeys);
  const uint32_t S = static_cast<uint32_t>(c.plan->S);
  SaeSampleArgs sa{gemm_of(c), c.seed, S, skeys, reinterpret_cast<CallState*>(c.ws + L.off_state),
                   reinterpret_cast<uint32_t*>(c.ws + L.off_segcnt), reinterpret_cast<uint32_t*>(c.ws + L.off_fhist),
                   L.big ? reinterpret_cast<uint32_t*>(c.ws + L.off_bcur) : nullptr,
                   L.big ? reinterpret_cast<uint32_t*>(c.ws + L.off_ghist) : nullptr};
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
