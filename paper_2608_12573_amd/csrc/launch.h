// Host view of the kernels: workspace layout and launch entry points.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "profk.h"

namespace profk {

// Per-call device state at the start of a workspace (256 bytes).
struct CallState {
  uint32_t tau_key;    // threshold key (stage 2)
  uint32_t ticket;     // last-block-done counter of the fallback
  uint32_t status;     // PROFK_STATUS_* of the call
  uint32_t tau_idx;    // lexicographic plans: index of the threshold pair
  uint32_t tie_above;  // draws above tau (k_tau_index)
  uint32_t tie_n;      // draws equal to tau, listed in the workspace
  uint32_t tie_ticket; // last-block-done counter of k_tau_index
  uint32_t grp_ticket[16];  // last-block-done counters of the fallback's chunk groups
  uint32_t big_ticket;  // last-block-done counter of the large-k radix digit passes
  uint32_t pad[40];
};
static_assert(sizeof(CallState) == 256, "call state size");

// Launch geometry.
constexpr uint32_t kXcds = 8;                 // MI355X: 8 XCDs of 32 CUs, each with its own L2
constexpr int kSampBS = 256;                  // threads of a sample block
constexpr int kSampPerBlock = 4 * kSampBS;    // draws per sample block
// Sample blocks of plans with t > kWaveTopMax (key rule): 1024 threads and
// 4096 draws, so that the union of the blocks' top-t lists, which one
// workgroup selects tau from, is four times smaller.
constexpr int kSampWideBS = 1024;
constexpr uint32_t kWaveTopMax = 32;          // largest t of the wave-level top-t
// Capped sample lists (key rule, t > kWaveTopMax): when the draws of one
// 1024-draw block that lie in the sample's top t are few (mean mu = 1024 t /
// S), each block keeps only its top c (c = 16 or 32, at least mu + 8
// sqrt(mu) + 2) and its c-th largest key, and the blocks store every key.
// The t-th largest of the union of the lists is the sample's t-th largest
// whenever no block that dropped keys has its c-th key at or above it;
// otherwise tau is selected again from all S keys.
constexpr uint32_t kCapListSmall = 16;
constexpr int kTauBS = 1024;
constexpr int kFiltBS = 256;                  // threads of a filter block
// 16-byte loads in flight per lane of a filter step: 4 for inputs of at
// least kFiltSparseMinBytes, 8 for smaller ones.  Measured on one MI355X:
// 4 loads streamed the 1 GiB inputs 1-3 % faster than 8 (N = 2^28: 161.8
// against 163.4 us; the BatchTopK shape: 170.6 against 175.2 us), and the
// 256 MiB inputs about 4 % slower; 2, 12 and 16 were slower everywhere.
constexpr int kFiltULarge = 4;
constexpr int kFiltUSmall = 8;
constexpr int kFiltMaxBlocks = 1024;
// Filter blocks per CU.  A large input whose survivors are rare streams
// fastest with two (fewer concurrent streams: about 5 % on a GiB, and a
// plain read kernel shows the same); where survivors are common, or the
// input is smaller, four hide the survivor work better.
constexpr int kFiltPerCuSparse = 2;
constexpr int kFiltPerCuDense = 4;
constexpr uint64_t kFiltSparseMinBytes = 512ull << 20;  // "large"
constexpr uint64_t kFiltSparseInvDensity = 4096;        // "rare": t/(S+1) below 1/4096
constexpr uint32_t kFiltTauMax = 2048;        // largest sample union a filter block selects from
constexpr uint32_t kFiltTauWave = 4;          // union keys per lane when one wave selects tau
constexpr uint32_t kFiltTauInMaxT = 32;       // largest t the filter blocks select tau for themselves
static_assert(kFiltTauInMaxT <= kWaveTopMax, "the filter selects tau with the wave-level top-t");
constexpr uint32_t kStage = 1024;             // survivors a filter block stages in LDS
constexpr int kSegs = 8;                      // candidate segments (one counter each)
constexpr int kSegStride = 64;                // words between segment counters
constexpr int kFinBS = 1024;
constexpr int kFinMaxK = 4096;                // largest k of the one-block refinement
constexpr int kFbMaxBlocks = 256;
constexpr int kFbGroup = 16;                  // fallback chunks merged together first
static_assert(kFbMaxBlocks / kFbGroup <= 16, "group counters in CallState");
constexpr uint32_t kFastCap = 8192;           // candidates the bucket refinement holds in LDS
// It ranks each candidate within its bucket by comparison: sum over the
// buckets at or above rank k of size^2 comparisons in all, at most this many.
constexpr uint32_t kFastCost = 1u << 23;
constexpr uint32_t kFastBucket = 128;         // the per-row kernel: largest bucket it ranks by comparison
constexpr uint32_t kFbMinChunk = 8192;

// Multi-block refinement for k > kFinMaxK.
constexpr int kBigBS = 256;
constexpr int kBigDigit = 11;
constexpr uint32_t kBigBins = 1u << kBigDigit;
constexpr int kBigStage = 4096;               // composites a collect block stages in LDS
constexpr uint32_t kBigTile = 4096;           // composites a merge block writes
constexpr uint32_t kBigSortTile = 16384;      // composites sorted per block before the merges
constexpr int kBigMaxBlocks = 256;
constexpr uint32_t kBktCap = 4096;            // largest bucket one sort block holds
constexpr uint32_t kBktPad = 32;              // words between bucket fill counters (own 128-byte line)
constexpr int kBktSortBlocks = 512;           // bucket-sort grid (loops over the bucket list)

// Workspace layout of one flat (vector) call.
struct FlatLayout {
  uint32_t G_s = 0, tcap = 0, union_n = 0;    // sampling
  uint32_t samp_bs = 0;                       // threads of a sample block (four draws each)
  uint32_t cap_list = 0;                      // capped sample lists: their length, else 0
  size_t off_cut = 0, off_all_keys = 0;       // capped lists: each block's cut key, every sample key
  uint32_t G_f = 0;                           // filter blocks
  int filt_u = 0;                             // 16-byte loads per lane and filter step
  bool filt_db = true;                        // filter steps double-buffered (all but the sparse launch)
  uint32_t seg_cap = 0;                       // entries per candidate segment (= M)
  uint32_t G_fb = 0;                          // fallback blocks (at most)
  size_t off_state = 0, off_segcnt = 0, off_union = 0, off_blk_max = 0;
  size_t off_seg_key = 0, off_seg_idx = 0;
  size_t off_cand_key = 0, off_cand_idx = 0, off_grp_key = 0, off_grp_idx = 0;
  size_t off_fhist = 0;                       // log-bin histogram of the candidates
  size_t off_tie = 0;                         // lexicographic plans: indices of the draws equal to tau
  bool big = false;                           // k > kFinMaxK: multi-block refinement
  uint32_t G_big = 0;
  size_t off_big_state = 0, off_ghist = 0, off_staging = 0, off_runs = 0;
  size_t off_bcur = 0;                        // bucket fill counts
  size_t off_blist = 0;                       // non-empty buckets at or above b*: 16 bytes each
  size_t bytes = 0;
};

FlatLayout flat_layout(const profk_plan_t& plan, int dtype, int num_cus);

struct FlatCall {
  const profk_plan_t* plan;
  int dtype;
  const void* values;
  uint32_t n, k;
  uint64_t seed;
  uint64_t row;
  void* out_vals;
  int64_t* out_idx;
  uint8_t* ws;
  FlatLayout L;
  hipStream_t stream;
  profk_info_t* info;
  int use_tau;          // 1: threshold given by the caller
  uint32_t tau_key;
  hipEvent_t ev_before = nullptr, ev_after = nullptr;  // around the filter launch
};

hipError_t launch_flat(const FlatCall& c);
// The filter pass of c into the workspace's candidate segments; tau from
// the sample union when union_keys is given, else from st.
hipError_t launch_filter(const FlatCall& c, CallState* st, const uint32_t* union_keys, bool lex);
// Filter workgroups one CU holds at once, at most `want`.
int filter_blocks_per_cu(int dtype, int want);
// Refinement of the candidates a filter left in c.ws by G_f workgroups
// (the fallback reads c.values), and tau from a stage-1 union into st.
hipError_t launch_refine(const FlatCall& c, uint32_t G_f);
hipError_t launch_select_tau(const uint32_t* union_keys, uint32_t n, uint32_t t, int keybits, CallState* st,
                             hipStream_t s);
// tau over n 32-bit keys in memory: per-block top-t lists into union_keys
// (union_words long) first when that shrinks the set, then one block.
hipError_t launch_select_tau_keys(const uint32_t* keys, uint32_t n, uint32_t t, uint32_t* union_keys,
                                  size_t union_words, CallState* st, hipStream_t s);

struct BigCall {
  int dtype;
  const void* values;
  uint32_t n, k, k_req, M;
  int direct;
  const uint32_t *seg_cnt, *seg_key, *seg_idx, *blk_max;
  uint32_t seg_cap, G_f;
  CallState* st;
  void* big_state;
  uint32_t* ghist;
  uint64_t *staging, *runs;
  const uint32_t* fhist;
  uint32_t *bcur, *blist;
  uint32_t G_big;
  void* out_vals;
  int64_t* out_idx;
  profk_info_t* info;
  hipStream_t stream;
};

hipError_t launch_big(const BigCall& c);

// Per-row kernel: one workgroup per row, everything in LDS.
constexpr int kRowBS = 256;                   // threads of a row block
constexpr int kRowU = 8;                      // 16-byte loads in flight per lane
constexpr int kRowMaxK = 4 * kRowBS;          // largest k per row
constexpr uint32_t kRowMaxLds = 144 * 1024;   // dynamic LDS the row layout may use

// Dynamic LDS of a row block: region a holds the sample keys and then the
// buffer keys (and, last, the sort exchange), region b the buffer indices.
struct RowLayout {
  uint32_t off_a = 0, off_b = 0, off_hist = 0, off_collect = 0, off_comp = 0, bytes = 0;
};

RowLayout row_layout(const profk_plan_t& plan, int dtype);

struct RowCall {
  const profk_plan_t* plan;
  int dtype;
  const void* values;
  uint32_t B, D, k;
  uint64_t row_stride;
  uint64_t seed;
  void* out_vals;
  int64_t* out_idx;
  profk_info_t* info;
  RowLayout L;
  hipStream_t stream;
};

hipError_t launch_rows(const RowCall& c);

// BatchTopK SAE encoder with the filter in its GEMM epilogue.  The
// workspace is the vector path's (same plan) followed by a dense fp32
// [B, d_dict] latent buffer that only the exact fallback writes.
struct SaeLayout {
  FlatLayout flat;
  uint32_t G = 0;                                 // filter workgroups (persistent)
  size_t off_skeys = 0;                           // every draw's latent key (S words)
  size_t off_thr = 0;                             // per-column {threshold, bias}, padded to whole filter tiles
  size_t off_dense = 0, bytes = 0;
};

SaeLayout sae_layout(const profk_plan_t& plan, uint32_t B, uint32_t d_dict, int num_cus);

struct SaeCall {
  const profk_plan_t* plan;
  const void* x;     // bf16 [B, d_model]
  const void* w;     // bf16 [d_dict, d_model]
  const float* bias; // [d_dict]
  uint32_t B, d_model, d_dict, K;
  uint64_t seed;
  float* out_vals;
  int64_t* out_idx;
  uint8_t* ws;
  SaeLayout L;
  hipStream_t stream;
  profk_info_t* info;
  uint32_t* sample_keys;  // optional: the S sampled latents' keys
  hipEvent_t ev_before = nullptr, ev_after = nullptr;  // around the fused filter launch
};

hipError_t launch_sae_topk(const SaeCall& c);
hipError_t launch_sae_sample(const SaeCall& c);  // stage 1 only, with c.sample_keys
hipError_t launch_sae_dense(const SaeCall& c, float* out);

struct SaeDecodeCall {
  const float* vals;
  const int64_t* idx;
  uint32_t K, B, d_model, d_dict;
  const void* w;      // bf16 [d_dict, d_model]
  const float* bias;  // [d_model]
  float* out;         // [B, d_model]
  void* ws;
  hipStream_t stream;
};

size_t sae_decode_workspace(uint32_t B, uint32_t K);
uint32_t sae_decode_max_dict();
hipError_t launch_sae_decode(const SaeDecodeCall& c);

// Inspection helpers.
hipError_t launch_sample_indices(uint64_t seed, uint64_t row, uint32_t S, uint64_t N,
                                 int64_t* out, hipStream_t s);
hipError_t launch_debug_filter(const FlatCall& c, uint32_t* buf_key, uint32_t* buf_idx,
                               uint32_t* count_dev);

// Read-only stream probe: XOR fold of nvec 16-byte vectors, one word per
// workgroup into out (kFiltMaxBlocks words at most); *grid_out = workgroups.
hipError_t launch_read_probe(const void* values, uint64_t nvec, int blocks_per_cu, int loads_per_lane,
                             uint32_t* out, uint32_t* grid_out, hipStream_t s);

int device_cu_count();

}  // namespace profk
