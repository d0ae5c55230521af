/*
 * profk.h -- C ABI of libprofk.so, Prof-K top-k selection on MI355X (gfx950).
 *
 * Prof-K (Sec. 3, "The Prof-K Algorithm") selects the k largest of N values
 * in four stages: draw a uniform sample of S indices, take the t-th largest
 * sampled value as a threshold tau, stream the input once keeping every
 * x_i >= tau in a buffer of capacity M, and finish with an exact top-k of
 * the buffer -- or of the whole input when fewer than k candidates survived
 * or more than M did.  The result is therefore always exact.
 *
 * Conventions shared by every entry point
 *   Total order.  Elements are ranked by an order-preserving integer key of
 *     their bit pattern (negatives: all bits flipped; non-negatives: sign bit
 *     set), larger key first, smaller index first among equal keys.  So
 *     -0.0 ranks below +0.0, +NaN above +inf, -NaN below -inf.  Outputs are
 *     sorted in this order; values are bit copies of the inputs.
 *   Memory.  `values`, outputs, `ws` and `info_dev` are device pointers owned
 *     by the caller.  The library neither frees nor retains them.  `values`
 *     may have any 2-byte (bf16) or 4-byte (fp32) alignment.
 *   Streams.  `stream` is a hipStream_t passed as void* (NULL = the null
 *     stream).  Every call only enqueues work on it and returns without
 *     synchronising, except profk_topk_simple.  `info_dev` is valid once the
 *     caller has synchronised the stream.
 *   Errors.  Return 0 on success or a negative PROFK_E* code.  A fallback to
 *     the exact path is not an error: it is reported in profk_info_t.status.
 *     All calls are reentrant; calls that share a workspace must not overlap.
 *   Limits.  1 <= k <= N <= 2^32 - 1; dtypes fp32 and bf16.
 */
#ifndef PROFK_H
#define PROFK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PROFK_F32 = 0, PROFK_BF16 = 1 } profk_dtype;

enum {
  PROFK_OK = 0,
  PROFK_EINVAL = -1,     /* bad size, k, eps, recall, or plan/argument mismatch */
  PROFK_EDTYPE = -2,     /* dtype is neither PROFK_F32 nor PROFK_BF16 */
  PROFK_EWORKSPACE = -3, /* ws_bytes smaller than profk_workspace_size() */
  PROFK_ENULL = -4,      /* a required pointer is NULL */
  PROFK_EHIP = -5        /* a HIP call failed; see profk_last_hip_error() */
};

enum { PROFK_MODE_FILTER = 0, PROFK_MODE_DIRECT = 1 };
enum { PROFK_FORCE_AUTO = 0, PROFK_FORCE_FILTER = 1, PROFK_FORCE_DIRECT = 2 };

enum {
  PROFK_STATUS_FILTERED = 0,  /* k_req <= count <= M: refined from the buffer */
  PROFK_STATUS_UNDERFLOW = 1, /* count < k_req: exact fallback on the input */
  PROFK_STATUS_OVERFLOW = 2,  /* count > M: exact fallback on the input */
  PROFK_STATUS_DIRECT = 3     /* plan chose the exact path; no sampling */
};

/* Planner options.  Pass NULL for the defaults of profk_default_opts(). */
typedef struct {
  int32_t S_min;        /* lower clamp of S (Sec. 4, "Optimal Sample Size"): 32768 */
  int32_t S_max;        /* upper clamp of S: 131072 */
  double cost_ratio;    /* tau_B / tau_A of the cost model, eq. (cost_model): 1.0 */
  double eps_split;     /* eps_A = eps_split * eps, eps_B = the rest (Theorem 1): 0.5 */
  int32_t paper_literal;/* 1: t and M from Algorithm 1 verbatim (reporting only) */
  int32_t force_mode;   /* PROFK_FORCE_*: override the FILTER/DIRECT choice */
  int32_t lexicographic;/* 1: tie-exact filter on (key, -index) pairs; 0: key >= tau
                         * as in Sec. 3 (default).  Copied into the plan. */
} profk_plan_opts_t;

/* A plan: (S, t, M) for one (N, k, eps, recall). */
typedef struct {
  int64_t N, k;
  double eps, recall;
  int64_t k_req;        /* ceil(recall * k): the recall target of the filter */
  int64_t S;            /* sample size, Algorithm 1 */
  int64_t t;            /* threshold rank within the sample, 1-based */
  int64_t M;            /* buffer capacity */
  int32_t mode;         /* PROFK_MODE_* */
  int32_t lexicographic;/* 1: the threshold is the t-th largest sampled (key, -index)
                         * pair (tau, -i_tau) and element i survives iff key > tau, or
                         * key == tau and i <= i_tau.  Pairs never tie, so count is the
                         * exact rank of the threshold and the eps bound of Theorem 1
                         * holds for inputs with repeated values too (with key >= tau
                         * it holds for distinct values).  The result is the same exact
                         * top-k either way.  0: the paper's key >= tau. */
  double p_underflow;   /* Pr(count < k_req) = Pr(Bin(S, (k_req-1)/N) >= t) */
  double p_overflow;    /* Pr(count > M)     = Pr(Bin(S, M/N) <= t-1) */
} profk_plan_t;

/* Per-call report, written on the device. */
typedef struct {
  uint64_t count;       /* survivors of the filter, counted exactly (0 in DIRECT) */
  uint32_t tau_key;     /* key of the threshold (0 in DIRECT) */
  int32_t status;       /* PROFK_STATUS_* */
  int64_t n_valid;      /* valid outputs: k, or fewer in relaxed-recall mode */
} profk_info_t;

/* Fill `opts` with the defaults for a flat vector (S_min 32768, S_max 2^17,
 * cost ratio 1, even eps split; Sec. 4 "Optimal Sample Size", Theorem 1). */
void profk_default_opts(profk_plan_opts_t* opts);

/* Defaults for one row of a batch: as above with S_min = 256, because a
 * 32768-draw floor oversamples rows of ~10^5 elements, and cost ratio 0.5,
 * the measured tau_B / tau_A of the per-row kernel on MI355X (Sec. 4,
 * "Optimal Sample Size", leaves the ratio to a benchmark of the hardware). */
void profk_default_row_opts(profk_plan_opts_t* opts);

/* Defaults for profk_sae_encode_topk plans (N = B * d_dict, k = B * k_row):
 * the flat defaults with cost ratio 1/64.  A draw of the fused SAE path is
 * a d_model-long dot product on the matrix cores (two row reads), far
 * dearer than the flat path's one gathered element, so Algorithm 1's S*
 * falls to S_min; the measured fused step at the paper's shape (B = 4096,
 * d_model = 512, d_dict = 12288, k = 32) is fastest there (Sec. 4,
 * "Optimal Sample Size", leaves the ratio to a benchmark of the hardware). */
void profk_default_sae_opts(profk_plan_opts_t* opts);

/* Parameter selection, host only, pure and thread-safe (Algorithm 1 for S;
 * t and M as the smallest integers whose exact binomial failure tails stay
 * within eps_A and eps_B -- the design goal of Sec. 3 and Theorem 1).
 * Errors: PROFK_ENULL if out is NULL; PROFK_EINVAL unless 1 <= k <= N <
 * 2^32, 0 < eps < 1, 0 < recall <= 1 and the opts are sane. */
int profk_plan(int64_t N, int64_t k, double eps, double recall,
               const profk_plan_opts_t* opts, profk_plan_t* out);

/* profk_plan with N = D and the row defaults when opts is NULL. */
int profk_plan_rows(int64_t D, int64_t k, double eps, double recall,
                    const profk_plan_opts_t* opts, profk_plan_t* out);

/* Device workspace in bytes for `batch` independent vectors under `plan`
 * (batch = 1 for profk_topk and profk_batchtopk, B for profk_topk_rows).
 * It holds the sample keys, the candidate buffer, counters and the scratch
 * of the exact fallback: O(S + M + k) bytes per vector, never O(N).  For
 * profk_topk_rows it is a token 256 bytes when the row plan fits the
 * one-workgroup row kernel, else one row's vector workspace.
 * Returns 0 when the plan or dtype is invalid. */
size_t profk_workspace_size(const profk_plan_t* plan, int32_t dtype, int64_t batch);

/* Top-k of one vector (Sec. 3).  values[N] of `dtype`; out_vals[k] (same
 * dtype), out_idx[k] int64 in [0, N).  `plan` must come from profk_plan with
 * the same N and k.  In relaxed-recall plans (recall < 1) entries past
 * info.n_valid hold index -1 and value -inf.  info_dev may be NULL. */
int profk_topk(const profk_plan_t* plan, int32_t dtype, const void* values,
               int64_t N, int64_t k, uint64_t seed, void* out_vals,
               int64_t* out_idx, void* ws, size_t ws_bytes, void* stream,
               profk_info_t* info_dev);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * profk_topk with the workspace taken from a fixed device array of
 * PROFK_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on,
 * until the process ends.  The call allocates nothing and frees nothing; the
 * caller still provides values, out_vals, out_idx and (optionally) info_dev
 * on the current device, and `stream` must belong to that device.
 *   Limit: profk_workspace_size(plan, dtype, 1) <= PROFK_NOALLOC_SCRATCH_BYTES
 *     (16 MiB: every k <= 4096 for N <= 2^28), else PROFK_EWORKSPACE and
 *     nothing is enqueued.
 *   Sharing: every call on one GPU uses that GPU's one array, and each call
 *     initialises the parts it reads, so consecutive calls on one stream are
 *     safe; calls that overlap on one GPU (other streams, other threads
 *     without ordering) race on the array and give wrong results.
 *   Other arguments, results and errors as profk_topk; a failed lookup of
 *     the array's device address returns PROFK_EHIP. */
#define PROFK_NOALLOC_SCRATCH_BYTES (16u << 20)
int profk_topk_noalloc(const profk_plan_t* plan, int32_t dtype, const void* values,
                       int64_t N, int64_t k, uint64_t seed, void* out_vals,
                       int64_t* out_idx, void* stream, profk_info_t* info_dev);

/* The short form: fp32, eps = 1e-6, recall 1, the null stream, a workspace
 * held by the library (released by profk_release), synchronous. */
int profk_topk_simple(const float* values, int64_t N, int64_t k, uint64_t seed,
                      float* out_vals, int64_t* out_idx);

/* Per-row top-k of a [B, D] matrix whose rows start row_stride elements
 * apart (Sec. 3: the procedure is applied to each batch element).  Row r
 * draws its own sample (Philox counter word 1 = r) and falls back on its
 * own.  out_vals[B, k] and out_idx[B, k] (column indices) are contiguous.
 * `row_plan` comes from profk_plan_rows(D, k, ...).  info_dev is NULL or an
 * array of B reports.
 *   Plans with k <= 1024 whose sample and buffer fit one workgroup's LDS
 *   (4*max(S, M) + 4*M + 16*k bytes plus about 14 KiB, within 144 KiB) run
 *   one workgroup per row entirely in LDS; `ws` is then not used (NULL, 0
 *   are accepted).  Any other plan (wider rows, larger k) runs the vector
 *   path of profk_topk on each row in turn, on `stream`, with the same
 *   per-row sample stream and result; `ws` must then hold
 *   profk_workspace_size(row_plan, dtype, B) bytes (one row's workspace,
 *   reused by every row), else PROFK_ENULL or PROFK_EWORKSPACE. */
int profk_topk_rows(const profk_plan_t* row_plan, int32_t dtype,
                    const void* values, int64_t B, int64_t D,
                    int64_t row_stride, int64_t k, uint64_t seed,
                    void* out_vals, int64_t* out_idx, void* ws,
                    size_t ws_bytes, void* stream, profk_info_t* info_dev);

/* BatchTopK (Sec. 5, BatchTopK SAEs): a contiguous [B, D] matrix is read as
 * one vector of N = B*D and its K = B*k_row largest entries are selected.
 * `plan` comes from profk_plan(B*D, B*k_row, eps, recall).  out_vals[K],
 * out_flat_idx[K] = row*D + col.  With recall < 1 the call may return
 * info.n_valid < K entries (the exact top-n_valid), padded as in
 * profk_topk. */
int profk_batchtopk(const profk_plan_t* plan, int32_t dtype, const void* values,
                    int64_t B, int64_t D, int64_t k_row, uint64_t seed,
                    void* out_vals, int64_t* out_flat_idx, void* ws,
                    size_t ws_bytes, void* stream, profk_info_t* info_dev);

/* ---- Inspection entry points (used by the test suite) ------------------ */

/* Stage 1 alone: the S sample indices of row `row` (Philox4x64-10, key
 * (seed, 0), counter (j/4, row, 0, 0), word j%4, index = floor(u*N/2^64)).
 * out_dev: S int64 on the device. */
int profk_debug_sample_indices(uint64_t seed, int64_t row, int64_t S, int64_t N,
                               int64_t* out_dev, void* stream);

/* Stage 3 alone with a caller-given threshold key: the keys and indices of
 * every i with key(values[i]) >= tau_key, gathered into buf_key/buf_idx
 * (capacity plan->M; the first min(count, M) entries are written, in
 * unspecified order), and *count_dev = the exact number of survivors.
 * `plan` (from profk_plan for this N) sizes the buffer and `ws`, which must
 * hold profk_workspace_size(plan, dtype, 1) bytes.  count_dev: one uint32
 * on the device. */
int profk_debug_filter(const profk_plan_t* plan, int32_t dtype,
                       const void* values, int64_t N, uint32_t tau_key,
                       uint32_t* buf_key, uint32_t* buf_idx,
                       uint32_t* count_dev, void* ws, size_t ws_bytes,
                       void* stream);

/* A read-only stream over `bytes` bytes of device memory (a multiple of 16,
 * 16-byte aligned), with the filter pass's access pattern: a persistent grid
 * of blocks_per_cu (1..8) workgroups per compute unit, at most 1024, taking
 * tiles of 16-byte vectors in turn, each lane with loads_per_lane (4 or 8)
 * nontemporal loads in flight.  Nothing is compared or written but one word
 * per workgroup: out_dev[w] = the XOR of every 32-bit word workgroup w read
 * (so the XOR over out_dev[0 .. *grid) is the XOR of the whole buffer).
 * out_dev: 1024 uint32 on the device; *grid (host) receives the number of
 * workgroups launched.  bytes / 16 <= 2^32 - 2^22 - 1, else PROFK_EINVAL.  Measurement tools time it as the practical read
 * ceiling of the filter pass (Sec. 3, stage "Filtering", a single streaming
 * pass over the input). */
int profk_debug_read_probe(const void* values, uint64_t bytes, int32_t blocks_per_cu,
                           int32_t loads_per_lane, uint32_t* out_dev, uint32_t* grid,
                           void* stream);

/* ---- BatchTopK SAE layer (Sec. 5, "Application: BatchTopK Sparse
 * Autoencoders"; the encoder and decoder are those of the BatchTopK SAE the
 * paper builds on) ----
 *
 * Latents z[b, j] = max(sum_m x[b, m] W_enc[j, m] + b_enc[j], +0.0): bf16
 * inputs, fp32 sums (MFMA: each 16-product step and its accumulator are
 * rounded once), fp32 bias; a non-positive or NaN pre-activation gives +0.0.
 *
 * profk_sae_encode_topk selects the K = B*k_row largest latents of the
 * flattened [B, d_dict] matrix (flat index b*d_dict + j) with Prof-K inside
 * the encoder GEMM: the S sampled latents are computed with the GEMM's own
 * MFMA sequence (bit-identical values), and the filter runs in the GEMM's
 * epilogue, so the latent matrix is never written to memory -- except by
 * the exact fallback, which writes it to `ws` and selects from it.  The
 * result is the exact top-K of the latents under the total order (value
 * descending, then index ascending), sorted, as profk_batchtopk's.
 *   plan   profk_plan(B*d_dict, B*k_row, eps, recall), key rule only
 *          (lexicographic plans: PROFK_EINVAL).
 *   x      bf16 [B, d_model] row-major, 16-byte aligned; d_model a multiple
 *          of 64 (at most 65536).
 *   w_enc  bf16 [d_dict, d_model] row-major (one row per latent), 16-byte
 *          aligned.  b_enc: fp32 [d_dict].
 *   out_vals fp32 [K], out_flat_idx int64 [K]; relaxed recall pads as
 *          profk_topk does.  ws: profk_sae_workspace_size(plan, B, d_dict)
 *          bytes (the vector path's workspace plus 4*B*d_dict bytes for the
 *          fallback's latent matrix).
 * Errors as profk_topk; B*d_dict < 2^32. */
size_t profk_sae_workspace_size(const profk_plan_t* plan, int64_t B, int64_t d_dict);
int profk_sae_encode_topk(const profk_plan_t* plan, const void* x, const void* w_enc,
                          const float* b_enc, int64_t B, int64_t d_model, int64_t d_dict,
                          int64_t k_row, uint64_t seed, float* out_vals, int64_t* out_flat_idx,
                          void* ws, size_t ws_bytes, void* stream, profk_info_t* info_dev);

/* The latent matrix itself, out = fp32 [B, d_dict] (the same values the
 * fused path filters).  Same argument rules as profk_sae_encode_topk. */
int profk_sae_encode_dense(const void* x, const void* w_enc, const float* b_enc, int64_t B,
                           int64_t d_model, int64_t d_dict, float* out, void* stream);

/* Sparse decode: out[b, :] = sum over the entries i < K with flat_idx[i] =
 * b*d_dict + j of vals[i] * W_dec[j, :], plus b_dec.  Entries with a
 * negative or out-of-range index (relaxed-recall padding) are skipped.  Each
 * row's terms are summed in fp32 in ascending j, so the result does not
 * depend on the order of the list.  w_dec: bf16 [d_dict, d_model]
 * row-major; b_dec fp32 [d_model]; out fp32 [B, d_model]; d_dict <= 16384;
 * ws: profk_sae_decode_workspace_size(B, K) bytes. */
size_t profk_sae_decode_workspace_size(int64_t B, int64_t K);
int profk_sae_decode(const float* vals, const int64_t* flat_idx, int64_t K, const void* w_dec,
                     const float* b_dec, int64_t B, int64_t d_model, int64_t d_dict, float* out,
                     void* ws, size_t ws_bytes, void* stream);

/* Inspection: the keys of the S latents profk_sae_encode_topk samples for
 * this plan and seed (draw j at keys_dev[j], S entries); ws as for
 * profk_sae_encode_topk.  The draws' flat indices are
 * profk_debug_sample_indices(seed, 0, S, B*d_dict). */
int profk_debug_sae_sample(const profk_plan_t* plan, const void* x, const void* w_enc,
                           const float* b_enc, int64_t B, int64_t d_model, int64_t d_dict,
                           uint64_t seed, uint32_t* keys_dev, void* ws, size_t ws_bytes,
                           void* stream);

/* profk_topk with stages 1-2 replaced by a caller-given threshold key, to
 * drive the underflow and overflow paths on purpose.  A key alone names no
 * threshold pair, so this entry point filters with key >= tau_key also for
 * lexicographic plans. */
int profk_topk_tau(const profk_plan_t* plan, int32_t dtype, const void* values,
                   int64_t N, int64_t k, uint32_t tau_key, void* out_vals,
                   int64_t* out_idx, void* ws, size_t ws_bytes, void* stream,
                   profk_info_t* info_dev);

/* Timing hook for measurement tools: while set, every flat call records
 * `before` on its stream immediately before the filter-pass launch (stage 3)
 * and `after` immediately after it.  Both are hipEvent_t passed as void*;
 * NULL, NULL clears the hook.  The setting is per calling thread. */
void profk_set_trace_events(void* before, void* after);

/* ---- Status ------------------------------------------------------------- */

const char* profk_status_string(int code);
/* The last hipError_t seen by this thread (0 if none). */
int profk_last_hip_error(void);
/* Free the workspace held for profk_topk_simple. */
void profk_release(void);

#ifdef __cplusplus
}
#endif

#endif /* PROFK_H */
