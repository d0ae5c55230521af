// extern "C" entry points of libprofk.so: argument checks, workspace
// carving and launches.  Declarations and contracts are in include/profk.h.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "launch.h"
#include "plan_internal.h"
#include "profk.h"

namespace {

thread_local int g_last_hip_error = 0;
thread_local hipEvent_t g_ev_before = nullptr;
thread_local hipEvent_t g_ev_after = nullptr;

int hip_fail(hipError_t e) {
  g_last_hip_error = static_cast<int>(e);
  return PROFK_EHIP;
}

bool plan_consistent(const profk_plan_t* p) {
  return p->N >= 1 && p->N <= static_cast<int64_t>(UINT32_MAX) && p->k >= 1 && p->k <= p->N &&
         p->k_req >= 1 && p->k_req <= p->k && p->S >= 1 && p->t >= 1 && p->t <= p->S &&
         p->S <= static_cast<int64_t>(UINT32_MAX) && p->M >= p->k && p->M <= p->N &&
         (p->mode == PROFK_MODE_FILTER || p->mode == PROFK_MODE_DIRECT) &&
         (p->lexicographic == 0 || p->lexicographic == 1);
}

bool dtype_ok(int32_t dt) { return dt == PROFK_F32 || dt == PROFK_BF16; }

size_t elem_size(int32_t dt) { return dt == PROFK_F32 ? 4 : 2; }

// Shared checks of the flat entry points.  Returns PROFK_OK and fills the
// layout when the call may proceed.
int check_flat(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N, int64_t k,
               const void* out_vals, const int64_t* out_idx, const void* ws, size_t ws_bytes,
               profk::FlatLayout* L) {
  if (!plan || !values || !out_vals || !out_idx || !ws) return PROFK_ENULL;
  if (!dtype_ok(dtype)) return PROFK_EDTYPE;
  if (!plan_consistent(plan) || plan->N != N || plan->k != k) return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(values) % elem_size(dtype) != 0) return PROFK_EINVAL;
  *L = profk::flat_layout(*plan, dtype, profk::device_cu_count());
  if (ws_bytes < L->bytes) return PROFK_EWORKSPACE;
  return PROFK_OK;
}

int run_flat(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N, int64_t k,
             uint64_t seed, uint64_t row, void* out_vals, int64_t* out_idx, void* ws, size_t ws_bytes,
             void* stream, profk_info_t* info, int use_tau, uint32_t tau_key) {
  profk::FlatLayout L;
  const int rc = check_flat(plan, dtype, values, N, k, out_vals, out_idx, ws, ws_bytes, &L);
  if (rc != PROFK_OK) return rc;
  profk::FlatCall c{plan, dtype, values, static_cast<uint32_t>(N), static_cast<uint32_t>(k), seed, row,
                    out_vals, out_idx, static_cast<uint8_t*>(ws), L, static_cast<hipStream_t>(stream),
                    info, use_tau, tau_key, g_ev_before, g_ev_after};
  const hipError_t e = profk::launch_flat(c);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

// Row plans the one-workgroup row kernel takes: k within its collect limit
// and the sample, buffer and refinement within its LDS budget.  The buffer
// alone takes 4*M bytes (and a large sample 4*S), so larger plans are
// refused before row_layout's 32-bit sums could wrap.
bool rows_fit_block(const profk_plan_t* p, int32_t dtype) {
  constexpr int64_t kMaxWords = profk::kRowMaxLds / 4;
  return p->k <= profk::kRowMaxK && p->M <= kMaxWords && p->S <= kMaxWords &&
         profk::row_layout(*p, dtype).bytes <= profk::kRowMaxLds;
}

int check_sae_shape(const void* x, const void* w_enc, const float* b_enc, int64_t B, int64_t d_model,
                    int64_t d_dict) {
  if (!x || !w_enc || !b_enc) return PROFK_ENULL;
  if (B < 1 || d_model < 64 || d_model % 64 != 0 || d_dict < 1) return PROFK_EINVAL;
  if (d_model > (1 << 16) || B > static_cast<int64_t>(UINT32_MAX) / d_dict) return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(x) % 16 != 0 || reinterpret_cast<uintptr_t>(w_enc) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(b_enc) % 4 != 0)
    return PROFK_EINVAL;
  return PROFK_OK;
}

}  // namespace

extern "C" {

void profk_default_opts(profk_plan_opts_t* o) {
  if (!o) return;
  o->S_min = 32768;
  o->S_max = 131072;
  o->cost_ratio = 1.0;
  o->eps_split = 0.5;
  o->paper_literal = 0;
  o->force_mode = PROFK_FORCE_AUTO;
  o->lexicographic = 0;
}

void profk_default_row_opts(profk_plan_opts_t* o) {
  profk_default_opts(o);
  if (!o) return;
  o->S_min = 256;
  // tau_B / tau_A measured for the per-row kernel on MI355X: a sampled
  // element costs a scattered line fetch, so fewer draws and a larger buffer
  // are faster than the unit ratio.
  o->cost_ratio = 0.5;
}

int profk_plan(int64_t N, int64_t k, double eps, double recall, const profk_plan_opts_t* opts,
               profk_plan_t* out) {
  profk_plan_opts_t o;
  if (opts) o = *opts; else profk_default_opts(&o);
  return profk::make_plan(N, k, eps, recall, o, out);
}

void profk_default_sae_opts(profk_plan_opts_t* o) {
  profk_default_opts(o);
  if (!o) return;
  // tau_B / tau_A measured for the fused SAE path on MI355X: a draw is a
  // d_model-long dot product on the matrix cores with two row reads, not a
  // single gathered element, so fewer draws and a larger buffer are faster.
  o->cost_ratio = 1.0 / 64.0;
}

int profk_plan_rows(int64_t D, int64_t k, double eps, double recall, const profk_plan_opts_t* opts,
                    profk_plan_t* out) {
  profk_plan_opts_t o;
  if (opts) o = *opts; else profk_default_row_opts(&o);
  return profk::make_plan(D, k, eps, recall, o, out);
}

size_t profk_workspace_size(const profk_plan_t* plan, int32_t dtype, int64_t batch) {
  if (!plan || !dtype_ok(dtype) || !plan_consistent(plan) || batch < 1) return 0;
  // The one-workgroup row kernel keeps everything in LDS; rows outside its
  // envelope run the vector kernels one row after another on one workspace.
  if (batch > 1 && rows_fit_block(plan, dtype)) return 256;
  return profk::flat_layout(*plan, dtype, profk::device_cu_count()).bytes;
}

int profk_topk(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N, int64_t k,
               uint64_t seed, void* out_vals, int64_t* out_idx, void* ws, size_t ws_bytes,
               void* stream, profk_info_t* info_dev) {
  return run_flat(plan, dtype, values, N, k, seed, 0, out_vals, out_idx, ws, ws_bytes, stream,
                  info_dev, 0, 0);
}

int profk_topk_tau(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N, int64_t k,
                   uint32_t tau_key, void* out_vals, int64_t* out_idx, void* ws, size_t ws_bytes,
                   void* stream, profk_info_t* info_dev) {
  return run_flat(plan, dtype, values, N, k, 0, 0, out_vals, out_idx, ws, ws_bytes, stream, info_dev,
                  1, tau_key);
}

int profk_batchtopk(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t B, int64_t D,
                    int64_t k_row, uint64_t seed, void* out_vals, int64_t* out_flat_idx, void* ws,
                    size_t ws_bytes, void* stream, profk_info_t* info_dev) {
  if (B < 1 || D < 1 || k_row < 1 || k_row > D) return PROFK_EINVAL;
  if (B > static_cast<int64_t>(UINT32_MAX) / D) return PROFK_EINVAL;
  return run_flat(plan, dtype, values, B * D, B * k_row, seed, 0, out_vals, out_flat_idx, ws, ws_bytes,
                  stream, info_dev, 0, 0);
}

// ---- BatchTopK SAE layer ----

size_t profk_sae_workspace_size(const profk_plan_t* plan, int64_t B, int64_t d_dict) {
  if (!plan || !plan_consistent(plan) || B < 1 || d_dict < 1 || plan->N != B * d_dict) return 0;
  return profk::sae_layout(*plan, static_cast<uint32_t>(B), static_cast<uint32_t>(d_dict),
                           profk::device_cu_count())
      .bytes;
}

int profk_sae_encode_topk(const profk_plan_t* plan, const void* x, const void* w_enc, const float* b_enc,
                          int64_t B, int64_t d_model, int64_t d_dict, int64_t k_row, uint64_t seed,
                          float* out_vals, int64_t* out_flat_idx, void* ws, size_t ws_bytes, void* stream,
                          profk_info_t* info_dev) {
  if (!plan || !out_vals || !out_flat_idx || !ws) return PROFK_ENULL;
  int rc = check_sae_shape(x, w_enc, b_enc, B, d_model, d_dict);
  if (rc != PROFK_OK) return rc;
  if (k_row < 1 || k_row > d_dict) return PROFK_EINVAL;
  if (!plan_consistent(plan) || plan->N != B * d_dict || plan->k != B * k_row || plan->lexicographic)
    return PROFK_EINVAL;
  const profk::SaeLayout L = profk::sae_layout(*plan, static_cast<uint32_t>(B), static_cast<uint32_t>(d_dict),
                                               profk::device_cu_count());
  if (ws_bytes < L.bytes) return PROFK_EWORKSPACE;
  profk::SaeCall c{plan, x, w_enc, b_enc, static_cast<uint32_t>(B), static_cast<uint32_t>(d_model),
                   static_cast<uint32_t>(d_dict), static_cast<uint32_t>(B * k_row), seed, out_vals, out_flat_idx,
                   static_cast<uint8_t*>(ws), L, static_cast<hipStream_t>(stream), info_dev, nullptr,
                   g_ev_before, g_ev_after};
  const hipError_t e = profk::launch_sae_topk(c);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

int profk_sae_encode_dense(const void* x, const void* w_enc, const float* b_enc, int64_t B, int64_t d_model,
                           int64_t d_dict, float* out, void* stream) {
  if (!out) return PROFK_ENULL;
  int rc = check_sae_shape(x, w_enc, b_enc, B, d_model, d_dict);
  if (rc != PROFK_OK) return rc;
  profk::SaeCall c{};
  c.x = x;
  c.w = w_enc;
  c.bias = b_enc;
  c.B = static_cast<uint32_t>(B);
  c.d_model = static_cast<uint32_t>(d_model);
  c.d_dict = static_cast<uint32_t>(d_dict);
  c.stream = static_cast<hipStream_t>(stream);
  const hipError_t e = profk::launch_sae_dense(c, out);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

int profk_debug_sae_sample(const profk_plan_t* plan, const void* x, const void* w_enc, const float* b_enc,
                           int64_t B, int64_t d_model, int64_t d_dict, uint64_t seed, uint32_t* keys_dev,
                           void* ws, size_t ws_bytes, void* stream) {
  if (!plan || !keys_dev || !ws) return PROFK_ENULL;
  int rc = check_sae_shape(x, w_enc, b_enc, B, d_model, d_dict);
  if (rc != PROFK_OK) return rc;
  if (!plan_consistent(plan) || plan->N != B * d_dict || plan->mode != PROFK_MODE_FILTER) return PROFK_EINVAL;
  const profk::SaeLayout L = profk::sae_layout(*plan, static_cast<uint32_t>(B), static_cast<uint32_t>(d_dict),
                                               profk::device_cu_count());
  if (ws_bytes < L.bytes) return PROFK_EWORKSPACE;
  profk::SaeCall c{plan, x, w_enc, b_enc, static_cast<uint32_t>(B), static_cast<uint32_t>(d_model),
                   static_cast<uint32_t>(d_dict), static_cast<uint32_t>(plan->k), seed, nullptr, nullptr,
                   static_cast<uint8_t*>(ws), L, static_cast<hipStream_t>(stream), nullptr, keys_dev};
  const hipError_t e = profk::launch_sae_sample(c);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

size_t profk_sae_decode_workspace_size(int64_t B, int64_t K) {
  if (B < 1 || K < 0 || B > static_cast<int64_t>(INT32_MAX) || K > static_cast<int64_t>(UINT32_MAX)) return 0;
  return profk::sae_decode_workspace(static_cast<uint32_t>(B), static_cast<uint32_t>(K));
}

int profk_sae_decode(const float* vals, const int64_t* flat_idx, int64_t K, const void* w_dec,
                     const float* b_dec, int64_t B, int64_t d_model, int64_t d_dict, float* out, void* ws,
                     size_t ws_bytes, void* stream) {
  if (!vals || !flat_idx || !w_dec || !b_dec || !out || !ws) return PROFK_ENULL;
  if (K < 1 || B < 1 || d_model < 1 || d_dict < 1 || d_dict > static_cast<int64_t>(profk::sae_decode_max_dict()))
    return PROFK_EINVAL;
  if (B > static_cast<int64_t>(UINT32_MAX) / d_dict || K > B * d_dict || d_model > (1 << 16)) return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(w_dec) % 2 != 0) return PROFK_EINVAL;
  if (ws_bytes < profk_sae_decode_workspace_size(B, K)) return PROFK_EWORKSPACE;
  profk::SaeDecodeCall c{vals, flat_idx, static_cast<uint32_t>(K), static_cast<uint32_t>(B),
                         static_cast<uint32_t>(d_model), static_cast<uint32_t>(d_dict), w_dec, b_dec, out, ws,
                         static_cast<hipStream_t>(stream)};
  const hipError_t e = profk::launch_sae_decode(c);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

int profk_topk_rows(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t B, int64_t D,
                    int64_t row_stride, int64_t k, uint64_t seed, void* out_vals, int64_t* out_idx,
                    void* ws, size_t ws_bytes, void* stream, profk_info_t* info_dev) {
  if (!plan || !values || !out_vals || !out_idx) return PROFK_ENULL;
  if (!dtype_ok(dtype)) return PROFK_EDTYPE;
  if (!plan_consistent(plan) || plan->N != D || plan->k != k) return PROFK_EINVAL;
  if (B < 1 || B > static_cast<int64_t>(INT32_MAX) || row_stride < D) return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(values) % elem_size(dtype) != 0) return PROFK_EINVAL;
  if (!rows_fit_block(plan, dtype)) {
    // Wide rows or large k: each row runs the vector path (sample, filter,
    // refinement or fallback) with its own Philox stream, counter word 1 =
    // row, in turn on `stream`, so the rows share one workspace.
    if (!ws) return PROFK_ENULL;
    const profk::FlatLayout FL = profk::flat_layout(*plan, dtype, profk::device_cu_count());
    if (ws_bytes < FL.bytes) return PROFK_EWORKSPACE;
    const uint64_t es = elem_size(dtype);
    (void)hipGetLastError();
    for (int64_t r = 0; r < B; ++r) {
      profk::FlatCall fc{plan, dtype, static_cast<const uint8_t*>(values) + static_cast<uint64_t>(r) * row_stride * es,
                         static_cast<uint32_t>(D), static_cast<uint32_t>(k), seed, static_cast<uint64_t>(r),
                         static_cast<uint8_t*>(out_vals) + static_cast<uint64_t>(r) * k * es, out_idx + r * k,
                         static_cast<uint8_t*>(ws), FL, static_cast<hipStream_t>(stream),
                         info_dev ? info_dev + r : nullptr, 0, 0};
      const hipError_t e = profk::launch_flat(fc);
      if (e != hipSuccess) return hip_fail(e);
    }
    return PROFK_OK;
  }
  const profk::RowLayout L = profk::row_layout(*plan, dtype);
  profk::RowCall c{plan, dtype, values, static_cast<uint32_t>(B), static_cast<uint32_t>(D),
                   static_cast<uint32_t>(k), static_cast<uint64_t>(row_stride), seed, out_vals, out_idx,
                   info_dev, L, static_cast<hipStream_t>(stream)};
  const hipError_t e = profk::launch_rows(c);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

int profk_debug_sample_indices(uint64_t seed, int64_t row, int64_t S, int64_t N, int64_t* out_dev,
                               void* stream) {
  if (!out_dev) return PROFK_ENULL;
  if (S < 1 || S > static_cast<int64_t>(UINT32_MAX) || N < 1 || row < 0) return PROFK_EINVAL;
  const hipError_t e = profk::launch_sample_indices(seed, static_cast<uint64_t>(row),
                                                    static_cast<uint32_t>(S), static_cast<uint64_t>(N),
                                                    out_dev, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

int profk_debug_filter(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N,
                       uint32_t tau_key, uint32_t* buf_key, uint32_t* buf_idx, uint32_t* count_dev,
                       void* ws, size_t ws_bytes, void* stream) {
  if (!plan || !values || !buf_key || !buf_idx || !count_dev || !ws) return PROFK_ENULL;
  if (!dtype_ok(dtype)) return PROFK_EDTYPE;
  if (!plan_consistent(plan) || plan->N != N) return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(values) % elem_size(dtype) != 0) return PROFK_EINVAL;
  const profk::FlatLayout L = profk::flat_layout(*plan, dtype, profk::device_cu_count());
  if (ws_bytes < L.bytes) return PROFK_EWORKSPACE;
  profk::FlatCall c{plan, dtype, values, static_cast<uint32_t>(N), static_cast<uint32_t>(plan->k), 0, 0,
                    nullptr, nullptr, static_cast<uint8_t*>(ws), L, static_cast<hipStream_t>(stream),
                    nullptr, 1, tau_key};
  const hipError_t e = profk::launch_debug_filter(c, buf_key, buf_idx, count_dev);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

// ---- Entry point that allocates nothing ----
//
// profk_topk_noalloc runs profk_topk's kernels on a fixed device array
// instead of a caller's workspace.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up once per
// device with hipGetSymbolAddress and only that address is passed on.
static __device__ __align__(256) uint8_t scratch[PROFK_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on the first call on
// that device (with it current); NULL with *err set when the lookup fails.
void* device_scratch(hipError_t* err) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) { *err = e; return nullptr; }
  if (dev < 0 || dev >= kMaxDevices) { *err = hipErrorInvalidDevice; return nullptr; }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) { *err = e != hipSuccess ? e : hipErrorInvalidSymbol; return nullptr; }
    g_scratch_dev[dev] = ptr;
  }
  return g_scratch_dev[dev];
}
}  // namespace

int profk_topk_noalloc(const profk_plan_t* plan, int32_t dtype, const void* values, int64_t N, int64_t k,
                       uint64_t seed, void* out_vals, int64_t* out_idx, void* stream, profk_info_t* info_dev) {
  if (!plan || !values || !out_vals || !out_idx) return PROFK_ENULL;
  if (!dtype_ok(dtype)) return PROFK_EDTYPE;
  if (!plan_consistent(plan) || plan->N != N || plan->k != k) return PROFK_EINVAL;
  const size_t need = profk_workspace_size(plan, dtype, 1);
  if (need == 0) return PROFK_EINVAL;
  if (need > static_cast<size_t>(PROFK_NOALLOC_SCRATCH_BYTES)) return PROFK_EWORKSPACE;
  hipError_t e = hipSuccess;
  void* ws = device_scratch(&e);
  if (!ws) return hip_fail(e);
  return run_flat(plan, dtype, values, N, k, seed, 0, out_vals, out_idx, ws, PROFK_NOALLOC_SCRATCH_BYTES,
                  stream, info_dev, 0, 0);
}

int profk_debug_read_probe(const void* values, uint64_t bytes, int32_t blocks_per_cu, int32_t loads_per_lane,
                           uint32_t* out_dev, uint32_t* grid, void* stream) {
  if (!values || !out_dev || !grid) return PROFK_ENULL;
  // the probe's vector indices and its grid stride (at most 2^21 vectors)
  // stay below 2^32
  if (bytes < 16 || bytes % 16 != 0 || bytes / 16 > static_cast<uint64_t>(UINT32_MAX) - (1u << 22))
    return PROFK_EINVAL;
  if (reinterpret_cast<uintptr_t>(values) % 16 != 0) return PROFK_EINVAL;
  if (blocks_per_cu < 1 || blocks_per_cu > 8 || (loads_per_lane != 4 && loads_per_lane != 8)) return PROFK_EINVAL;
  const hipError_t e = profk::launch_read_probe(values, bytes / 16, blocks_per_cu, loads_per_lane, out_dev, grid,
                                                static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

namespace {
std::mutex g_simple_mu;
void* g_simple_ws = nullptr;
size_t g_simple_bytes = 0;
}  // namespace

int profk_topk_simple(const float* values, int64_t N, int64_t k, uint64_t seed, float* out_vals,
                      int64_t* out_idx) {
  profk_plan_t plan;
  int rc = profk_plan(N, k, 1e-6, 1.0, nullptr, &plan);
  if (rc != PROFK_OK) return rc;
  std::lock_guard<std::mutex> lock(g_simple_mu);
  const size_t need = profk_workspace_size(&plan, PROFK_F32, 1);
  if (need == 0) return PROFK_EINVAL;
  if (need > g_simple_bytes) {
    if (g_simple_ws) (void)hipFree(g_simple_ws);
    g_simple_ws = nullptr;
    g_simple_bytes = 0;
    hipError_t e = hipMalloc(&g_simple_ws, need);
    if (e != hipSuccess) return hip_fail(e);
    g_simple_bytes = need;
  }
  rc = profk_topk(&plan, PROFK_F32, values, N, k, seed, out_vals, out_idx, g_simple_ws, g_simple_bytes,
                  nullptr, nullptr);
  if (rc != PROFK_OK) return rc;
  const hipError_t e = hipStreamSynchronize(nullptr);
  return e == hipSuccess ? PROFK_OK : hip_fail(e);
}

void profk_release(void) {
  std::lock_guard<std::mutex> lock(g_simple_mu);
  if (g_simple_ws) (void)hipFree(g_simple_ws);
  g_simple_ws = nullptr;
  g_simple_bytes = 0;
}

const char* profk_status_string(int code) {
  switch (code) {
    case PROFK_OK: return "ok";
    case PROFK_EINVAL: return "invalid argument";
    case PROFK_EDTYPE: return "unsupported dtype";
    case PROFK_EWORKSPACE: return "workspace too small";
    case PROFK_ENULL: return "null pointer";
    case PROFK_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int profk_last_hip_error(void) { return g_last_hip_error; }

void profk_set_trace_events(void* before, void* after) {
  g_ev_before = static_cast<hipEvent_t>(before);
  g_ev_after = static_cast<hipEvent_t>(after);
}

}  // extern "C"
