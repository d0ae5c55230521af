// A read-only stream over device memory with the filter's access pattern:
// the practical ceiling the filter pass is measured against.  A persistent
// grid deals tiles of 16-byte vectors to its workgroups in turn, each lane
// keeping U nontemporal loads in flight; the words are XOR-folded so that
// no load can be dropped, and each workgroup writes its fold.
#include "device_common.h"
#include "filter_tile.h"
#include "launch.h"

namespace profk {

template <int U>
__global__ __launch_bounds__(kFiltBS) void k_read_probe(const u32x4* vec, uint32_t nvec, uint32_t* out) {
  constexpr uint32_t kTile = kFiltBS * U;
  const uint32_t tid = threadIdx.x;
  const uint32_t vstride = gridDim.x * kTile;
  uint32_t acc = 0;
  for (uint32_t vb = blockIdx.x * kTile; vb < nvec; vb += vstride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t vi = vb + u * kFiltBS + tid;
      v[u] = vi < nvec ? __builtin_nontemporal_load(vec + vi) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  // fold the workgroup: wave XOR through LDS
  __shared__ uint32_t s_x[kFiltBS];
  s_x[tid] = acc;
  __syncthreads();
  for (uint32_t h = kFiltBS / 2; h > 0; h >>= 1) {
    if (tid < h) s_x[tid] ^= s_x[tid + h];
    __syncthreads();
  }
  if (tid == 0) out[blockIdx.x] = s_x[0];
}

hipError_t launch_read_probe(const void* values, uint64_t nvec, int blocks_per_cu, int loads_per_lane,
                             uint32_t* out, uint32_t* grid_out, hipStream_t s) {
  const int cus = device_cu_count();
  uint64_t g = static_cast<uint64_t>(cus) * blocks_per_cu;
  if (g > static_cast<uint64_t>(kFiltMaxBlocks)) g = kFiltMaxBlocks;
  const uint64_t tiles = (nvec + static_cast<uint64_t>(kFiltBS) * loads_per_lane - 1) /
                         (static_cast<uint64_t>(kFiltBS) * loads_per_lane);
  if (tiles < g) g = tiles < 1 ? 1 : tiles;
  *grid_out = static_cast<uint32_t>(g);
  (void)hipGetLastError();
  const u32x4* vec = static_cast<const u32x4*>(values);
  const uint32_t n = static_cast<uint32_t>(nvec);
  if (loads_per_lane == 4) hipLaunchKernelGGL(k_read_probe<4>, dim3(g), dim3(kFiltBS), 0, s, vec, n, out);
  else hipLaunchKernelGGL(k_read_probe<8>, dim3(g), dim3(kFiltBS), 0, s, vec, n, out);
  return hipGetLastError();
}

}  // namespace profk
