// HBM read-bandwidth probe for gfx950: the measured ceiling that the decode
// kernel's KV stream is compared with.  Decode attention is bound by how fast
// the cached K and V can be read (Sec. 3 effect 4; Sec. 4.4), so the useful
// peak is what a plain read of HBM reaches on this device, beside the
// published 8 TB/s.
//
// Two access patterns:
//   * contiguous: every byte of a buffer read once, 16 bytes per lane per
//     load, the grid sweeping the buffer front to back;
//   * tile gather: 4 KiB tiles read in the order of a list of tile ids - the
//     access pattern of the decode kernel, which reads one contiguous 4 KiB
//     (block, KV head) tile per block-table entry.
// Loads are nontemporal (the data is read once), and the values are folded
// into one word per workgroup that is written only if it equals a constant
// no real data produces, so the loads cannot be optimised away and the
// probe writes nothing in practice.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"

namespace dpool_hip {

typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;  // 16-byte loads in flight per lane
constexpr int kTileBytes = 4096;
constexpr int kSinkMagic = 0x5eed1e55;

// Grid-stride over spans of kProbeThreads * kProbeUnroll vectors: in each
// round the workgroups read consecutive spans, so the whole grid sweeps the
// buffer front to back and its reads spread over every memory channel (a
// contiguous share per workgroup would start every workgroup at the same
// channel offset).
__global__ __launch_bounds__(kProbeThreads) void hbm_stream_read_kernel(const i32x4* __restrict__ src, size_t n_vec,
                                                                        int32_t* sink) {
  constexpr size_t kSpan = (size_t)kProbeThreads * kProbeUnroll;
  const size_t stride = (size_t)gridDim.x * kSpan;
  i32x4 acc = {0, 0, 0, 0};
  size_t base = (size_t)blockIdx.x * kSpan;
  for (; base + kSpan <= n_vec; base += stride) {
    i32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(src + base + u * kProbeThreads + threadIdx.x);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u];
  }
  if (base < n_vec)  // the one partial span (at most one workgroup has it)
    for (size_t i = base + threadIdx.x; i < n_vec; i += kProbeThreads) acc ^= __builtin_nontemporal_load(src + i);
  const int r = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (r == kSinkMagic) sink[blockIdx.x] = r;
}

// One wave reads one 4 KiB tile per step (four 16-byte loads per lane), four
// tiles in flight; each wave takes a contiguous share of the tile list.
__global__ __launch_bounds__(kProbeThreads) void hbm_tile_gather_kernel(const char* __restrict__ base,
                                                                        const int32_t* __restrict__ ids,
                                                                        int64_t n_tiles, int64_t max_id,
                                                                        int32_t* sink) {
  constexpr int kInFlight = 4;
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (kProbeThreads / 64);
  const int64_t gw = (int64_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6);
  const int64_t per = (n_tiles + waves - 1) / waves;
  const int64_t t0 = gw * per;
  const int64_t t1 = t0 + per < n_tiles ? t0 + per : n_tiles;
  i32x4 acc = {0, 0, 0, 0};
  for (int64_t t = t0; t < t1; t += kInFlight) {
    i32x4 v[kInFlight][4];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int64_t tt = t + u < t1 ? t + u : t1 - 1;  // the last tile is re-read: same lines, no extra traffic
      int64_t id = ids[tt];
      id = id < 0 ? 0 : (id > max_id ? max_id : id);
      const char* tile = base + id * kTileBytes;
#pragma unroll
      for (int k = 0; k < 4; ++k) v[u][k] = __builtin_nontemporal_load((const i32x4*)(tile + k * 1024 + lane * 16));
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc ^= v[u][k];
  }
  const int r = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (r == kSinkMagic) sink[blockIdx.x] = r;
}

}  // namespace dpool_hip

extern "C" int dp_hbm_read_probe(const void* buf, size_t bytes, const int32_t* tile_ids, int64_t n_tiles,
                                 int32_t workgroups, int32_t* sink, size_t sink_bytes, void* stream) {
  using dpool::fail;
  using namespace dpool_hip;
  if (!buf || !sink) return fail(DP_EINVAL, "hbm_read_probe: null buffer or sink");
  if (((uintptr_t)buf & 15) || (bytes & 15)) return fail(DP_EINVAL, "hbm_read_probe: buffer and size must be 16-byte multiples");
  if (workgroups <= 0 || workgroups > (1 << 20)) return fail(DP_EINVAL, "hbm_read_probe: workgroups %d outside [1, 2^20]", workgroups);
  if (sink_bytes < (size_t)workgroups * sizeof(int32_t))
    return fail(DP_EINVAL, "hbm_read_probe: sink needs %zu bytes", (size_t)workgroups * sizeof(int32_t));
  if (tile_ids) {
    if (n_tiles <= 0 || bytes < (size_t)kTileBytes) return fail(DP_EINVAL, "hbm_read_probe: empty tile list or buffer");
    if ((uintptr_t)tile_ids & 3) return fail(DP_EINVAL, "hbm_read_probe: tile ids must be 4-byte aligned");
  } else if (n_tiles != 0) {
    return fail(DP_EINVAL, "hbm_read_probe: n_tiles must be 0 without a tile list");
  }
  (void)hipGetLastError();
  if (tile_ids)
    hipLaunchKernelGGL(hbm_tile_gather_kernel, dim3(workgroups), dim3(kProbeThreads), 0, (hipStream_t)stream,
                       (const char*)buf, tile_ids, n_tiles, (int64_t)(bytes / kTileBytes) - 1, sink);
  else
    hipLaunchKernelGGL(hbm_stream_read_kernel, dim3(workgroups), dim3(kProbeThreads), 0, (hipStream_t)stream,
                       (const i32x4*)buf, bytes / 16, sink);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DP_EIO, "hbm_read_probe: kernel launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}
