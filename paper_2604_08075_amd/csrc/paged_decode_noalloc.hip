// paged_decode_attention without a caller workspace, for callers that cannot
// allocate device memory.  The split-K arrival counters and partial records
// live in one fixed device array per GPU (`scratch`), which the library
// holds until the process ends; the decode itself is the same launch as
// paged_decode_attention's, with that array as its workspace.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device (hipGetSymbolAddress, with the
// device current) and only that address is ever handed to a kernel.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "common.h"

namespace {

constexpr size_t kScratchBytes = (size_t)32 << 20;  // 32 MiB per GPU
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Zero the whole array once per device before its first use: the decode
// requires its arrival counters to start at zero (every call leaves them so).
__global__ __launch_bounds__(256) void scratch_clear_kernel(i32x4* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    p[i] = i32x4{0, 0, 0, 0};
}

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's scratch, set up (looked up and cleared on
// `stream`) on the first call made on the device.
int scratch_on_device(void* stream, void** out) {
  using dpool::fail;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    const hipError_t e = hipGetLastError();
    return fail(DP_EIO, "paged_decode_attention_noalloc: no current device: %s", hipGetErrorString(e));
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(DP_ENOTSUP, "paged_decode_attention_noalloc: device %d", dev);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(DP_EIO, "paged_decode_attention_noalloc: scratch address lookup failed: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    hipLaunchKernelGGL(scratch_clear_kernel, dim3(1024), dim3(256), 0, (hipStream_t)stream, (i32x4*)p,
                       kScratchBytes / sizeof(i32x4));
    const hipError_t le = hipGetLastError();
    if (le != hipSuccess)
      return fail(DP_EIO, "paged_decode_attention_noalloc: scratch clear failed: %s", hipGetErrorString(le));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DP_OK;
}

}  // namespace

extern "C" int paged_decode_attention_noalloc(const void* q, const void* k_blocks, const void* v_blocks,
                                              const int32_t* block_tables, const int32_t* context_lens, float scale,
                                              const float* k_scale, const float* v_scale, void* out,
                                              const dp_decode_shape* shape, void* stream) {
  size_t need = 0;
  const int rc = dpool::decode_workspace_bytes(shape, &need);
  if (rc != DP_OK) return rc;
  if (need > kScratchBytes)
    return dpool::fail(DP_ENOMEM,
                       "paged_decode_attention_noalloc: this shape needs %zu bytes of scratch, more than the %zu "
                       "the library holds per GPU (use paged_decode_attention with a workspace)",
                       need, kScratchBytes);
  void* ws = nullptr;
  const int src = scratch_on_device(stream, &ws);
  if (src != DP_OK) return src;
  return paged_decode_attention(q, k_blocks, v_blocks, block_tables, context_lens, scale, k_scale, v_scale, out,
                                shape, ws, kScratchBytes, stream);
}
