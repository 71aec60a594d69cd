// KV-cache append for gfx950: write each sequence's new token into its slot
// of the block-paged cache.
//
// Every decode step adds one token per sequence to the cache before the
// attention reads it (one KV-cache lookup per layer per generated token,
// Sec. 4.4 "Why TPOT also improves"); pages are 16-token blocks handed out on
// demand (Sec. 3 effects 1 and 3), and the FP8 deployment of Sec. 4.7 stores
// the cache in 8-bit floats.  For sequence s with new-token position
// t = positions[s] and KV head g:
//   blk = block_tables[s][t / 16], slot = t % 16
//   k_blocks[blk, g, slot, :] = enc(k_new[s, g, :] / k_scale[g])   (token-major tile)
//   v_blocks[blk, g, :, slot] = enc(v_new[s, g, :] / v_scale[g])   (dims-major tile)
// enc() is the identity for a bf16 cache (scales unused); for an e4m3 cache it
// is a correctly rounded fp32 division, clamped to +-448, rounded to the
// nearest OCP E4M3FN value (ties to even).
//
// One wave per (sequence, KV head): lane l owns head dimensions 2l and 2l+1,
// so the K row is one coalesced 256-byte (bf16) or 128-byte (e4m3) store;
// the V column is a strided scatter of 2-byte or 1-byte stores (one per head
// dimension, one per 32- or 16-byte tile row).  A position outside the
// sequence's block table, or a block id outside the pool, writes nothing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "common.h"

namespace dpool_hip {

constexpr int kAppendHeadDim = 128;
constexpr int kAppendBlock = 16;
constexpr int kAppendWaves = 4;  // (sequence, head) pairs per workgroup
constexpr float kE4M3Max = 448.0f;

struct AppendArgs {
  const uint16_t* k_new;  // [B, Hkv, 128] bf16
  const uint16_t* v_new;
  char* k;                // [num_blocks, Hkv, 16, 128] bf16 or e4m3
  char* v;                // [num_blocks, Hkv, 128, 16]
  const int32_t* block_tables;
  const int32_t* positions;
  const float* k_scale;   // [Hkv] (e4m3 only)
  const float* v_scale;
  int32_t batch, hkv, max_blocks_per_seq;
  int64_t num_blocks;
};

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Two fp32 values -> two OCP e4m3 codes (low byte: a), after the clamp that
// makes the conversion saturating.
__device__ __forceinline__ uint16_t f32x2_to_e4m3(float a, float b) {
  a = fminf(fmaxf(a, -kE4M3Max), kE4M3Max);
  b = fminf(fmaxf(b, -kE4M3Max), kE4M3Max);
  return (uint16_t)(__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xffff);
}

template <bool FP8>
__global__ __launch_bounds__(kAppendWaves * 64) void kv_append_kernel(AppendArgs a) {
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * kAppendWaves + (threadIdx.x >> 6);
  if (pair >= a.batch * a.hkv) return;
  const int s = pair / a.hkv, g = pair - s * a.hkv;
  const int t = a.positions[s];
  if (t < 0 || t >= a.max_blocks_per_seq * kAppendBlock) return;
  const int blk = a.block_tables[(size_t)s * a.max_blocks_per_seq + t / kAppendBlock];
  if (blk < 0 || blk >= a.num_blocks) return;
  const int slot = t % kAppendBlock;
  const size_t tile = (size_t)blk * a.hkv + g;
  const size_t src = ((size_t)s * a.hkv + g) * kAppendHeadDim + 2 * lane;
  const uint32_t kb = *(const uint32_t*)(a.k_new + src);  // dims 2l, 2l+1
  const uint32_t vb = *(const uint32_t*)(a.v_new + src);
  const int d = 2 * lane;
  if constexpr (FP8) {
    const float ks = a.k_scale[g], vs = a.v_scale[g];
    const uint16_t kc = f32x2_to_e4m3(bf16_bits_to_f32(kb & 0xffff) / ks, bf16_bits_to_f32(kb >> 16) / ks);
    const uint16_t vc = f32x2_to_e4m3(bf16_bits_to_f32(vb & 0xffff) / vs, bf16_bits_to_f32(vb >> 16) / vs);
    char* kt = a.k + tile * (kAppendBlock * kAppendHeadDim);
    *(uint16_t*)(kt + slot * kAppendHeadDim + d) = kc;
    char* vt = a.v + tile * (kAppendBlock * kAppendHeadDim);
    vt[d * kAppendBlock + slot] = (char)(vc & 0xff);
    vt[(d + 1) * kAppendBlock + slot] = (char)(vc >> 8);
  } else {
    uint16_t* kt = (uint16_t*)a.k + tile * (kAppendBlock * kAppendHeadDim);
    *(uint32_t*)(kt + slot * kAppendHeadDim + d) = kb;
    uint16_t* vt = (uint16_t*)a.v + tile * (kAppendBlock * kAppendHeadDim);
    vt[d * kAppendBlock + slot] = (uint16_t)(vb & 0xffff);
    vt[(d + 1) * kAppendBlock + slot] = (uint16_t)(vb >> 16);
  }
}

template __global__ void kv_append_kernel<false>(AppendArgs);
template __global__ void kv_append_kernel<true>(AppendArgs);

}  // namespace dpool_hip

using namespace dpool_hip;

extern "C" int kv_cache_append(const void* k_new, const void* v_new, void* k_blocks, void* v_blocks,
                               const int32_t* block_tables, const int32_t* positions, const float* k_scale,
                               const float* v_scale, const dp_decode_shape* sh, void* stream) {
  using dpool::fail;
  if (!sh) return fail(DP_EINVAL, "kv_cache_append: null shape");
  if (sh->head_dim != kAppendHeadDim) return fail(DP_ENOTSUP, "kv_cache_append: head_dim %d (only 128)", sh->head_dim);
  if (sh->block_size != kAppendBlock)
    return fail(DP_ENOTSUP, "kv_cache_append: block_size %d (only 16)", sh->block_size);
  if (sh->kv_dtype != DP_KV_BF16 && sh->kv_dtype != DP_KV_FP8_E4M3)
    return fail(DP_ENOTSUP, "kv_cache_append: kv_dtype %d", sh->kv_dtype);
  if (sh->reserved != 0) return fail(DP_EINVAL, "kv_cache_append: reserved must be 0");
  if (sh->batch < 0 || sh->n_kv_heads <= 0 || sh->max_blocks_per_seq <= 0 || sh->num_blocks <= 0)
    return fail(DP_EINVAL, "kv_cache_append: batch, n_kv_heads, max_blocks_per_seq and num_blocks must be positive");
  if ((int64_t)sh->batch * sh->n_kv_heads > INT32_MAX / 64 ||
      (int64_t)sh->max_blocks_per_seq * kAppendBlock > INT32_MAX)
    return fail(DP_EINVAL, "kv_cache_append: batch * n_kv_heads or the per-sequence capacity is too large");
  if (sh->batch == 0) return DP_OK;
  if (!k_new || !v_new || !k_blocks || !v_blocks || !block_tables || !positions)
    return fail(DP_EINVAL, "kv_cache_append: null tensor pointer");
  const bool fp8 = sh->kv_dtype == DP_KV_FP8_E4M3;
  if (fp8 && (!k_scale || !v_scale)) return fail(DP_EINVAL, "kv_cache_append: e4m3 cache needs k_scale and v_scale");
  if (!fp8 && (k_scale || v_scale))
    return fail(DP_EINVAL, "kv_cache_append: k_scale/v_scale must be NULL for a bf16 cache");
  if (((uintptr_t)k_new | (uintptr_t)v_new | (uintptr_t)k_blocks | (uintptr_t)v_blocks |
       (uintptr_t)block_tables | (uintptr_t)positions) & 3)
    return fail(DP_EINVAL, "kv_cache_append: pointers must be 4-byte aligned");
  AppendArgs a;
  a.k_new = (const uint16_t*)k_new;
  a.v_new = (const uint16_t*)v_new;
  a.k = (char*)k_blocks;
  a.v = (char*)v_blocks;
  a.block_tables = block_tables;
  a.positions = positions;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.batch = sh->batch;
  a.hkv = sh->n_kv_heads;
  a.max_blocks_per_seq = sh->max_blocks_per_seq;
  a.num_blocks = sh->num_blocks;
  const int pairs = sh->batch * sh->n_kv_heads;
  const dim3 grid((pairs + kAppendWaves - 1) / kAppendWaves);
  (void)hipGetLastError();
  if (fp8)
    hipLaunchKernelGGL(kv_append_kernel<true>, grid, dim3(kAppendWaves * 64), 0, (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(kv_append_kernel<false>, grid, dim3(kAppendWaves * 64), 0, (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DP_EIO, "kv_cache_append: kernel launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}
