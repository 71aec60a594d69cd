// Per-GPU KV pool sizing (Sec. 1.1, Eq. 1 and Eq. 2) and the paged block
// allocator behind it (16-token blocks handed out on demand: Sec. 3,
// effects 1 and 3).  Host only.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <new>
#include <vector>

#include "common.h"

struct dp_kv_pool {
  dp_pool_config cfg;
  int64_t m_seq;
  int64_t n_seq;
  int64_t blocks_per_seq;
  int64_t num_blocks;
  std::vector<int32_t> free_ids;  // stack of free block ids; allocation pops from the back
  std::vector<uint8_t> is_free;   // per block id
};

namespace {

// SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a counter advanced by the golden-ratio constant,
// finalised by two xor-shift-multiply rounds.
struct SplitMix64 {
  uint64_t state;
  uint64_t next() {
    uint64_t z = (state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
};

bool mul_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); }

}  // namespace

extern "C" int kv_pool_create(const dp_pool_config* cfg, uint64_t shuffle_seed, dp_kv_pool** out) {
  using dpool::fail;
  if (!cfg || !out) return fail(DP_EINVAL, "kv_pool_create: null argument");
  if (cfg->n_layers <= 0 || cfg->n_kv_heads <= 0 || cfg->head_dim <= 0 || cfg->dtype_bytes <= 0 ||
      cfg->block_size <= 0 || cfg->c_max <= 0 || cfg->reserved != 0)
    return fail(DP_EINVAL, "kv_pool_create: sizes must be positive (reserved must be 0)");
  if (!(cfg->util > 0.0 && cfg->util <= 1.0) || !(cfg->m_gpu_bytes > 0.0) || !(cfg->m_model_bytes >= 0.0))
    return fail(DP_EINVAL, "kv_pool_create: need m_gpu > 0, 0 < util <= 1, m_model >= 0");
  // Eq. 1: M_seq = 2 * n_l * n_h * d_h * b_dtype * C_max
  int64_t m = 2;
  if (!mul_ok(m, cfg->n_layers, &m) || !mul_ok(m, cfg->n_kv_heads, &m) || !mul_ok(m, cfg->head_dim, &m) ||
      !mul_ok(m, cfg->dtype_bytes, &m) || !mul_ok(m, cfg->c_max, &m))
    return fail(DP_EINVAL, "kv_pool_create: M_seq overflows int64");
  // Eq. 2: N_seq = floor((M_gpu * u - M_model) / M_seq), clamped at 0
  double x = std::floor((cfg->m_gpu_bytes * cfg->util - cfg->m_model_bytes) / (double)m);
  int64_t n_seq = x > 0.0 ? (int64_t)x : 0;
  int64_t bps = (cfg->c_max + cfg->block_size - 1) / cfg->block_size;
  int64_t nb;
  if (!mul_ok(n_seq, bps, &nb) || nb > std::numeric_limits<int32_t>::max())
    return fail(DP_EINVAL, "kv_pool_create: %lld blocks do not fit int32 block ids", (long long)nb);
  dp_kv_pool* p = new (std::nothrow) dp_kv_pool();
  if (!p) return fail(DP_ENOMEM, "kv_pool_create: out of host memory");
  try {
    p->free_ids.resize((size_t)nb);
    p->is_free.assign((size_t)nb, 1);
  } catch (...) {
    delete p;
    return fail(DP_ENOMEM, "kv_pool_create: out of host memory for %lld blocks", (long long)nb);
  }
  p->cfg = *cfg;
  p->m_seq = m;
  p->n_seq = n_seq;
  p->blocks_per_seq = bps;
  p->num_blocks = nb;
  for (int64_t i = 0; i < nb; ++i) p->free_ids[(size_t)i] = (int32_t)i;
  // Fisher-Yates shuffle of the free list driven by SplitMix64(seed).
  SplitMix64 rng{shuffle_seed};
  for (int64_t i = nb - 1; i > 0; --i) {
    int64_t j = (int64_t)(rng.next() % (uint64_t)(i + 1));
    std::swap(p->free_ids[(size_t)i], p->free_ids[(size_t)j]);
  }
  *out = p;
  dpool::clear_error();
  return DP_OK;
}

extern "C" int kv_pool_info(const dp_kv_pool* pool, int64_t* m_seq_bytes, int64_t* n_seq,
                            int64_t* blocks_per_seq, int64_t* num_blocks, int64_t* free_blocks) {
  if (!pool) return dpool::fail(DP_EINVAL, "kv_pool_info: null pool");
  if (m_seq_bytes) *m_seq_bytes = pool->m_seq;
  if (n_seq) *n_seq = pool->n_seq;
  if (blocks_per_seq) *blocks_per_seq = pool->blocks_per_seq;
  if (num_blocks) *num_blocks = pool->num_blocks;
  if (free_blocks) *free_blocks = (int64_t)pool->free_ids.size();
  return DP_OK;
}

extern "C" int kv_pool_alloc_seq(dp_kv_pool* pool, int64_t n_tokens, int32_t* block_ids_out) {
  using dpool::fail;
  if (!pool) return fail(DP_EINVAL, "kv_pool_alloc_seq: null pool");
  if (n_tokens < 0 || n_tokens > pool->cfg.c_max)
    return fail(DP_EINVAL, "kv_pool_alloc_seq: n_tokens %lld outside [0, C_max=%lld]", (long long)n_tokens,
                (long long)pool->cfg.c_max);
  int64_t need = (n_tokens + pool->cfg.block_size - 1) / pool->cfg.block_size;
  if (need == 0) return DP_OK;
  if (!block_ids_out) return fail(DP_EINVAL, "kv_pool_alloc_seq: null output");
  if (need > (int64_t)pool->free_ids.size())
    return fail(DP_ENOMEM, "kv_pool_alloc_seq: need %lld blocks, %zu free", (long long)need,
                pool->free_ids.size());
  for (int64_t i = 0; i < need; ++i) {
    int32_t id = pool->free_ids.back();
    pool->free_ids.pop_back();
    pool->is_free[(size_t)id] = 0;
    block_ids_out[i] = id;
  }
  return DP_OK;
}

extern "C" int kv_pool_free_seq(dp_kv_pool* pool, const int32_t* block_ids, int64_t n_blocks) {
  using dpool::fail;
  if (!pool) return fail(DP_EINVAL, "kv_pool_free_seq: null pool");
  if (n_blocks < 0) return fail(DP_EINVAL, "kv_pool_free_seq: negative count");
  if (n_blocks == 0) return DP_OK;
  if (!block_ids) return fail(DP_EINVAL, "kv_pool_free_seq: null ids");
  // validate everything first so that an error returns nothing
  std::vector<uint8_t> seen;
  for (int64_t i = 0; i < n_blocks; ++i) {
    int32_t id = block_ids[i];
    if (id < 0 || id >= pool->num_blocks) return fail(DP_EINVAL, "kv_pool_free_seq: id %d out of range", id);
    if (pool->is_free[(size_t)id]) return fail(DP_EINVAL, "kv_pool_free_seq: id %d is already free", id);
  }
  try {
    seen.assign((size_t)pool->num_blocks, 0);
  } catch (...) {
    return fail(DP_ENOMEM, "kv_pool_free_seq: out of host memory");
  }
  for (int64_t i = 0; i < n_blocks; ++i) {
    if (seen[(size_t)block_ids[i]]) return fail(DP_EINVAL, "kv_pool_free_seq: id %d repeated", block_ids[i]);
    seen[(size_t)block_ids[i]] = 1;
  }
  for (int64_t i = 0; i < n_blocks; ++i) {
    pool->is_free[(size_t)block_ids[i]] = 1;
    pool->free_ids.push_back(block_ids[i]);
  }
  return DP_OK;
}

extern "C" void kv_pool_destroy(dp_kv_pool* pool) { delete pool; }
