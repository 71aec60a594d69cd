/*
 * dpool.h - C ABI of libdpool: MI355X (gfx950) paged decode attention for
 * dual-pool token-budget serving, plus the host-side pool sizing and router
 * that decide which pool (and so which decode shape) a request lands in.
 *
 * Paper: "Dual-Pool Token-Budget Routing for Cost-Efficient and Reliable LLM
 * Serving".  Citations below name its sections, equations and algorithm.
 *
 * Conventions (every entry point):
 *   - returns int status: DP_OK (0) or a negative errno-style code:
 *       DP_EINVAL  (-22) bad argument or shape
 *       DP_ENOMEM  (-12) block pool exhausted / workspace too small
 *       DP_ENOTSUP (-95) head_dim, block size, dtype or GQA group not supported
 *       DP_EIO     (-5)  a HIP runtime error (text via dp_last_error())
 *   - no exception, abort or exit crosses the ABI; on error, caller-visible
 *     state is left unchanged;
 *   - the caller owns every buffer it passes.  The library owns only the
 *     opaque dp_kv_pool handle (host memory);
 *   - device pointers are HIP device addresses on the current device; the
 *     decode call is asynchronous on the given stream and never synchronises.
 */
#ifndef DPOOL_H
#define DPOOL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DP_OK 0
#define DP_EIO (-5)
#define DP_ENOMEM (-12)
#define DP_EINVAL (-22)
#define DP_ENOTSUP (-95)

/* Text of the last error raised on the calling thread ("" if none). */
const char* dp_last_error(void);

/* Library version string. */
const char* dp_version(void);

/* ------------------------------------------------------------------------ */
/* KV-cache sizing and paged block pool (host only).                         */
/*                                                                           */
/* Sec. 1.1 Eq. 1: M_seq = 2 * n_layers * n_kv_heads * head_dim             */
/*                         * dtype_bytes * c_max   (bytes per sequence)      */
/* Sec. 1.1 Eq. 2: N_seq = floor((m_gpu_bytes * util - m_model_bytes)       */
/*                               / M_seq), clamped at 0                      */
/* The pool backs N_seq sequences of ceil(c_max / block_size) blocks each   */
/* (16-token PagedAttention blocks, pages handed out on demand: Sec. 3,     */
/* effects 1 and 3).  Free block ids are kept in a list shuffled once with  */
/* a seeded SplitMix64 stream (Steele, Lea & Flood 2014), so that a         */
/* sequence's blocks are scattered over the pool as in a long-running       */
/* server.                                                                   */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_layers;     /* n_l: layers whose KV this GPU holds             */
  int32_t n_kv_heads;   /* n_h: KV heads on this GPU                        */
  int32_t head_dim;     /* d_h                                              */
  int32_t dtype_bytes;  /* b_dtype: 2 for bf16, 1 for fp8                   */
  int32_t block_size;   /* tokens per block (16)                            */
  int32_t reserved;     /* must be 0                                        */
  int64_t c_max;        /* C_max: tokens reserved per sequence              */
  double m_gpu_bytes;   /* M_gpu                                             */
  double util;          /* u, fraction of HBM usable (0, 1]                  */
  double m_model_bytes; /* M_model (weights + activations)                   */
} dp_pool_config;

typedef struct dp_kv_pool dp_kv_pool; /* opaque, host memory, owned by the library */

/* Size a pool (Eq. 1, Eq. 2) and build its shuffled free list.
 * DP_EINVAL on non-positive sizes, util outside (0,1] or reserved != 0;
 * DP_ENOMEM if the free list cannot be allocated.  *out is set only on success. */
int kv_pool_create(const dp_pool_config* cfg, uint64_t shuffle_seed, dp_kv_pool** out);

/* Sizing results: Eq. 1 M_seq, Eq. 2 N_seq, ceil(c_max/bs), N_seq*blocks_per_seq,
 * and the number of blocks currently free.  Any output pointer may be NULL. */
int kv_pool_info(const dp_kv_pool* pool, int64_t* m_seq_bytes, int64_t* n_seq,
                 int64_t* blocks_per_seq, int64_t* num_blocks, int64_t* free_blocks);

/* Hand out ceil(n_tokens / block_size) blocks for one sequence (on-demand
 * pages, Sec. 3 effect 1).  block_ids_out must hold that many int32.
 * DP_EINVAL if n_tokens < 0 or n_tokens > c_max; DP_ENOMEM if the pool has
 * too few free blocks (the OOM of Sec. 1.3), in which case nothing is taken. */
int kv_pool_alloc_seq(dp_kv_pool* pool, int64_t n_tokens, int32_t* block_ids_out);

/* Return blocks to the pool.  DP_EINVAL (nothing returned) if any id is out
 * of range or already free. */
int kv_pool_free_seq(dp_kv_pool* pool, const int32_t* block_ids, int64_t n_blocks);

void kv_pool_destroy(dp_kv_pool* pool);

/* ------------------------------------------------------------------------ */
/* Token-budget routing (host only): Sec. 2.1 Eq. 3-5, Sec. 2.2 Algorithm 1 */
/*                                                                           */
/* Route:  c* = c_hat_k - gamma * sigma_k (Eq. 5), clamped below at c_min;   */
/*         L_total = ceil(bytes / c*) + max_output_tokens (Eq. 3);           */
/*         step 1  L_total > C_max(short)           -> long                  */
/*         step 2  L_total <= b_short ? short : long                         */
/*         step 3  spill to the other pool if the chosen one is overloaded   */
/*                 (in_flight >= spill_theta * capacity) and the other can   */
/*                 take the request (L_total <= its C_max, not overloaded);  */
/*         final   L_total > C_max(chosen)          -> long.                 */
/*         The chosen pool's in_flight is incremented.                       */
/* OnResponse: c_obs = bytes / prompt_tokens;                                */
/*         c_hat = beta*c_hat + (1-beta)*c_obs (Eq. 4);                      */
/*         sigma = beta*sigma + (1-beta)*|c_obs - c_hat| (updated c_hat).    */
/* All arithmetic is IEEE double in exactly that order (no FMA contraction), */
/* so results are reproducible bit for bit by any IEEE-754 implementation.   */
/* ------------------------------------------------------------------------ */
typedef struct {
  double b_short;     /* B_short threshold in tokens (default 8192)        */
  double beta;        /* EMA decay (0.95)                                   */
  double gamma;       /* conservativeness (1.0)                             */
  double c0;          /* cold-start bytes/token (4.0)                       */
  double c_min;       /* floor of the conservative ratio (1.0)              */
  double spill_theta; /* overload fraction of capacity (1.0)                */
} dp_route_params;

typedef struct {
  double c_hat; /* calibrated bytes per token of the category */
  double sigma; /* EMA of |c_obs - c_hat|                      */
} dp_cat_state;

typedef struct {
  int64_t c_max;     /* longest total budget the pool can serve */
  int64_t capacity;  /* concurrent sequences (N_seq * instances) */
  int64_t in_flight; /* requests currently assigned             */
} dp_pool_state;      /* pools[0] = short pool, pools[1] = long pool */

/* Fill params with the paper's defaults. */
int route_default_params(dp_route_params* params);

/* Cold-start every category: c_hat = c0, sigma = 0. */
int route_init(const dp_route_params* params, dp_cat_state* cats, int32_t n_cats);

/* Route n requests in order (Algorithm 1, Route).  req_bytes[i] >= 0,
 * 0 <= req_cat[i] < n_cats, req_max_out[i] >= 0; otherwise DP_EINVAL and
 * nothing is written.  out_pool[i] = 0 (short) or 1 (long); out_l_total[i]
 * = the estimated budget (either output may be NULL).  pools[*].in_flight is
 * updated.  Host arrays, O(n), no allocation. */
int route_requests(const dp_route_params* params, const dp_cat_state* cats, int32_t n_cats,
                   dp_pool_state pools[2], const int64_t* req_bytes, const int32_t* req_cat,
                   const int64_t* req_max_out, int64_t n, int8_t* out_pool,
                   int64_t* out_l_total);

/* Algorithm 1, OnResponse.  DP_EINVAL (state unchanged) if cat is out of
 * range, req_bytes < 0 or prompt_tokens <= 0. */
int route_on_response(const dp_route_params* params, dp_cat_state* cats, int32_t n_cats,
                      int32_t cat, int64_t req_bytes, int64_t prompt_tokens);

/* ------------------------------------------------------------------------ */
/* Adaptive B_short (host only).  Sec. 7 names, as future work, a routing   */
/* threshold that adjusts itself from preemption rate, OOM events and        */
/* request rejections; Sec. 6 recommends alerting on a preemption rate above */
/* 1%, and Sec. 4.6 finds any B_short in 4K-16K within 80% of peak savings.  */
/* The paper gives no update rule; this is the library's, one call per       */
/* control interval:                                                         */
/*   e_i = w_preempt*preempted_i + w_oom*oom_i + w_reject*rejected_i         */
/*   x_i = e_i / max(admitted_i, 1) - target        (i = 0 short, 1 long)    */
/*   x_0 > 0 and x_0 > x_1:  b = b - step*b   (short pool under pressure:    */
/*                                             send borderline traffic long) */
/*   x_1 > 0 and x_1 > x_0:  b = b + step*b   (long pool under pressure)     */
/*   otherwise               b unchanged                                     */
/*   then b is clamped into [b_min, b_max].                                  */
/* IEEE double, in exactly that order, no FMA contraction.                   */
/* ------------------------------------------------------------------------ */
typedef struct {
  int64_t admitted;  /* requests routed to the pool during the interval */
  int64_t preempted; /* sequences preempted for want of KV cache         */
  int64_t oom;       /* out-of-memory events                             */
  int64_t rejected;  /* requests refused at admission                    */
} dp_pool_signals;   /* signals[0] = short pool, signals[1] = long pool  */

typedef struct {
  double w_preempt; /* weight of a preemption (1.0)                          */
  double w_oom;     /* weight of an OOM event (1.0)                          */
  double w_reject;  /* weight of a rejection (1.0)                           */
  double target;    /* tolerated events per admitted request (0.01)          */
  double step;      /* relative change of B_short per interval (0.05)        */
  double b_min;     /* lower bound of B_short in tokens (4096)               */
  double b_max;     /* upper bound (16384; no use above the short C_max)     */
} dp_adapt_params;

/* Fill ap with the defaults above. */
int route_adapt_default_params(dp_adapt_params* ap);

/* One control step on *b_short (in/out).  *action (may be NULL) = -1, 0 or
 * +1 for lowered, unchanged, raised (before the clamp).  DP_EINVAL, nothing
 * written, unless every count is >= 0, the weights and target are >= 0,
 * 0 < step < 1, 0 < b_min <= b_max and *b_short is finite and > 0. */
int route_adapt_threshold(const dp_adapt_params* ap, const dp_pool_signals signals[2], double* b_short,
                          int32_t* action);

/* ------------------------------------------------------------------------ */
/* Fleet cost model (host only): Sec. 3, "Cost Model: Why Splitting Always  */
/* Helps".                                                                   */
/*   G_homo = ceil(lambda / mu_long)                                         */
/*   G_dual = ceil(alpha * lambda / mu_short)                                */
/*          + ceil((1 - alpha) * lambda / mu_long)                           */
/*   rho = mu_short / mu_long;  savings_formula = alpha * (1 - 1 / rho)      */
/*   (the boxed equation);  savings_fleet = (G_homo - G_dual) / G_homo       */
/* lambda: request rate; alpha: fraction of traffic short; mu_*: per-GPU     */
/* throughput of each pool, same unit as lambda.  IEEE double, in that       */
/* order, no FMA contraction.  DP_EINVAL (nothing written) unless           */
/* lambda > 0, 0 <= alpha <= 1 and both throughputs are positive.           */
/* ------------------------------------------------------------------------ */
typedef struct {
  int64_t g_homo;         /* GPUs of the homogeneous fleet           */
  int64_t g_dual;         /* GPUs of the dual-pool fleet             */
  double rho;             /* throughput gain ratio                   */
  double savings_formula; /* alpha (1 - 1/rho)                       */
  double savings_fleet;   /* (G_homo - G_dual) / G_homo, with ceilings */
} dp_cost_result;

int dp_cost_model(double lambda, double alpha, double mu_short, double mu_long, dp_cost_result* out);

/* ------------------------------------------------------------------------ */
/* Paged decode attention (device, asynchronous).                           */
/*                                                                           */
/* The per-step KV read the paper's cost model calls memory-bandwidth bound */
/* (Sec. 3 effect 4; Sec. 4.4 "Why TPOT also improves"), over 16-token      */
/* PagedAttention blocks (Sec. 3 effect 3).  For sequence s with            */
/* T = context_lens[s] and query head h (KV head g = h / G, G = Hq / Hkv):  */
/*   K_t = k_scale[g] * k_blocks[block_tables[s][t/16], g, t%16, :]          */
/*   V_t = v_scale[g] * v_blocks[block_tables[s][t/16], g, :, t%16]          */
/*   out[s,h,:] = softmax_t(scale * q[s,h,:] . K_t) @ V                     */
/* T = 0 gives a zero row.                                                   */
/*                                                                           */
/* Layouts (row-major, device memory, 16-byte aligned):                      */
/*   q            [batch, n_q_heads, head_dim]            bf16               */
/*   k_blocks     [num_blocks, n_kv_heads, block_size, head_dim]             */
/*                (token-major: one token's dims are contiguous)             */
/*   v_blocks     [num_blocks, n_kv_heads, head_dim, block_size]             */
/*                (dims-major: one dim's 16 tokens are contiguous)           */
/*                both bf16 (DP_KV_BF16) or OCP e4m3 bytes (DP_KV_FP8_E4M3); */
/*                each (block, KV head) tile of K and of V is contiguous     */
/*   block_tables [batch, max_blocks_per_seq] int32; entries past            */
/*                ceil(T/16) are never read (may hold -1); ids outside       */
/*                [0, num_blocks) are clamped into range, never dereferenced */
/*   context_lens [batch] int32, each <= max_context_len (a caller promise;  */
/*                larger values are clamped, never read out of bounds).      */
/*                Cache slots at t >= T of a sequence's last block are never */
/*                used, whatever they hold                                   */
/*   k_scale,     [n_kv_heads] fp32 per-head dequantisation scales (fp8      */
/*   v_scale        only; must be NULL for bf16)                             */
/*   out          [batch, n_q_heads, head_dim] bf16 (DP_OUT_BF16) or fp32    */
/*   workspace    >= paged_decode_workspace_size(shape) bytes, 256-byte      */
/*                aligned, caller-owned.  It must be zero-filled before its  */
/*                first use; every completed call leaves its arrival         */
/*                counters at zero again, so one workspace serves any number */
/*                of later calls, of any shape, in stream order.  Calls that */
/*                share a workspace must not overlap in time.                */
/* Supported: head_dim 128, block_size 16, 1 <= Hq/Hkv <= 16, batch <= 4096. */
/* ------------------------------------------------------------------------ */
#define DP_KV_BF16 0
#define DP_KV_FP8_E4M3 1
#define DP_OUT_BF16 0
#define DP_OUT_FP32 1

typedef struct {
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  int32_t max_blocks_per_seq;
  int32_t max_context_len;
  int32_t kv_dtype;          /* DP_KV_*                                       */
  int32_t out_dtype;         /* DP_OUT_*                                      */
  int32_t partition_tokens;  /* minimum tokens of KV one wave processes (the  */
                             /* split-K granularity): a multiple of 32 (bf16) */
                             /* or 64 (fp8); 0 = library's choice             */
  int32_t workgroups_per_cu; /* resident workgroups per compute unit, 1..8    */
                             /* (capped by occupancy); 0 = library's choice   */
  int32_t reserved;          /* must be 0                                     */
  int64_t num_blocks;        /* blocks in k_blocks / v_blocks                  */
} dp_decode_shape;

/* Bytes of workspace paged_decode_attention needs for this shape (it depends
 * on the device's compute-unit count and the GQA group).  Returns 0 for
 * invalid shapes (the reason is in dp_last_error()). */
size_t paged_decode_workspace_size(const dp_decode_shape* shape);

/* The minimum tokens per wave slice the library uses for this shape
 * (0 for invalid shapes). */
int32_t paged_decode_partition_tokens(const dp_decode_shape* shape);

/* Enqueue the decode attention on `stream` (a hipStream_t; NULL = default
 * stream) as one kernel launch.  Validates the shape and pointer alignment
 * on the host (DP_EINVAL / DP_ENOTSUP; DP_ENOMEM for a short workspace;
 * nothing is enqueued then); DP_EIO if the launch fails.
 *
 * Split-K over the context: the cached tokens of all (sequence, KV head)
 * pairs are cut into equal slices, one per wave; a pair cut by slice
 * boundaries leaves per-slice softmax partials (o_p, m_p, l_p), which are
 * merged with log-sum-exp weights M = max_p m_p, w_p = l_p * 2^(m_p - M),
 * out = sum_p w_p o_p / sum_p w_p: first inside each workgroup (through its
 * LDS), then, for pairs whose slices span several workgroups, the
 * workgroups' partials through the workspace, by the last to finish.
 * The workspace also keeps, for each wave, the cache tiles its first unit
 * read; the next call starts loading those tiles before it has found its
 * own, and loads again where they differ.  A call with the context lengths
 * and block tables of the previous call on the workspace (every layer of a
 * decode step after the first) starts its reads earlier; results never
 * depend on what the workspace holds.
 * Results are deterministic: the same inputs and shape give the same bits. */
int paged_decode_attention(const void* q, const void* k_blocks, const void* v_blocks,
                           const int32_t* block_tables, const int32_t* context_lens,
                           float scale, const float* k_scale, const float* v_scale,
                           void* out, const dp_decode_shape* shape, void* workspace,
                           size_t workspace_bytes, void* stream);

/* paged_decode_attention for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops and harnesses that forbid
 * hipMalloc).  Same arguments, layouts, results and errors as
 * paged_decode_attention, without the workspace: the library keeps a fixed
 * 32 MiB device array per GPU (held until the process ends, its address
 * looked up and the array zero-filled by one small kernel on `stream` at
 * the first call made on that device) and uses it as the workspace.  Nothing
 * is allocated, on the first call or later.
 * DP_ENOMEM (nothing enqueued) if the shape needs more than 32 MiB (see
 * paged_decode_workspace_size): every GQA group up to 16 fits with one
 * workgroup per compute unit (workgroups_per_cu 0 or 1) on a 256-CU device.
 * Every call on a device shares its array: calls that overlap in time on
 * one device (different streams, host threads) race and must not be made. */
int paged_decode_attention_noalloc(const void* q, const void* k_blocks, const void* v_blocks,
                                   const int32_t* block_tables, const int32_t* context_lens,
                                   float scale, const float* k_scale, const float* v_scale,
                                   void* out, const dp_decode_shape* shape, void* stream);

/* ------------------------------------------------------------------------ */
/* KV-cache append (device, asynchronous).                                   */
/*                                                                           */
/* Each decode step adds one token per sequence to the cache before the     */
/* attention reads it (Sec. 4.4: one KV-cache lookup per layer per          */
/* generated token); pages are 16-token blocks handed out on demand (Sec. 3 */
/* effects 1 and 3); the FP8 deployment of Sec. 4.7 stores 8-bit floats.   */
/* For sequence s, t = positions[s], KV head g:                             */
/*   blk = block_tables[s][t / 16], slot = t % 16                           */
/*   k_blocks[blk, g, slot, :] = enc(k_new[s, g, :] / k_scale[g])            */
/*   v_blocks[blk, g, :, slot] = enc(v_new[s, g, :] / v_scale[g])            */
/* enc() copies the bf16 bits for a bf16 cache (no scales); for an e4m3     */
/* cache it is a correctly rounded fp32 division, clamped to +-448 and      */
/* rounded to the nearest OCP E4M3FN value (ties to even).  Inputs are      */
/* finite (a caller promise).                                                */
/*                                                                           */
/*   k_new, v_new [batch, n_kv_heads, 128] bf16, 4-byte aligned             */
/*   k_blocks, v_blocks, block_tables: as for paged_decode_attention        */
/*   positions    [batch] int32: the slot index of the new token; a          */
/*                position outside [0, 16 * max_blocks_per_seq), or a block */
/*                id outside [0, num_blocks), writes nothing for that        */
/*                sequence                                                   */
/*   k_scale, v_scale [n_kv_heads] fp32 (e4m3 only; NULL for bf16)          */
/*   shape        uses batch, n_kv_heads, head_dim (128), block_size (16),   */
/*                max_blocks_per_seq, kv_dtype, num_blocks; the other        */
/*                fields are ignored except reserved (must be 0)            */
/* One launch on `stream`; DP_EINVAL / DP_ENOTSUP for bad arguments (nothing */
/* enqueued), DP_EIO if the launch fails.  Two sequences that name the same */
/* (block, slot) race.                                                       */
/* ------------------------------------------------------------------------ */
int kv_cache_append(const void* k_new, const void* v_new, void* k_blocks, void* v_blocks,
                    const int32_t* block_tables, const int32_t* positions,
                    const float* k_scale, const float* v_scale, const dp_decode_shape* shape,
                    void* stream);

/* ------------------------------------------------------------------------ */
/* Chunked-prefill attention (device, asynchronous).                        */
/*                                                                           */
/* Each pool runs chunked prefill internally (Sec. 1.2): a prompt is        */
/* attended in chunks (2,048 tokens by default) whose K and V are already   */
/* in the paged cache (kv_cache_append, or any writer of the same layout).  */
/* For sequence s with T = context_lens[s] cached tokens (the chunk         */
/* included) and n = q_start[s+1] - q_start[s] query rows, row              */
/* r = q_start[s] + i sits at position p = T - n + i and, for query head h  */
/* (KV head g = h / G):                                                      */
/*   out[r,h,:] = sum_{t <= p} softmax_t(scale * q[r,h,:] . K_t) V_t         */
/* with K_t, V_t gathered exactly as for paged_decode_attention.  Decode is */
/* the case n = 1.                                                           */
/*                                                                           */
/* Layouts: q and out [total_q, n_q_heads, 128] (bf16 / out_dtype), rows    */
/* packed sequence after sequence as q_start says; k_blocks, v_blocks,      */
/* block_tables, context_lens, k_scale, v_scale as for decode; q_start      */
/* [batch + 1] int32 on the device, non-decreasing, q_start[0] = 0,         */
/* q_start[batch] <= total_q.  A caller promise: n <= T for every sequence. */
/* Values that break it (or q_start out of order) are clamped: no access    */
/* leaves the buffers, rows past min(n, T) are left unwritten and rows of   */
/* overlapping ranges are unspecified.  No workspace; nothing is allocated. */
/* Supported: head_dim 128, block_size 16, Hq a multiple of Hkv,            */
/* batch <= 4096, max_context_len <= 65536 (the long pool's C_max).          */
/* ------------------------------------------------------------------------ */
typedef struct {
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  int32_t max_blocks_per_seq;
  int32_t max_context_len;
  int32_t kv_dtype;   /* DP_KV_*                                             */
  int32_t out_dtype;  /* DP_OUT_*                                            */
  int32_t query_tile; /* query tokens per work item: 0 or 32 (the only size) */
  int32_t reserved;   /* must be 0                                           */
  int64_t total_q;    /* rows of q and out                                   */
  int64_t num_blocks; /* blocks in k_blocks / v_blocks                       */
} dp_prefill_shape;

/* Enqueue the chunked-prefill attention on `stream` as one kernel launch.
 * Host-side validation as for decode (DP_EINVAL / DP_ENOTSUP, nothing
 * enqueued); DP_EIO if the launch fails. */
int chunked_prefill_attention(const void* q, const void* k_blocks, const void* v_blocks,
                              const int32_t* block_tables, const int32_t* context_lens,
                              const int32_t* q_start, float scale, const float* k_scale,
                              const float* v_scale, void* out, const dp_prefill_shape* shape,
                              void* stream);

/* ------------------------------------------------------------------------ */
/* HBM read probe (device, asynchronous; measurement only).                 */
/*                                                                           */
/* Decode attention is bound by the rate at which the cached K and V can be */
/* read (Sec. 3 effect 4; Sec. 4.4).  This call reads device memory as a    */
/* plain read would, so that the decode kernel's bandwidth can be set       */
/* against what this device reaches, beside its published peak:             */
/*   tile_ids == NULL: every byte of buf[0, bytes) once, the grid sweeping   */
/*                     it front to back (n_tiles must be 0);                 */
/*   tile_ids != NULL: the 4 KiB tiles buf + 4096 * tile_ids[i],             */
/*                     i = 0 .. n_tiles-1, in list order (the decode's       */
/*                     (block, KV head) tile reads); ids are clamped into    */
/*                     [0, bytes / 4096).                                    */
/* buf and bytes are 16-byte multiples; workgroups (of 256 threads) sets    */
/* the launch width; sink holds at least `workgroups` int32 and is written   */
/* only in the practically impossible case that a workgroup's folded data   */
/* equals a fixed constant (it exists so the loads cannot be elided).       */
/* One launch on `stream`; DP_EINVAL for bad arguments (nothing enqueued),  */
/* DP_EIO if the launch fails.  The caller owns every buffer.               */
/* ------------------------------------------------------------------------ */
int dp_hbm_read_probe(const void* buf, size_t bytes, const int32_t* tile_ids, int64_t n_tiles,
                      int32_t workgroups, int32_t* sink, size_t sink_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* DPOOL_H */
