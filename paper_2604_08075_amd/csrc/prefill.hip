// Chunked-prefill attention over the block-paged KV cache, for gfx950.
//
// What it computes: each pool runs chunked prefill internally (Sec. 1.2): a
// long prompt is attended in fixed-size chunks (2,048 tokens by default)
// whose K and V are written into the paged cache first.  For sequence s with
// T = context_lens[s] cached tokens and n = q_start[s+1] - q_start[s] query
// tokens, query row r = q_start[s] + i sits at position p = T - n + i and
// attends causally over the cache:
//     out[r,h] = sum_{t <= p} softmax_t(scale * q[r,h] . K_t) V_t,  g = h / G,
// with K_t, V_t gathered through the block table exactly as for decode
// (token-major K tiles, dims-major V tiles, per-head fp8 scales).
//
// Unlike decode, a chunk reuses every K/V tile for many query rows, so the
// work is a dense contraction and belongs on the matrix cores.  An item is
// one tile of QT query tokens of one sequence and eight query heads of one
// GQA group; a workgroup of eight waves takes it (one head per wave: the K/V
// tile staged in LDS feeds 8 * QT (query, head) columns).  The grid is one
// persistent workgroup per compute unit, taking items in turn, so a short
// item costs no dispatch and no repeated set-up.  Per 32-token KV tile:
//   * all 512 threads copy the two 16-token blocks of K and V from the cache
//     into LDS (fp8 widened to bf16 on the way, exactly), double buffered:
//     the next tile's global loads are in flight while the current one is
//     computed, and one barrier per tile separates the two;
//   * each wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (rows:
//     KV tokens, columns: 16 query tokens), the K rows read from LDS in a
//     token order chosen so that each lane's eight scores are exactly the
//     eight tokens its operand of O^T += V^T P^T needs (no cross-lane
//     movement of probabilities), and a column's max and sum reduce over
//     four lanes (two swaps);
//   * online softmax in base 2 (scale * log2 e folded into one fused
//     multiply-add in the exponent), the running rescale skipped when no
//     column's max grew; causal masking by select on the diagonal tiles only;
//   * V comes from LDS in its dims-major layout: one 16-byte read per lane
//     is the A operand (8 tokens of one head dimension).
// Tokens at or past T inside the last tile are zero in LDS (their V could be
// stale or poisoned; zero keeps 0 * V finite) and masked by causality.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "common.h"

namespace dpool_prefill {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kBS = 16;
constexpr int kKT = 32;               // KV tokens per LDS tile (two blocks)
constexpr int kWaves = 8;             // query heads per workgroup
// LDS tiles are unpadded, their 16-byte chunks XOR-swizzled by row (see ksw/vsw)
constexpr int kKRow = kD;             // LDS row of K: one token's 128 dims (16 chunks)
constexpr int kVRow = kKT;            // LDS row of V: one head dimension's 32 tokens (4 chunks)
constexpr int kKStage = kKT * kKRow;  // bf16 per K stage
constexpr int kVStage = kD * kVRow;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kSlack = 8.0f;        // probabilities may reach 2^8 before the reference max moves
constexpr int kMaxBatch = 4096;
constexpr int kIdCap = 4096;          // block ids staged in LDS: contexts up to 65,536 tokens

struct PrefillArgs {
  const uint16_t* q;            // [total_q, Hq, 128] bf16
  const char* k;                // [num_blocks, Hkv, 16, 128]
  const char* v;                // [num_blocks, Hkv, 128, 16]
  const int32_t* block_tables;  // [B, max_blocks_per_seq]
  const int32_t* context_lens;  // [B]
  const int32_t* q_start;       // [B + 1]
  const float* k_scale;
  const float* v_scale;
  void* out;                    // [total_q, Hq, 128] bf16 or fp32
  float scale_log2;             // scale * log2(e)
  int32_t batch, hq, hkv, group, nquad;
  int32_t max_blocks_per_seq, max_ctx, num_blocks_m1, out_fp32;
  int32_t total_q;
};

// Max over the four lanes li, li + 16, li + 32, li + 48: the permlane swaps
// pair each lane's value with its partner 16 (then 32) lanes away without a
// trip through LDS.
__device__ __forceinline__ float xor_max(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = fmaxf(__builtin_bit_cast(float, (unsigned)a[0]), __builtin_bit_cast(float, (unsigned)a[1]));
  const unsigned v = __builtin_bit_cast(unsigned, x);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__builtin_bit_cast(float, (unsigned)b[0]), __builtin_bit_cast(float, (unsigned)b[1]));
}

// Eight e4m3 bytes -> eight bf16 (exact).
__device__ __forceinline__ i32x4 fp8x8_to_bf16(int lo, int hi) {
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true);
  bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false);
  bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true);
  return i32x4{__builtin_bit_cast(int, a), __builtin_bit_cast(int, b), __builtin_bit_cast(int, c),
               __builtin_bit_cast(int, d)};
}

// Zero the 16-bit lanes of a 4-word bf16 chunk whose token index (first + k) is >= lim.
__device__ __forceinline__ i32x4 zero_tokens_from(i32x4 x, int first, int lim) {
#pragma unroll
  for (int wd = 0; wd < 4; ++wd) {
    unsigned m = 0;
    if (first + 2 * wd < lim) m |= 0xffffu;
    if (first + 2 * wd + 1 < lim) m |= 0xffff0000u;
    x[wd] &= (int)m;
  }
  return x;
}

// Chunk swizzles, chosen by measurement (the LDS bank-conflict counter on
// these exact read patterns reads zero): the sixteen K rows one MFMA reads
// at once (tokens 8q + 4m + e, q, e = 0..3) and the sixteen V rows 16 nn + li.
__device__ __forceinline__ int ksw(int row) { return (row & 3) | (((row >> 3) & 3) << 2); }
__device__ __forceinline__ int vsw(int row) { return (row >> 1) & 3; }
__device__ __forceinline__ int kpos(int row, int chunk) { return row * kKRow + ((chunk ^ ksw(row)) << 3); }
__device__ __forceinline__ int vpos(int row, int chunk) { return row * kVRow + ((chunk ^ vsw(row)) << 3); }

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// R: 16-token query column blocks per wave, so QT = 16 R query tokens per item.
template <bool FP8, int R>
__global__ __launch_bounds__(kWaves * 64, 1) void prefill_kernel(PrefillArgs a) {
  constexpr int QT = 16 * R;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kKStage];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][kVStage];
  __shared__ int ids_lds[kIdCap];    // the sequence's block ids, clamped into the pool
  extern __shared__ int tile_pre[];  // [B + 1] query tiles of sequences 0..s-1, then r0[B], r1[B], T[B]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, lj = lane >> 4;
  const int B = a.batch;
  int* const row0 = tile_pre + B + 1;  // first query row of each sequence (clamped)
  int* const row1 = row0 + B;          // one past its last
  int* const ctx = row1 + B;           // cached tokens (clamped)

  // ---- the items: (sequence, query tile, KV head, head quad) ----
  // Query tiles are numbered from the end of the batch backwards (the last
  // tile of the last sequence first): later tiles attend more tokens, so
  // the longest items are handed out first.
  if (tid == 0) tile_pre[0] = 0;
  {
    // exclusive prefix of ceil(n_s / QT) over sequences (serial per 256 sequences: B is small)
    for (int base = 0; base < B; base += kWaves * 64) {
      __syncthreads();
      const int s = base + tid;
      int cnt = 0;
      if (s < B) {
        const int r0 = min(max(a.q_start[s], 0), a.total_q);
        const int r1 = min(max(a.q_start[s + 1], r0), a.total_q);
        cnt = (r1 - r0 + QT - 1) / QT;
        row0[s] = r0;
        row1[s] = r1;
        ctx[s] = min(max(a.context_lens[s], 0), a.max_ctx);
      }
      // inclusive scan over the workgroup in LDS-free form: wave scans, then carry
      int incl = cnt;
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
      }
      __shared__ int wsum[kWaves];
      if (lane == 63) wsum[w] = incl;
      __syncthreads();
      int carry = tile_pre[base];
      for (int k = 0; k < w; ++k) carry += wsum[k];
      if (s < B) tile_pre[s + 1] = carry + incl;
    }
    __syncthreads();
  }
  const int total_tiles = tile_pre[B];
  const int per_tile = a.hkv * a.nquad;
  const int total_items = total_tiles * per_tile;
  // Persistent workgroups: round k hands the next gridDim.x items of the
  // longest-first order out forwards (k even) or backwards (k odd), so every
  // workgroup's items sum to about the same work, and its next item needs no
  // dispatch, no prefix and no global lookup of its sequence.
  for (int round = 0; round * (int)gridDim.x < total_items; ++round) {
    const int nwg = gridDim.x, wg = blockIdx.x;
    const int item = round * nwg + ((round & 1) ? nwg - 1 - wg : wg);
    if (item >= total_items) continue;  // uniform over the workgroup
    __syncthreads();  // every wave is done with the previous item's LDS tiles and block ids
    const int tile_rank = item / per_tile;
    const int rem = item - tile_rank * per_tile;
    const int g = rem / a.nquad;
    const int quad = rem - g * a.nquad;
    const int idx = total_tiles - 1 - tile_rank;
    int s;
    {
      int lo = 0, hi = B - 1;  // largest s with tile_pre[s] <= idx
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tile_pre[mid] <= idx) lo = mid;
        else hi = mid - 1;
      }
      s = __builtin_amdgcn_readfirstlane(lo);
    }
    const int qt = idx - tile_pre[s];
    const int r0 = row0[s];
    const int r1 = row1[s];
    const int T = ctx[s];
    const int n = min(r1 - r0, T);  // rows past the cached tokens are left unwritten
    const int q0 = qt * QT;
    if (q0 >= n) continue;  // uniform over the workgroup
    const int q1 = min(q0 + QT, n);
    const int p_first = T - n + q0;          // position of the tile's first query row
    const int n_kv = T - n + q1;             // tokens the tile attends: 0 .. n_kv - 1
    const int ntile = (n_kv + kKT - 1) / kKT;
    const int nb = (T + kBS - 1) / kBS;      // blocks in use
    const int32_t* bt = a.block_tables + (size_t)s * a.max_blocks_per_seq;

    const int hl = quad * kWaves + w;        // head index inside the group
    const bool active = hl < a.group;
    const int h = g * a.group + (active ? hl : 0);

    float cmul = a.scale_log2, vsc = 1.0f;
    if constexpr (FP8) {
      cmul *= a.k_scale[g];
      vsc = a.v_scale[g];
    }

    // ---- query fragments: B operand of S^T = K Q^T, column li = query q0 + 16 rb + li ----
    i32x4 qf[R][4];
#pragma unroll
    for (int rb = 0; rb < R; ++rb) {
      const int row = r0 + min(q0 + 16 * rb + li, n - 1);  // idle columns repeat the last row
      const uint16_t* qp = a.q + ((size_t)row * a.hq + h) * kD + 8 * lj;
#pragma unroll
      for (int c = 0; c < 4; ++c) qf[rb][c] = *(const i32x4*)(qp + 32 * c);
    }

    // ---- cooperative tile copy: cache -> registers -> LDS ----
    constexpr int NCH = 1;  // 16-byte chunks per thread, each of K and V (fp8: waves 0-3 copy K, 4-7 V)
    // Block ids come from LDS, staged once: a block-table load inside the loop
    // would sit behind the tile loads on the in-order memory counter, and
    // waiting for it would drain the tile prefetch.
    const int n_ids = min(min(2 * ntile, nb), kIdCap);
    for (int i = tid; i < n_ids; i += kWaves * 64) {
      const int id = bt[i];
      ids_lds[i] = id < 0 ? 0 : (id > a.num_blocks_m1 ? a.num_blocks_m1 : id);
    }
    __syncthreads();
    // The tile's block ids are the same for a whole wave: read once, kept in
    // scalar registers, so the loads address a uniform base plus a fixed lane
    // offset.
    auto tile_base = [&](int j, int b) __attribute__((always_inline)) {
      int bi = 2 * j + b;
      if (bi >= nb) bi = 2 * j;  // a block past the sequence re-reads the tile's first (then zeroed / masked)
      return __builtin_amdgcn_readfirstlane(ids_lds[bi]) * a.hkv + g;
    };
    // per-lane byte offsets inside a (block, head) tile, fixed for the kernel
    const int kx = FP8 ? ((tid & 127) >> 3) * 128 + (tid & 7) * 16 : ((tid & 255) >> 4) * 256 + (tid & 15) * 16;
    const int vx = FP8 ? (tid & 127) * 16 : ((tid & 255) >> 1) * 32 + (tid & 1) * 16;
    auto load_tile = [&](int j, i32x4 (&kreg)[NCH], i32x4 (&vreg)[NCH]) __attribute__((always_inline)) {
      if constexpr (FP8) {
        // waves 0-3 copy K, 4-7 V; waves 4m, 4m+1 the tile's first block, 4m+2, 4m+3 its second
        const size_t tile = (size_t)tile_base(j, (w >> 1) & 1);
        if (w < 4) kreg[0] = *(const i32x4*)(a.k + tile * 2048 + kx);
        else vreg[0] = *(const i32x4*)(a.v + tile * 2048 + vx);
      } else {
        const size_t tile = (size_t)tile_base(j, w >> 2);  // waves 0-3: first block, 4-7: second
        kreg[0] = *(const i32x4*)(a.k + tile * 4096 + kx);
        vreg[0] = *(const i32x4*)(a.v + tile * 4096 + vx);
      }
    };
    auto store_tile = [&](int j, int buf, const i32x4 (&kreg)[NCH], const i32x4 (&vreg)[NCH])
                          __attribute__((always_inline)) {
      uint16_t* kl = k_lds[buf];
      uint16_t* vl = v_lds[buf];
      const int t0 = kKT * j;
      if constexpr (FP8) {
        const int b = (w >> 1) & 1, x = tid & 127;
        if (w < 4) {
          // K: token 16b + x/8, dims 16 (x%8) .. +16
          const int krow = 16 * b + (x >> 3);
          *(i32x4*)(kl + kpos(krow, 2 * (x & 7))) = fp8x8_to_bf16(kreg[0][0], kreg[0][1]);
          *(i32x4*)(kl + kpos(krow, 2 * (x & 7) + 1)) = fp8x8_to_bf16(kreg[0][2], kreg[0][3]);
        } else {
          // V: dim x, tokens 16b .. +16
          i32x4 v0 = fp8x8_to_bf16(vreg[0][0], vreg[0][1]), v1 = fp8x8_to_bf16(vreg[0][2], vreg[0][3]);
          if (t0 + kKT > T) {  // the sequence ends inside this tile
            v0 = zero_tokens_from(v0, t0 + 16 * b, T);
            v1 = zero_tokens_from(v1, t0 + 16 * b + 8, T);
          }
          *(i32x4*)(vl + vpos(x, 2 * b)) = v0;
          *(i32x4*)(vl + vpos(x, 2 * b + 1)) = v1;
        }
      } else {
        const int b = w >> 2, x = tid & 255;
        *(i32x4*)(kl + kpos(16 * b + (x >> 4), x & 15)) = kreg[0];
        const int first = 16 * b + 8 * (x & 1);
        *(i32x4*)(vl + vpos(x >> 1, first >> 3)) = t0 + kKT > T ? zero_tokens_from(vreg[0], t0 + first, T) : vreg[0];
      }
    };

    // ---- per-lane LDS offsets of the MFMA operands ----
    // K row of MFMA m, row li: token 8 (li / 4) + 4 m + li % 4, so lane (li, lj)'s
    // scores are tokens 8 lj + 4 m + e: its eight P^T operand values.
    int koff[2][4], voff[8];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int c = 0; c < 4; ++c) koff[m][c] = kpos(8 * (li >> 2) + 4 * m + (li & 3), 4 * c + lj);
#pragma unroll
    for (int nn = 0; nn < 8; ++nn) voff[nn] = vpos(16 * nn + li, lj);

    f32x4 acc[R][8];
    float m_run[R], mlim[R];  // reference max (raw score) and the scaled score that forces a rescale
    f32x4 lsum[R];  // column sums of P, accumulated by the matrix cores (every row holds the sum)
#pragma unroll
    for (int rb = 0; rb < R; ++rb) {
      m_run[rb] = -INFINITY;
      mlim[rb] = -INFINITY;
      lsum[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int nn = 0; nn < 8; ++nn) acc[rb][nn] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Tiles stream through two register sets and two LDS stages: the loads of
    // tile j+2 are issued before tile j is computed and land in LDS after tile
    // j+1's computation, so each load has two tiles of compute to arrive in.
    // Loads and LDS stores are unconditional (a tile index past the end
    // re-reads the last tile, whose copy is never read), so the compiler's
    // wait counts never have to cover both register sets at once.
    bf16x8 ones;
#pragma unroll
    for (int x = 0; x < 8; ++x) ones[x] = (__bf16)1.0f;
    auto compute = [&](int j, int buf) __attribute__((always_inline)) {
        const uint16_t* kl = k_lds[buf];
        const uint16_t* vl = v_lds[buf];
        i32x4 kf[2][4], vf[8];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
          for (int c = 0; c < 4; ++c) kf[m][c] = *(const i32x4*)(kl + koff[m][c]);
#pragma unroll
        for (int nn = 0; nn < 8; ++nn) vf[nn] = *(const i32x4*)(vl + voff[nn]);
        const int tok0 = kKT * j + 8 * lj;            // token of this lane's score e = 0, m = 0
        const bool diag = kKT * j + kKT - 1 > p_first;  // some (token, query) pair is in the future
        // S^T = K Q^T for every column block first, so that the matrix cores
        // have independent work while the scores of one block are reduced.
        float z[R][8];
#pragma unroll
        for (int rb = 0; rb < R; ++rb) {
#pragma unroll
          for (int m = 0; m < 2; ++m) {
            f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < 4; ++c)
              sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[m][c]),
                                                             __builtin_bit_cast(bf16x8, qf[rb][c]), sacc, 0, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) z[rb][4 * m + e] = sacc[e];
          }
        }
        if (diag) {
#pragma unroll
          for (int rb = 0; rb < R; ++rb) {
            const int pcol = min(p_first + 16 * rb + li, T - 1);  // this column's query position
#pragma unroll
            for (int x = 0; x < 8; ++x)
              if (tok0 + x > pcol) z[rb][x] = -INFINITY;
          }
        }
        // Lazy rescale: the reference max m_run only moves when some score
        // exceeds it by more than 2^kSlack in probability (then to the exact
        // column max), so probabilities stay below 2^kSlack and the common
        // path has no cross-lane reduction, no rescale and no branch.
        float lmax[R];
        bool grow = false;
#pragma unroll
        for (int rb = 0; rb < R; ++rb) {
          lmax[rb] = z[rb][0];
#pragma unroll
          for (int x = 1; x < 8; ++x) lmax[rb] = fmaxf(lmax[rb], z[rb][x]);
          grow |= lmax[rb] * cmul > mlim[rb];
        }
        if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
          for (int rb = 0; rb < R; ++rb) {
            if (__builtin_amdgcn_ballot_w64(lmax[rb] * cmul > mlim[rb]) == 0) continue;
            const float m_new = fmaxf(m_run[rb], xor_max(lmax[rb]));
            const float alpha = __builtin_amdgcn_exp2f((m_run[rb] - m_new) * cmul);
            lsum[rb] *= alpha;
#pragma unroll
            for (int nn = 0; nn < 8; ++nn) acc[rb][nn] *= alpha;
            m_run[rb] = m_new;
            mlim[rb] = m_new * cmul + kSlack;
          }
        }
#pragma unroll
        for (int rb = 0; rb < R; ++rb) {
          const float mc = m_run[rb] * cmul;
          bf16x8 p;
#pragma unroll
          for (int x = 0; x < 8; ++x) p[x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(z[rb][x], cmul, -mc));
          // the softmax denominator sums the rounded probabilities the PV product uses
          lsum[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, p, lsum[rb], 0, 0, 0);
#pragma unroll
          for (int nn = 0; nn < 8; ++nn)
            acc[rb][nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[nn]), p, acc[rb][nn],
                                                                  0, 0, 0);
        }
        // Scheduling hint: the probabilities of block rb+1 are computed while
        // the matrix cores run block rb's PV product.
        __builtin_amdgcn_sched_group_barrier(0x002, 21, 0);
#pragma unroll
        for (int i = 0; i < 9 * (R - 1); ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 9, 0);
    };
    i32x4 kA[NCH], vA[NCH], kB[NCH], vB[NCH];
    load_tile(0, kA, vA);
    store_tile(0, 0, kA, vA);
    load_tile(min(1, ntile - 1), kA, vA);
    __syncthreads();
    // buf = j mod 2, a constant in each half of the unrolled loop
    auto iter = [&](int j, int buf, const i32x4 (&kc)[NCH], const i32x4 (&vc)[NCH], i32x4 (&kn)[NCH],
                    i32x4 (&vn)[NCH]) __attribute__((always_inline)) {
      load_tile(min(j + 2, ntile - 1), kn, vn);
      if (active && j < ntile) compute(j, buf);
      store_tile(j + 1, buf ^ 1, kc, vc);
      __syncthreads();
    };
    for (int j = 0; j < ntile; j += 2) {
      iter(j, 0, kA, vA, kB, vB);
      iter(j + 1, 1, kB, vB, kA, vA);
    }

    // ---- normalise and store: lane (li, lj) holds dims 16 nn + 4 lj + e of column li ----
    if (active) {
#pragma unroll
      for (int rb = 0; rb < R; ++rb) {
        const float inv = vsc / lsum[rb][0];
        const int qrow = q0 + 16 * rb + li;
        if (qrow >= q1) continue;
        const size_t base = ((size_t)(r0 + qrow) * a.hq + h) * kD + 4 * lj;
#pragma unroll
        for (int nn = 0; nn < 8; ++nn) {
          const f32x4 o = acc[rb][nn] * inv;
          if (a.out_fp32) {
            *(f32x4*)((float*)a.out + base + 16 * nn) = o;
          } else {
            u16x4 ob;
#pragma unroll
            for (int e = 0; e < 4; ++e) ob[e] = f32_to_bf16_bits(o[e]);
            *(u16x4*)((uint16_t*)a.out + base + 16 * nn) = ob;
          }
        }
      }
    }
  }
}

template __global__ void prefill_kernel<false, 2>(PrefillArgs);
template __global__ void prefill_kernel<true, 2>(PrefillArgs);

}  // namespace dpool_prefill

using namespace dpool_prefill;

namespace {

// Compute units of the current device (cached per device); 256 without one.
int compute_units() {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 256;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      n = 256;
    }
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace

extern "C" int chunked_prefill_attention(const void* q, const void* k_blocks, const void* v_blocks,
                                         const int32_t* block_tables, const int32_t* context_lens,
                                         const int32_t* q_start, float scale, const float* k_scale,
                                         const float* v_scale, void* out, const dp_prefill_shape* sh, void* stream) {
  using dpool::fail;
  if (!sh) return fail(DP_EINVAL, "chunked_prefill_attention: null shape");
  if (sh->head_dim != kD) return fail(DP_ENOTSUP, "chunked_prefill_attention: head_dim %d (only 128)", sh->head_dim);
  if (sh->block_size != kBS)
    return fail(DP_ENOTSUP, "chunked_prefill_attention: block_size %d (only 16)", sh->block_size);
  if (sh->kv_dtype != DP_KV_BF16 && sh->kv_dtype != DP_KV_FP8_E4M3)
    return fail(DP_ENOTSUP, "chunked_prefill_attention: kv_dtype %d", sh->kv_dtype);
  if (sh->out_dtype != DP_OUT_BF16 && sh->out_dtype != DP_OUT_FP32)
    return fail(DP_ENOTSUP, "chunked_prefill_attention: out_dtype %d", sh->out_dtype);
  if (sh->query_tile != 0 && sh->query_tile != 32)
    return fail(DP_EINVAL, "chunked_prefill_attention: query_tile must be 0 or 32");
  if (sh->reserved != 0) return fail(DP_EINVAL, "chunked_prefill_attention: reserved must be 0");
  if (sh->batch < 0) return fail(DP_EINVAL, "chunked_prefill_attention: batch < 0");
  if (sh->batch > kMaxBatch) return fail(DP_ENOTSUP, "chunked_prefill_attention: batch above 4096");
  if (sh->n_kv_heads <= 0 || sh->n_q_heads <= 0 || sh->n_q_heads % sh->n_kv_heads != 0)
    return fail(DP_EINVAL, "chunked_prefill_attention: n_q_heads must be a positive multiple of n_kv_heads");
  if (sh->max_blocks_per_seq <= 0 || sh->max_context_len < 0 ||
      (int64_t)sh->max_blocks_per_seq * kBS < sh->max_context_len || sh->num_blocks <= 0 ||
      sh->num_blocks > INT32_MAX)
    return fail(DP_EINVAL, "chunked_prefill_attention: need max_blocks_per_seq * 16 >= max_context_len and "
                           "0 < num_blocks <= INT32_MAX");
  if (sh->max_context_len > kIdCap * kBS)
    return fail(DP_ENOTSUP, "chunked_prefill_attention: max_context_len above %d", kIdCap * kBS);
  if (sh->total_q < 0 || sh->total_q > INT32_MAX / 2)
    return fail(DP_EINVAL, "chunked_prefill_attention: total_q out of range");
  if (sh->batch == 0 || sh->total_q == 0) return DP_OK;
  if (!q || !k_blocks || !v_blocks || !block_tables || !context_lens || !q_start || !out)
    return fail(DP_EINVAL, "chunked_prefill_attention: null tensor pointer");
  if (((uintptr_t)q | (uintptr_t)k_blocks | (uintptr_t)v_blocks | (uintptr_t)out) & 15)
    return fail(DP_EINVAL, "chunked_prefill_attention: q, k_blocks, v_blocks and out must be 16-byte aligned");
  const bool fp8 = sh->kv_dtype == DP_KV_FP8_E4M3;
  if (fp8 && (!k_scale || !v_scale))
    return fail(DP_EINVAL, "chunked_prefill_attention: e4m3 cache needs k_scale and v_scale");
  if (!fp8 && (k_scale || v_scale))
    return fail(DP_EINVAL, "chunked_prefill_attention: k_scale/v_scale must be NULL for a bf16 cache");
  if (!(scale > 0.0f) || !std::isfinite(scale))
    return fail(DP_EINVAL, "chunked_prefill_attention: scale must be finite and > 0");

  constexpr int QT = 32;  // one eight-wave workgroup per compute unit, two waves per SIMD
  const int group = sh->n_q_heads / sh->n_kv_heads;
  const int nquad = (group + kWaves - 1) / kWaves;
  // an upper bound of sum_s ceil(n_s / QT) items (the kernel counts them exactly)
  const int64_t tiles = (sh->total_q + QT - 1) / QT + sh->batch;
  const int64_t items = tiles * sh->n_kv_heads * nquad;
  if (items > INT32_MAX / 2) return fail(DP_EINVAL, "chunked_prefill_attention: too many query tiles");
  // one persistent workgroup per compute unit (the kernel's registers allow one)
  const int64_t grid = std::min<int64_t>(items, compute_units());

  PrefillArgs a;
  a.q = (const uint16_t*)q;
  a.k = (const char*)k_blocks;
  a.v = (const char*)v_blocks;
  a.block_tables = block_tables;
  a.context_lens = context_lens;
  a.q_start = q_start;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.out = out;
  a.scale_log2 = scale * kLog2e;
  a.batch = sh->batch;
  a.hq = sh->n_q_heads;
  a.hkv = sh->n_kv_heads;
  a.group = group;
  a.nquad = nquad;
  a.max_blocks_per_seq = sh->max_blocks_per_seq;
  a.max_ctx = sh->max_context_len;
  a.num_blocks_m1 = (int32_t)(sh->num_blocks - 1);
  a.out_fp32 = sh->out_dtype == DP_OUT_FP32;
  a.total_q = (int32_t)sh->total_q;
  const size_t dyn = (size_t)(4 * sh->batch + 1) * sizeof(int);  // tile prefix, rows, contexts
  (void)hipGetLastError();
  const dim3 g((unsigned)grid), b(kWaves * 64);
  hipStream_t st = (hipStream_t)stream;
  if (fp8) hipLaunchKernelGGL((prefill_kernel<true, 2>), g, b, dyn, st, a);
  else hipLaunchKernelGGL((prefill_kernel<false, 2>), g, b, dyn, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DP_EIO, "chunked_prefill_attention: kernel launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}
