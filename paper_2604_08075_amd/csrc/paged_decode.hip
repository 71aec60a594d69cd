// Paged decode attention for gfx950 (MI355X).
//
// What it computes: one new query token per sequence attends over that
// sequence's block-paged KV cache - the per-step KV read the paper's cost
// model names as the memory-bandwidth-bound phase (Sec. 3 effect 4, Sec. 4.4
// "Why TPOT also improves"), over 16-token PagedAttention blocks (Sec. 3
// effect 3).  Definition: for sequence s (T = context_lens[s] tokens) and
// query head h with KV head g = h / G,
//     out[s,h] = sum_t softmax_t(scale * q[s,h] . K_t) V_t,
//     K_t = k_blocks[block_tables[s][t/16], g, t%16, :]   (token-major tile)
//     V_t = v_blocks[block_tables[s][t/16], g, :, t%16]   (dims-major tile)
//     times the per-head fp8 scale when the cache is e4m3.
//
// Work decomposition (stream-K over the KV stream).  The cached tokens of
// every (sequence, KV head) "segment" form one flat stream of 16 KiB units
// (two 16-token blocks for bf16, four for fp8), segments in sequence-major,
// head-minor order.  A persistent grid gives every wave one contiguous,
// equal-length slice of that stream, so the load is balanced to one unit
// however skewed the context lengths are.  A wave walks its slice across
// segment boundaries without draining its load pipeline.  A segment that
// lies wholly inside one slice is finished in registers and written to
// `out`; a segment cut by slice boundaries leaves one softmax partial per
// piece (a wave has at most two such pieces: its first and its last), kept
// in the wave's LDS.  After a workgroup barrier each share of a cut segment
// held by the workgroup is merged by one of its waves, with log-sum-exp
// weights; a share that crosses the workgroup's edges then goes through
// device-wide arrival counters, and the workgroup that brings a group's last
// piece merges the group.  Every fold reads its partials in a fixed order
// (deterministic).
//
// A wave's first unit is issued at launch from the tiles it used in the
// previous call on the same workspace (every layer of a decode step but the
// first has the same context lengths and block tables), and loaded again if
// the true tiles, found by the prologue, differ.
//
// Per wave, the hot loop keeps one unit in flight while it computes the
// previous one, with every byte going straight to registers in the layout
// the matrix cores consume (no LDS staging):
//   * K: one 16-byte load per lane per (32-dim chunk, 16-token row group)
//     puts a token row's dims directly into the A operand of
//     v_mfma_f32_16x16x32_bf16; S^T = K Q^T gives 16 tokens x 16 query heads
//     (heads past the GQA group are zero padding), so every query head of
//     the group reuses the tile.  The tokens behind the MFMA rows are
//     permuted so that each lane's score accumulators are exactly the
//     tokens its PV operand needs: probabilities never move between lanes;
//   * V: the dims-major tile gives each lane 8 consecutive tokens of one
//     head dimension per 16-byte load: the A operand of O^T = V^T P^T;
//   * online softmax in base 2 (scale * log2 e folded into one multiply),
//     the per-head max crossing the four 16-lane rows by two lane swaps;
//     the running-max rescale is skipped when no head's max grew;
//   * fp8 e4m3 tiles widen to bf16 exactly (v_cvt_scalef32_pk_bf16_fp8 with
//     scale 1); the per-head K scale folds into the score multiplier, the V
//     scale into the final normalisation.
// Blocks past a sequence's last token are never loaded; tail slots of its
// last block are masked by select (scores to -inf, values to 0), so poisoned
// or stale cache contents cannot leak into the result.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>
#include <type_traits>

#include "common.h"

// Kernels live in a named namespace: hipcc does not emit the host-side launch
// stubs of templated kernels declared in an anonymous namespace.
namespace dpool_hip {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr int kHeadDim = 128;
constexpr int kBlock = 16;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kWaves = 4;              // waves per workgroup
constexpr int kMaxUnitsPerWave = 256;  // the host sizes the grid so that no slice is longer
// A piece's partial stays in its wave's LDS until the merge (no global store
// inside the loop, where stores would share the in-order memory counter with
// the KV loads).
constexpr int kRecBytes = 8192 + 512;  // a record in LDS: eight 1 KiB chunks of o, then (m, l) per lane

struct DecodeArgs {
  const uint16_t* q;            // [B, Hq, 128] bf16
  const char* k;                // [num_blocks, Hkv, 16, 128] bf16 or e4m3
  const char* v;                // [num_blocks, Hkv, 128, 16] bf16 or e4m3
  const int32_t* block_tables;  // [B, max_blocks_per_seq]
  const int32_t* context_lens;  // [B]
  const float* k_scale;         // [Hkv] (fp8)
  const float* v_scale;
  void* out;                    // [B, Hq, 128] bf16 or fp32
  int32_t* arrivals;            // [2, waves]: group and segment arrival counters; zero between calls
  float* rec_ml;                // [3 * waves, G, 2]    (max in log2 units, sum)
  float* rec_o;                 // [3 * waves, G, 128]  partial outputs (normalised, V-scaled)
  int32_t* tile_cache;          // [waves, 4]: tiles of each wave's first unit in the previous call (a hint)
  float qk_scale_log2;          // scale * log2(e)
  int32_t batch, hq, hkv, group;
  int32_t max_blocks_per_seq, max_ctx;
  int32_t num_blocks_m1;        // num_blocks - 1 (block ids are clamped into range)
  int32_t out_fp32;
  int32_t min_chunk;            // minimum units per slice
};

// Unit geometry: a unit is 16 KiB of K and V of one KV head.
template <bool FP8>
struct Geo {
  static constexpr int UB = FP8 ? 4 : 2;          // blocks per unit
  static constexpr int UT = UB * kBlock;          // tokens per unit
  static constexpr int TILE = FP8 ? 2048 : 4096;  // bytes of one (block, head) tile
  static constexpr int NZ = FP8 ? 16 : 8;         // scores per lane per unit
};

// One unit in registers: eight 16-byte K fragments and eight V fragments per lane.
struct UnitRegs {
  i32x4 k[8];
  i32x4 v[8];
};

__device__ __forceinline__ float xor_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float xor_sum(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// Eight e4m3 bytes -> eight bf16 (exact; every e4m3 value is a bf16 value).
__device__ __forceinline__ bf16x8 fp8x8_to_bf16(int lo, int hi) {
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true);
  bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false);
  bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true);
  bf16x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
  return r;
}

// Mask of the live bytes of 32-bit word w of a V fragment whose first nv
// tokens are live: tokens of `per_word` bytes each (2: bf16, 1: fp8), so a
// word holds 4 / per_word tokens.  Dead tokens (past the context, possibly
// NaN-poisoned slots) become +0.
template <int kTokBytes>
__device__ __forceinline__ unsigned live_mask(int w, int nv) {
  constexpr int kPerWord = 4 / kTokBytes;
  const int k = min(max(nv - kPerWord * w, 0), kPerWord);  // live tokens in this word
  return k == kPerWord ? 0xffffffffu : (1u << (8 * kTokBytes * k)) - 1u;
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

__device__ __forceinline__ int clamp_ctx(int c, int max_ctx) { return c < 0 ? 0 : (c > max_ctx ? max_ctx : c); }

template <bool FP8>
__device__ __forceinline__ int units_of(int ctx) {
  return (ctx + Geo<FP8>::UT - 1) / Geo<FP8>::UT;
}

// Partial records cross compute units on different XCDs, whose L2 caches are
// not coherent with each other.  They are written and read with the cache
// policy of an agent-scope atomic access (sc1: written through to, and read
// from, the coherence point), so no L2-wide writeback or invalidate is needed:
// those stall every wave streaming through the same L2.  (m, l) pairs use
// 8-byte agent-scope atomics; the o values use 16-byte buffer accesses with
// the sc1 bit, which halves the instructions of a merge's record reads and
// keeps a round of eight records under the 63 loads a wave can have in flight.
constexpr int kSc1 = 16;                  // buffer cache-policy bit: sc1 (device scope)
constexpr int kBufferWord3 = 0x00020000;  // buffer resource word 3 for gfx9: 32-bit data format
// Record slot `slot` (G * 128 floats) as a buffer resource; its base is the
// same for the whole wave, and an access outside the slot reads zero and
// writes nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t record_rsrc(float* rec_o, size_t slot, int G) {
  const int sl = __builtin_amdgcn_readfirstlane((int)slot);
  return __builtin_amdgcn_make_buffer_rsrc(rec_o + (size_t)sl * G * kHeadDim, (short)0, G * kHeadDim * 4,
                                           kBufferWord3);
}
__device__ __forceinline__ void coherent_store16(__amdgpu_buffer_rsrc_t r, int byte_off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, byte_off, 0, kSc1);
}
__device__ __forceinline__ f32x4 coherent_load16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kSc1);
}
__device__ __forceinline__ void coherent_store2(float* p, float a, float b) {
  typedef unsigned long long u64;
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  __hip_atomic_store((u64*)p, __builtin_bit_cast(u64, f32x2{a, b}), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void coherent_load2(const float* p, float& a, float& b) {
  typedef unsigned long long u64;
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const f32x2 v = __builtin_bit_cast(f32x2, __hip_atomic_load((u64*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  a = v[0];
  b = v[1];
}

// Write 8 consecutive output values (fp32 or bf16) of one row.
__device__ __forceinline__ void store_out8(const DecodeArgs& a, size_t off, f32x4 x0, f32x4 x1) {
  if (a.out_fp32) {
    *(f32x4*)((float*)a.out + off) = x0;
    *(f32x4*)((float*)a.out + off + 4) = x1;
  } else {
    u16x8 o;
    for (int e = 0; e < 4; ++e) {
      o[e] = f32_to_bf16_bits(x0[e]);
      o[4 + e] = f32_to_bf16_bits(x1[e]);
    }
    *(u16x8*)((uint16_t*)a.out + off) = o;
  }
}

// Records (o, m, l): o normalised by l, m in log2 units.  A segment cut by
// slice boundaries is merged in two stages: first inside each workgroup,
// from the records its waves keep in LDS, then across workgroups through
// the workspace.  Slots 2b and 2b + 1 hold workgroup b's
// first and last piece of segments that cross its edges, and
// 2 * workgroups + b the merged record of the group of workgroup pieces
// whose last is workgroup b's.  Workgroup pieces are merged in groups of
// kFanIn consecutive ones, then the group records, so that a segment cut
// into many pieces needs few memory round trips on each level.
constexpr int kFanIn = 16;

// Log-sum-exp fold of records, by one wave, in record order:
// M = max_p m_p, w_p = l_p 2^(m_p - M), o = sum_p w_p o_p / sum_p w_p,
// L = sum_p w_p.  Each lane folds NP (head, 8-value chunk) pairs: NP = 2
// covers the 128 pairs of a GQA group of up to 8 heads, NP = 4 the 256 pairs
// of up to 16, so one pass over the records covers every pair of the group.
template <int NP>
struct Fold {
  float M[NP], L[NP];
  f32x4 o0[NP], o1[NP];
};

// Records fetched per memory round trip: the same registers for either NP.
template <int NP>
constexpr int kRound = 16 / NP;

template <int NP>
__device__ __forceinline__ void fold_init(Fold<NP>& F) {
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    F.M[i] = -INFINITY;
    F.L[i] = 0.f;
    F.o0[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    F.o1[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// Fold records 0 .. n-1 (n the same for the whole wave) in order.
// rec(u, m, l, x0, x1) fetches record u's values for every pair of the lane;
// the fetches of kRound records are issued before any of them is folded.
// Per round: the new maximum first, then one exponential per record and
// o += w x as fused multiply-adds in record order (the running sums are
// rescaled once per round, not once per record).  The order of the sums is
// fixed by the record indices, so the fold is bit-identical whichever wave
// performs it.
template <int NP, int R = kRound<NP>, class Rec>
__device__ __forceinline__ void fold_records(Fold<NP>& F, int n, Rec rec) {
  n = __builtin_amdgcn_readfirstlane(n);
  for (int r0 = 0; r0 < n; r0 += R) {
    float m[R][NP], l[R][NP];
    f32x4 x0[R][NP], x1[R][NP];
#pragma unroll
    for (int u = 0; u < R; ++u)
      if (r0 + u < n) rec(r0 + u, m[u], l[u], x0[u], x1[u]);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      float M2 = F.M[i];
#pragma unroll
      for (int u = 0; u < R; ++u)
        if (r0 + u < n) M2 = fmaxf(M2, m[u][i]);
      if (r0 > 0) {  // the sums so far move to the new maximum
        const float c = __builtin_amdgcn_exp2f(F.M[i] - M2);
        F.o0[i] *= c;
        F.o1[i] *= c;
        F.L[i] *= c;
      }
#pragma unroll
      for (int u = 0; u < R; ++u) {
        if (r0 + u < n) {
          const float wgt = l[u][i] * __builtin_amdgcn_exp2f(m[u][i] - M2);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            F.o0[i][e] = __builtin_fmaf(x0[u][i][e], wgt, F.o0[i][e]);
            F.o1[i][e] = __builtin_fmaf(x1[u][i][e], wgt, F.o1[i][e]);
          }
          F.L[i] += wgt;
        }
      }
      F.M[i] = M2;
    }
  }
}

// The (head, first dim) of each pair of this lane (idle lanes re-read pair 0).
template <int NP>
struct Pairs {
  int hd[NP], d0[NP];
  bool ok[NP];
};

template <int NP>
__device__ __forceinline__ Pairs<NP> pairs_of(int lane, int npairs) {
  Pairs<NP> P;
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int p = lane + 64 * i;
    P.ok[i] = p < npairs;
    const int pp = P.ok[i] ? p : 0;
    P.hd[i] = pp >> 4;
    P.d0[i] = (pp & 15) * 8;
  }
  return P;
}

// Record u from global slot `slot`: (m, l) per head, o as [head][dim].
template <int NP>
__device__ __forceinline__ void fetch_record(const DecodeArgs& a, size_t slot, const Pairs<NP>& P, float (&m)[NP],
                                             float (&l)[NP], f32x4 (&x0)[NP], f32x4 (&x1)[NP]) {
  const int G = a.group;
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int hd = P.hd[i], d0 = P.d0[i];
    coherent_load2(a.rec_ml + (slot * G + hd) * 2, m[i], l[i]);
    const __amdgpu_buffer_rsrc_t r = record_rsrc(a.rec_o, slot, G);
    const int bo = (hd * kHeadDim + d0) * 4;
    x0[i] = coherent_load16(r, bo);
    x1[i] = coherent_load16(r, bo + 16);
  }
}

// Record u from a wave's LDS copy `own`: eight [lane] chunks of 4 floats
// (dims 16 nn + 4 lj .. + 4 of head li at lane li + 16 lj), then each lane's
// (m, l).  Only LDS: a fold whose loop holds no memory load needs no wait for
// loads issued before it.
template <int NP>
__device__ __forceinline__ void fetch_record_lds(const char* own, const Pairs<NP>& P, float (&m)[NP], float (&l)[NP],
                                                 f32x4 (&x0)[NP], f32x4 (&x1)[NP]) {
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int hd = P.hd[i], d0 = P.d0[i];
    const float* ml = (const float*)(own + 8192 + hd * 8);
    m[i] = ml[0];
    l[i] = ml[1];
    const int nn = d0 >> 4, q = (d0 & 15) >> 2;
    x0[i] = *(const f32x4*)(own + nn * 1024 + (hd + 16 * q) * 16);
    x1[i] = *(const f32x4*)(own + nn * 1024 + (hd + 16 * (q + 1)) * 16);
  }
}

// The fold normalised: exactly what a record of it holds (o / L, M, L).
template <int NP>
__device__ __forceinline__ void normalise(const Fold<NP>& F, float (&m)[NP], float (&l)[NP], f32x4 (&x0)[NP],
                                          f32x4 (&x1)[NP]) {
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const float inv = 1.0f / F.L[i];
    x0[i] = F.o0[i] * inv;
    x1[i] = F.o1[i] * inv;
    m[i] = F.M[i];
    l[i] = F.L[i];
  }
}

// Write the fold as the output rows of segment (s, g).
template <int NP>
__device__ __forceinline__ void write_rows(const DecodeArgs& a, const Fold<NP>& F, const Pairs<NP>& P, int s,
                                           int g) {
  const int G = a.group;
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    if (!P.ok[i]) continue;
    const float inv = 1.0f / F.L[i];
    store_out8(a, ((size_t)s * a.hq + (size_t)g * G + P.hd[i]) * kHeadDim + P.d0[i], F.o0[i] * inv,
               F.o1[i] * inv);
  }
}

// Write normalised values as record slot dst.
template <int NP>
__device__ __forceinline__ void write_record(const DecodeArgs& a, const Pairs<NP>& P, size_t dst,
                                             const float (&m)[NP], const float (&l)[NP], const f32x4 (&x0)[NP],
                                             const f32x4 (&x1)[NP]) {
  const int G = a.group;
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    if (!P.ok[i]) continue;
    const __amdgpu_buffer_rsrc_t r = record_rsrc(a.rec_o, dst, G);
    const int bo = (P.hd[i] * kHeadDim + P.d0[i]) * 4;
    coherent_store16(r, bo, x0[i]);
    coherent_store16(r, bo + 16, x1[i]);
    if (P.d0[i] == 0) coherent_store2(a.rec_ml + (dst * G + P.hd[i]) * 2, m[i], l[i]);
  }
}

// Per-wave walker over the flat unit stream: segment (s, g), unit j inside it.
struct Walker {
  int s, g, j, nus;
};

// Inclusive prefix sum over the 64 lanes of a wave, in the vector ALU (no
// LDS round trips): data-parallel-primitive moves shift each 16-lane row
// right by 1, 2, 4 and 8 lanes (a lane with no source adds 0), then lane 15
// of rows 0 and 2 is added into rows 1 and 3, and lane 31 into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
  return x;
}

// A workgroup barrier that waits for LDS accesses only, not for loads or
// stores to memory still in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// a / d for a >= 0, d >= 1 and a quotient below 2^22 (a wave or workgroup
// index): the float estimate is then off by at most one, and one step
// corrects it.  rd = 1 / d, rounded.
__device__ __forceinline__ int div_small(int a, int d, float rd) {
  const int q = (int)((float)a * rd);
  const int r = a - q * d;
  return q + (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
}

template <bool FP8>
__global__ __launch_bounds__(kWaves * 64) void paged_decode_kernel(DecodeArgs a) {
  using GE = Geo<FP8>;
  constexpr int UB = GE::UB, UT = GE::UT, TILE = GE::TILE, NZ = GE::NZ;
  __shared__ int tiles_lds[kWaves][kMaxUnitsPerWave * UB];
  __shared__ int wave_sums[kWaves];
  // Split pieces are first merged inside the workgroup: the segment (s, g)
  // of each wave's first and last split piece (s = -1: none).
  __shared__ int wg_seg[2 * kWaves][2];
  __shared__ __attribute__((aligned(16))) char stage_lds[kWaves][2 * kRecBytes];  // each wave's two records
  extern __shared__ int dyn[];  // pre[B + 1], ctxs[B], k_scale[Hkv], v_scale[Hkv]

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int B = a.batch, Hkv = a.hkv, G = a.group;
  const int li = lane & 15;  // MFMA row / column index
  const int lj = lane >> 4;  // k-group (16-lane row of the wave)
  int* pre = dyn;
  int* ctxs = dyn + B + 1;
  float* kscl = (float*)(dyn + 2 * B + 1);
  float* vscl = kscl + Hkv;

  // ---- per-lane operand offsets inside a tile ----
  int kofs[8], vofs[8];
  int kblk, vblk;  // which block of the unit this lane's K / V fragments come from
  if constexpr (FP8) {
    // K: MFMA m (0..3), row li = token 4m + (li & 3) of block li >> 2; fragment j = dims 64j + 16lj .. +16
    for (int m = 0; m < 4; ++m)
      for (int jj = 0; jj < 2; ++jj) kofs[2 * m + jj] = (4 * m + (li & 3)) * 128 + 64 * jj + 16 * lj;
    kblk = li >> 2;
    // V: dim 16nn + li, all 16 tokens of block lj
    for (int nn = 0; nn < 8; ++nn) vofs[nn] = (16 * nn + li) * 16;
    vblk = lj;
  } else {
    // K: MFMA m (0..1), row li = token 8((li >> 2) & 1) + 4m + (li & 3) of block li >> 3; chunk c = dims 32c + 8lj
    for (int m = 0; m < 2; ++m)
      for (int c = 0; c < 4; ++c) kofs[4 * m + c] = (8 * ((li >> 2) & 1) + 4 * m + (li & 3)) * 256 + 64 * c + 16 * lj;
    kblk = li >> 3;
    // V: dim 16nn + li, tokens 8(lj & 1) .. +8 of block lj >> 1
    for (int nn = 0; nn < 8; ++nn) vofs[nn] = (16 * nn + li) * 32 + 16 * (lj & 1);
    vblk = lj >> 1;
  }
  auto issue_at = [&](UnitRegs& R, int kt, int vt) __attribute__((always_inline)) {
    const char* kb = a.k + (size_t)kt * TILE;
    const char* vb = a.v + (size_t)vt * TILE;
#pragma unroll
    for (int x = 0; x < 8; ++x) R.k[x] = __builtin_nontemporal_load((const i32x4*)(kb + kofs[x]));
#pragma unroll
    for (int x = 0; x < 8; ++x) R.v[x] = __builtin_nontemporal_load((const i32x4*)(vb + vofs[x]));
  };

  // ---- 0. the first unit's loads, from the tiles of the previous call ----
  // Every layer of a decode step but the first repeats the previous call's
  // context lengths and block tables, and with them each wave's first unit.
  // A wave keeps that unit's tile indices in the workspace and issues the
  // unit's loads from them right away, while the prologue finds the true
  // tiles; if they differ, it loads the unit again.  The kept indices are
  // clamped into the pool, so whatever the workspace holds only decides
  // whether the early loads are of use.
  const int gw = blockIdx.x * kWaves + w;
  const int tmax = (a.num_blocks_m1 + 1) * Hkv - 1;
  const int ck = min(max(a.tile_cache[(size_t)gw * 4 + kblk], 0), tmax);
  const int cv = min(max(a.tile_cache[(size_t)gw * 4 + vblk], 0), tmax);
  UnitRegs RA;

  // ---- 1. prefix of units over sequences (every workgroup computes it) ----
  {
    const int T = kWaves * 64, tid = threadIdx.x;
    if constexpr (FP8) {
      for (int i = tid; i < Hkv; i += T) {
        kscl[i] = a.k_scale[i];
        vscl[i] = a.v_scale[i];
      }
    }
    const int per = (B + T - 1) / T;
    int local = 0;
    for (int k = 0; k < per; ++k) {
      const int s = tid * per + k;
      if (s < B) {
        const int c = clamp_ctx(a.context_lens[s], a.max_ctx);
        ctxs[s] = c;
        local += units_of<FP8>(c);
      }
    }
    issue_at(RA, ck, cv);
    const int incl = wave_incl_scan(local);
    if (lane == 63) wave_sums[w] = incl;
    lds_barrier();  // (LDS only: the first unit's loads stay in flight)
    int run = incl - local;
    for (int k = 0; k < w; ++k) run += wave_sums[k];
    for (int k = 0; k < per; ++k) {
      const int s = tid * per + k;
      if (s < B) {
        pre[s] = run;
        run += units_of<FP8>(ctxs[s]);
      }
    }
    if (tid == T - 1) pre[B] = run;
    lds_barrier();
  }
  const int U = Hkv * pre[B];
  const int TW = gridDim.x * kWaves;
  int C = (U + TW - 1) / TW;
  if (C < a.min_chunk) C = a.min_chunk;
  const float rC = 1.0f / (float)C, rCW = 1.0f / (float)(kWaves * C);  // for the merge's slice arithmetic

  // rows of empty sequences are zero
  for (int s = gw; s < B; s += TW) {
    if (ctxs[s] == 0) {
      const size_t row0 = (size_t)s * a.hq * kHeadDim;
      for (int e = lane * 8; e < a.hq * kHeadDim; e += 64 * 8)
        store_out8(a, row0 + e, f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f});
    }
  }

  // Waves take consecutive slices: a workgroup whose first wave has no units
  // has none at all, and leaves as a whole (a barrier follows the walk).
  if ((int)blockIdx.x * kWaves * C >= U) return;
  const int u0 = gw * C;
  const int u1 = min(u0 + C, U);
  // split segments this wave must signal: (s, g) of its first piece and of its last piece, s = -1 if none
  int arr_s0 = -1, arr_g0 = 0, arr_s1 = -1, arr_g1 = 0;
  if (u0 < u1) {  // a wave without units goes straight to the merge
    const int n = u1 - u0;

    // ---- 2. tile indices (block id * Hkv + head) of this wave's units ----
    int* tiles = tiles_lds[w];
    int f_s = 0, f_nus = 1, f_g = 0, f_j = 0;  // the position of unit u0 + lane (lane 0: the slice's first unit)
    for (int i = lane; i < n; i += 64) {
      const int u = u0 + i;
      int lo = 0, hi = B - 1;  // largest s with Hkv * pre[s] <= u
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (Hkv * pre[mid] <= u) lo = mid;
        else hi = mid - 1;
      }
      const int s = lo;
      const int nus = pre[s + 1] - pre[s];
      const int r = u - Hkv * pre[s];
      const int g = r / nus;
      const int j = r - g * nus;
      if (i == lane) {
        f_s = s;
        f_nus = nus;
        f_g = g;
        f_j = j;
      }
      const int nb = (ctxs[s] + kBlock - 1) / kBlock;
      for (int b = 0; b < UB; ++b) {
        // a block past the sequence's end is never fetched: its lanes re-read the
        // unit's first block (same addresses as other lanes of the same load
        // instruction, so no extra memory traffic) and its tokens are masked
        const int blk = j * UB + (j * UB + b < nb ? b : 0);
        int id = a.block_tables[(size_t)s * a.max_blocks_per_seq + blk];
        id = id < 0 ? 0 : (id > a.num_blocks_m1 ? a.num_blocks_m1 : id);
        tiles[i * UB + b] = id * Hkv + g;
      }
    }
    // the early loads were of the first unit's true tiles, or it is loaded again
    if (__ballot(tiles[kblk] != ck || tiles[vblk] != cv)) issue_at(RA, tiles[kblk], tiles[vblk]);
    if (lane < UB) a.tile_cache[(size_t)gw * 4 + lane] = tiles[lane];

    // query fragment c of head li: the dims its K fragment holds.  Columns past
    // the GQA group repeat a real head; they only ever affect their own
    // (unwritten) output columns.
    int qoff[4];
    for (int c = 0; c < 4; ++c) qoff[c] = FP8 ? 64 * (c >> 1) + 16 * lj + 8 * (c & 1) : 32 * c + 8 * lj;
    const int qhead = li < G ? li : li % G;

    // ---- 4. walk the slice ----
    Walker cs;  // compute side: the slice's first unit, as lane 0 located it above
    cs.s = __builtin_amdgcn_readlane(f_s, 0);
    cs.nus = __builtin_amdgcn_readlane(f_nus, 0);
    cs.g = __builtin_amdgcn_readlane(f_g, 0);
    cs.j = __builtin_amdgcn_readlane(f_j, 0);
    auto advance = [&](Walker& wk) __attribute__((always_inline)) {
      if (++wk.j == wk.nus) {
        wk.j = 0;
        if (++wk.g == Hkv) {
          wk.g = 0;
          do {
            ++wk.s;
          } while (wk.s < B - 1 && pre[wk.s + 1] == pre[wk.s]);  // skip empty sequences (bounded)
          // Stepping off the last sequence only happens to a look-ahead
          // position past the end of the stream (never computed); it stays on
          // the last sequence so that the query rows it prefetches exist.
          wk.s = __builtin_amdgcn_readfirstlane(wk.s > B - 1 ? B - 1 : wk.s);
        }
        wk.nus = __builtin_amdgcn_readfirstlane(pre[wk.s + 1] - pre[wk.s]);
      }
    };
    // Every load in the loop is unconditional, so the compiler's wait counts
    // stay exact: a wait for one unit never drains the unit behind it.
    auto load_q = [&](i32x4 (&qr)[4], int s, int g) __attribute__((always_inline)) {
      const uint16_t* qrow = a.q + ((size_t)s * a.hq + (size_t)g * G + qhead) * kHeadDim;
      for (int c = 0; c < 4; ++c) qr[c] = *(const i32x4*)(qrow + qoff[c]);
    };
    auto issue = [&](UnitRegs& R, int ui) __attribute__((always_inline)) {
      issue_at(R, tiles[ui * UB + kblk], tiles[ui * UB + vblk]);
    };

    // ---- the records of this wave's split pieces, in LDS ----
    // At most two: the slice's first piece (x = 0) at offset 0, its last
    // (x = 1) at kRecBytes.  Layout: eight 1 KiB chunks of o ([nn][lane], 16
    // bytes per lane), then each lane's (m, l).  They stay there for the merge.
    char* const stg = stage_lds[w];

    i32x4 qv[4];          // query group of the piece being computed
    i32x4 qE[4], qO[4];   // query groups of the segments of the next even / odd unit
    float m_run = -INFINITY, l_part = 0.f, cscale = 0.f, vsc = 1.0f;
    f32x4 acc[8];
    for (int nn = 0; nn < 8; ++nn) acc[nn] = f32x4{0.f, 0.f, 0.f, 0.f};
    int piece_j0 = 0, ctx_s = 0;
    bool piece_first = true;

    auto begin_piece = [&](int ui, const i32x4 (&qs)[4]) __attribute__((always_inline)) {
      if (ui == 0 || cs.j == 0) {  // a new piece starts: its query group, fresh softmax state
        piece_first = ui == 0;
        piece_j0 = cs.j;
        ctx_s = __builtin_amdgcn_readfirstlane(ctxs[cs.s]);
#pragma unroll
        for (int c = 0; c < 4; ++c) qv[c] = qs[c];
        float ksc = 1.0f;
        if constexpr (FP8) {
          ksc = kscl[cs.g];
          vsc = vscl[cs.g];
        }
        cscale = a.qk_scale_log2 * ksc;
        m_run = -INFINITY;
        l_part = 0.f;
#pragma unroll
        for (int nn = 0; nn < 8; ++nn) acc[nn] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };

    auto compute_unit = [&](const UnitRegs& R) __attribute__((always_inline)) {
      const int unit_tok0 = cs.j * UT;
      const bool ragged = unit_tok0 + UT > ctx_s;
      const int lane_tok0 = unit_tok0 + (FP8 ? 16 : 8) * lj;  // first unit token of this lane's scores

      // S^T = K Q^T: lane (li, lj) holds scores of head li for its NZ tokens
      float z[NZ];
      if constexpr (FP8) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const i32x4 raw = R.k[2 * m + jj];
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(raw[0], raw[1]),
                                                           __builtin_bit_cast(bf16x8, qv[2 * jj]), sacc, 0, 0, 0);
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(raw[2], raw[3]),
                                                           __builtin_bit_cast(bf16x8, qv[2 * jj + 1]), sacc, 0, 0,
                                                           0);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) z[4 * m + e] = sacc[e] * cscale;
        }
      } else {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < 4; ++c)
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, R.k[4 * m + c]),
                                                           __builtin_bit_cast(bf16x8, qv[c]), sacc, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) z[4 * m + e] = sacc[e] * cscale;
        }
      }
      // live tokens among this lane's NZ tokens (all of them unless the unit is ragged)
      const int nv = ragged ? min(max(ctx_s - lane_tok0, 0), NZ) : NZ;
      if (ragged)
#pragma unroll
        for (int e = 0; e < NZ; ++e)
          if (e >= nv) z[e] = -INFINITY;

      // online softmax (base 2) for head li over this unit's tokens
      float bmax = z[0];
      for (int e = 1; e < NZ; ++e) bmax = fmaxf(bmax, z[e]);
      bmax = xor_max(bmax);
      const float m_new = fmaxf(m_run, bmax);
      if (__builtin_amdgcn_ballot_w64(m_new > m_run) != 0) {  // some head's max grew: rescale
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_part *= alpha;
#pragma unroll
        for (int nn = 0; nn < 8; ++nn) acc[nn] *= alpha;
        m_run = m_new;
      }
      bf16x8 p[NZ / 8];
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < NZ; ++e) {
        const __bf16 pe = (__bf16)__builtin_amdgcn_exp2f(z[e] - m_run);
        p[e >> 3][e & 7] = pe;
        psum += (float)pe;
      }
      l_part += psum;

      // O^T += V^T P^T.  A V fragment is 16 bytes: 8 bf16 tokens, or 16 fp8
      // tokens (8 for each of two MFMAs); dead tokens are zeroed on the raw words.
      unsigned vmask[4] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
      if (ragged)
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) vmask[wd] = live_mask<FP8 ? 1 : 2>(wd, nv);
#pragma unroll
      for (int nn = 0; nn < 8; ++nn) {
        i32x4 raw = R.v[nn];
        if (ragged)
#pragma unroll
          for (int wd = 0; wd < 4; ++wd) raw[wd] &= (int)vmask[wd];
        if constexpr (FP8) {
          acc[nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(raw[0], raw[1]), p[0], acc[nn], 0, 0, 0);
          acc[nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fp8x8_to_bf16(raw[2], raw[3]), p[1], acc[nn], 0, 0, 0);
        } else {
          acc[nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, raw), p[0], acc[nn], 0, 0, 0);
        }
      }
    };

    // End of a piece: its rows (whole segment) or its partial record.
    auto finish_piece = [&](int ui) __attribute__((always_inline)) {
      const bool seg_end = cs.j == cs.nus - 1;
      if (!(seg_end || ui == n - 1)) return;
      const float l_tot = xor_sum(l_part);
      const float inv = vsc / l_tot;
      if (piece_j0 == 0 && seg_end) {  // the whole segment: final output, written straight out
        // (these stores follow the loads of the next unit, and a wait for any
        // later load comes a unit's computation after them)
        if (li < G) {
          const size_t row = ((size_t)cs.s * a.hq + (size_t)cs.g * G + li) * kHeadDim + 4 * lj;
#pragma unroll
          for (int nn = 0; nn < 8; ++nn) {
            const f32x4 o = acc[nn] * inv;
            if (a.out_fp32) {
              *(f32x4*)((float*)a.out + row + 16 * nn) = o;
            } else {
              u16x4 ob;
#pragma unroll
              for (int e = 0; e < 4; ++e) ob[e] = f32_to_bf16_bits(o[e]);
              *(u16x4*)((uint16_t*)a.out + row + 16 * nn) = ob;
            }
          }
        }
      } else {  // a piece of a segment cut by slice boundaries
        char* base = stg + (piece_first ? 0 : kRecBytes);
#pragma unroll
        for (int nn = 0; nn < 8; ++nn) *(f32x4*)(base + nn * 1024 + lane * 16) = acc[nn] * inv;
        float* ml = (float*)(base + 8192 + lane * 8);
        ml[0] = m_run;
        ml[1] = l_tot;
        if (piece_first) {
          arr_s0 = cs.s;
          arr_g0 = cs.g;
        } else {
          arr_s1 = cs.s;
          arr_g1 = cs.g;
        }
      }
    };

    // One unit in flight while the previous one is computed.  Per step, in
    // program order: the K and V tiles of unit u+1; at the start of a piece,
    // the query group of unit u's segment copied out of the ring slot of u's
    // parity; the computation of unit u; then, only if unit u+2 starts a
    // segment, its query group loaded into that slot.  The loop is unrolled by
    // two so that the unit buffers and query slots are static, runs pairs of
    // units with no exit in its body, and peels the last unit or two: with an
    // exit inside the body, or a conditional load placed before a wait that it
    // would join, the compiler's wait counts turn conservative and it drains
    // every load in flight.
    Walker w1 = cs, w2;  // positions of units u+1 and u+2
    advance(w1);
    w2 = w1;
    advance(w2);
    UnitRegs RB;  // (RA holds the first unit)
    load_q(qE, cs.s, cs.g);
    load_q(qO, w1.s, w1.g);
    auto step = [&](UnitRegs& cur, UnitRegs& nxt, i32x4 (&qs)[4], int ui) __attribute__((always_inline)) {
      issue(nxt, ui + 1);
      // keep the compiler's scheduler from hoisting the computation of unit u
      // above these loads (it would wait for unit u before issuing unit u+1)
      __builtin_amdgcn_sched_barrier(0);
      begin_piece(ui, qs);
      compute_unit(cur);
      // Unit u's operands are consumed.  If unit u+2 starts a segment, load its
      // query group into the slot just freed: a full step passes before any
      // wait can cover this (conditional) load.
      if (w2.j == 0) load_q(qs, w2.s, w2.g);
      finish_piece(ui);
      cs = w1;
      w1 = w2;
      advance(w2);
    };
    auto last = [&](UnitRegs& cur, const i32x4 (&qs)[4], int ui) __attribute__((always_inline)) {
      begin_piece(ui, qs);
      compute_unit(cur);
      finish_piece(ui);
    };
    int ui = 0;
    for (; ui + 2 < n; ui += 2) {
      step(RA, RB, qE, ui);
      step(RB, RA, qO, ui + 1);
    }
    if (ui + 1 < n) {  // two units left: the last one lands in RB; move it (and its query slot) over
      step(RA, RB, qE, ui);
      ++ui;
      RA = RB;
#pragma unroll
      for (int c = 0; c < 4; ++c) qE[c] = qO[c];
    }
    last(RA, qE, ui);
  }

  // ---- 5. merge the split pieces ----
  // Stage 1, inside the workgroup: after a barrier every wave's records are
  // in LDS, and the workgroup's shares of cut segments are merged at once,
  // each by one wave, which folds the share's pieces in order from their
  // owners' LDS.  A segment entirely inside the workgroup is then written;
  // the share of a segment that crosses the workgroup's edges is the
  // workgroup's piece for stage 2.
  // Stage 2, across workgroups: workgroup pieces are merged in groups of
  // kFanIn consecutive ones, then the groups, by the last arrival on
  // device-wide counters (the workgroup of a group's last piece, of a
  // segment's last piece).  The folds take records in a fixed order, so the
  // result does not depend on which wave performs them.
  int* const group_base = a.arrivals;
  int* const seg_base = a.arrivals + TW;
  auto group_cnt = [&](int k) __attribute__((always_inline)) { return group_base + k; };
  auto seg_cnt = [&](int k) __attribute__((always_inline)) { return seg_base + k; };
  const int wg_first = gw - w;          // first wave of this workgroup
  const int nwg = (int)gridDim.x;
  const int CW = kWaves * C;            // units per workgroup
  const size_t rec_wg = 0;                             // workgroup piece slots
  const size_t rec_grp = rec_wg + (size_t)2 * nwg;     // group record slots
  struct Part {
    int s, g, k0, first_slot, pk0, pkend;              // the segment's waves; this workgroup's share of them
    int bk0, bkend, nwp, first_wslot, rb, gfirst, gn, kg, ngroups;  // its workgroups
  };
  auto part_of = [&](int s, int g) __attribute__((always_inline)) {
    Part p;
    // the same for the whole wave: scalar registers, scalar branches
    const int nus = __builtin_amdgcn_readfirstlane(pre[s + 1] - pre[s]);
    const int a0 = __builtin_amdgcn_readfirstlane(Hkv * pre[s] + g * nus);  // first unit of the segment
    p.s = s;
    p.g = g;
    p.k0 = div_small(a0, C, rC);
    const int kend = div_small(a0 + nus - 1, C, rC);
    p.first_slot = 2 * p.k0 + (a0 > p.k0 * C ? 1 : 0);
    p.pk0 = max(p.k0, wg_first);
    p.pkend = min(kend, wg_first + kWaves - 1);
    p.bk0 = div_small(a0, CW, rCW);
    p.bkend = div_small(a0 + nus - 1, CW, rCW);
    p.nwp = p.bkend - p.bk0 + 1;
    p.first_wslot = 2 * p.bk0 + (a0 > p.bk0 * CW ? 1 : 0);
    p.rb = (int)blockIdx.x - p.bk0;
    p.gfirst = p.rb - p.rb % kFanIn;
    p.gn = min(p.nwp, p.gfirst + kFanIn) - p.gfirst;
    p.kg = p.bk0 + p.gfirst + p.gn - 1;
    p.ngroups = (p.nwp + kFanIn - 1) / kFanIn;
    return p;
  };
  // Piece x = 0 is a slice's first split piece, x = 1 its last; its record
  // is at x * kRecBytes in the wave's LDS.
  if (lane == 0) {
    wg_seg[2 * w][0] = arr_s0;
    wg_seg[2 * w][1] = arr_g0;
    wg_seg[2 * w + 1][0] = arr_s1;
    wg_seg[2 * w + 1][1] = arr_g1;
  }
  // Every record and entry of the workgroup is in LDS after this barrier (it
  // waits for LDS accesses only, not for the rows' stores to memory).
  lds_barrier();
  // The shares are the runs of equal segments among the entries (wave, x),
  // in order: at most kWaves + 1, as each crosses one of the workgroup's
  // kWaves + 1 slice boundaries.  Share i goes to wave min(pos, kWaves - 1),
  // pos = 0 for the first share, 1 for the last, i + 1 for the others: the
  // only shares that can cross the workgroup's edges and go on to stage 2,
  // the first and the last, run on different waves.  Lane e looks at entry
  // e: it starts a share if it is valid and differs from the closest valid
  // entry before it.
  int ms0 = 0, mg0 = 0, ms1 = 0, mg1 = 0;  // this wave's shares, in order
  int mine = 0;
  {
    int es = -1, eg = 0;
    if (lane < 2 * kWaves) {
      es = wg_seg[lane][0];
      eg = wg_seg[lane][1];
    }
    const unsigned long long below = (1ull << lane) - 1;
    const unsigned long long valid = __ballot(es >= 0);
    const unsigned long long vb = valid & below;
    const int prev = vb ? 63 - __clzll(vb) : lane;
    const int ps = __shfl(es, prev), pg = __shfl(eg, prev);
    const bool start = es >= 0 && (vb == 0 || ps != es || pg != eg);
    const unsigned long long starts = __ballot(start);
    const int nsh = __popcll(starts);
    const int i = __popcll(starts & below);
    const int pos = i == 0 ? 0 : (i == nsh - 1 ? 1 : i + 1);
    const unsigned long long my = __ballot(start && min(pos, kWaves - 1) == w);
    mine = __popcll(my);
    const int l0 = my ? __ffsll(my) - 1 : 0;
    const unsigned long long my1 = my & (my - 1);
    const int l1 = my1 ? __ffsll(my1) - 1 : 0;
    ms0 = __builtin_amdgcn_readlane(es, l0);
    mg0 = __builtin_amdgcn_readlane(eg, l0);
    ms1 = __builtin_amdgcn_readlane(es, l1);
    mg1 = __builtin_amdgcn_readlane(eg, l1);
  }
  if (mine == 0) return;

  // A device-wide counter is returned to zero by its last arrival, after
  // this wave's merges: no other wave touches it again in this launch, and a
  // store ahead of the record loads would make their wait include the
  // store's write-through (a wave's memory counter retires loads and stores
  // in issue order).  The group and segment counters of the wave's shares
  // x = 0, 1 that it was the last arrival of (-1: none; scalars, as an array
  // indexed by x would live in scratch memory):
  int rz_g0 = -1, rz_g1 = -1, rz_s0 = -1, rz_s1 = -1;
  auto merge = [&](auto np_c) __attribute__((always_inline)) {
    constexpr int NP = decltype(np_c)::value;
    const Pairs<NP> P = pairs_of<NP>(lane, G * 16);
    for (int x = 0; x < mine; ++x) {
      const Part p = part_of(x == 0 ? ms0 : ms1, x == 0 ? mg0 : mg1);
      // stage 1: the workgroup's pieces of the segment, in order
      Fold<NP> Fw;
      fold_init(Fw);
      // (at most one piece per wave of the workgroup: one round of kWaves)
      fold_records<NP, kWaves>(Fw, p.pkend - p.pk0 + 1, [&](int r, float(&m)[NP], float(&l)[NP], f32x4(&x0)[NP],
                                                          f32x4(&x1)[NP]) __attribute__((always_inline)) {
        const int k = p.pk0 + r;
        const int x = k == p.k0 ? (p.first_slot & 1) : 0;  // the wave's first or last piece
        const int ow = __builtin_amdgcn_readfirstlane(k - wg_first);
        fetch_record_lds((const char*)stage_lds[ow] + x * kRecBytes, P, m, l, x0, x1);
      });
      if (p.nwp == 1) {  // the segment lies inside the workgroup
        write_rows(a, Fw, P, p.s, p.g);
        continue;
      }
      // stage 2: this workgroup's piece, as it would be stored
      float wm[NP], wl[NP];
      f32x4 wx0[NP], wx1[NP];
      normalise(Fw, wm, wl, wx0, wx1);
      auto wslot = [&](int r) __attribute__((always_inline)) {
        return rec_wg + (r == 0 ? (size_t)p.first_wslot : (size_t)2 * (p.bk0 + r));
      };
      auto own_or = [&](bool own, size_t slot, const float(&om)[NP], const float(&ol)[NP], const f32x4(&ox0)[NP],
                        const f32x4(&ox1)[NP], float(&m)[NP], float(&l)[NP], f32x4(&x0)[NP], f32x4(&x1)[NP])
                        __attribute__((always_inline)) {
        if (own) {
#pragma unroll
          for (int i = 0; i < NP; ++i) {
            m[i] = om[i];
            l[i] = ol[i];
            x0[i] = ox0[i];
            x1[i] = ox1[i];
          }
        } else {
          fetch_record(a, slot, P, m, l, x0, x1);
        }
      };
      // A group counter that already shows every other workgroup piece of
      // the group (an atomic load, far quicker than an increment's round
      // trip) cannot change: this workgroup's piece is the last, and it merges
      // from registers without storing its record or counting it.
      int c = 0;
      if (lane == 0) c = __hip_atomic_load(group_cnt(p.kg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (__shfl(c, 0) != p.gn - 1) {  // not yet the group's last arrival: publish and count
        write_record(a, P, wslot(p.rb), wm, wl, wx0, wx1);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        int old = 0;
        if (lane == 0) old = __hip_atomic_fetch_add(group_cnt(p.kg), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__shfl(old, 0) != p.gn - 1) continue;
        asm volatile("" ::: "memory");  // record loads are issued after this branch resolves
      }
      if (x == 0) rz_g0 = p.kg;
      else rz_g1 = p.kg;
      // the group's workgroup pieces, in order (this workgroup's from registers)
      const int own_u = p.rb - p.gfirst;
      Fold<NP> Fg;
      fold_init(Fg);
      fold_records(Fg, p.gn, [&](int u, float(&m)[NP], float(&l)[NP], f32x4(&x0)[NP], f32x4(&x1)[NP])
                                 __attribute__((always_inline)) {
                                   own_or(u == own_u, wslot(p.gfirst + u), wm, wl, wx0, wx1, m, l, x0, x1);
                                 });
      if (p.ngroups == 1) {  // the group is the whole segment
        write_rows(a, Fg, P, p.s, p.g);
        continue;
      }
      // Two levels.  This group's record, as it would be stored:
      float gm[NP], gl[NP];
      f32x4 gx0[NP], gx1[NP];
      normalise(Fg, gm, gl, gx0, gx1);
      auto group_slot = [&](int c) __attribute__((always_inline)) {
        return rec_grp + p.bk0 + min(p.nwp, (c + 1) * kFanIn) - 1;
      };
      // If every other group of the segment is merged by now (checked after
      // this group's fold, so that the others had that long to finish),
      // finish the segment from here: no group record, no wait for its
      // store, no second counter round trip.  Bit-identical to the path
      // through memory.
      int done = 0;
      if (lane == 0) done = __hip_atomic_load(seg_cnt(p.bkend), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int c_own = p.gfirst / kFanIn;
      if (__shfl(done, 0) != p.ngroups - 1) {
        write_record(a, P, rec_grp + p.kg, gm, gl, gx0, gx1);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        int old = 0;
        if (lane == 0) old = __hip_atomic_fetch_add(seg_cnt(p.bkend), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__shfl(old, 0) != p.ngroups - 1) continue;
      }
      asm volatile("" ::: "memory");  // group record loads are issued after this branch resolves
      if (x == 0) rz_s0 = p.bkend;
      else rz_s1 = p.bkend;
      Fold<NP> F;
      fold_init(F);
      fold_records(F, p.ngroups, [&](int u, float(&m)[NP], float(&l)[NP], f32x4(&x0)[NP], f32x4(&x1)[NP])
                                     __attribute__((always_inline)) {
                                       own_or(u == c_own, group_slot(u), gm, gl, gx0, gx1, m, l, x0, x1);
                                     });
      write_rows(a, F, P, p.s, p.g);
    }
  };
  if (G > 8)
    merge(std::integral_constant<int, 4>{});
  else
    merge(std::integral_constant<int, 2>{});
  if (lane == 0) {
    if (rz_g0 >= 0) __hip_atomic_store(group_cnt(rz_g0), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (rz_g1 >= 0) __hip_atomic_store(group_cnt(rz_g1), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (rz_s0 >= 0) __hip_atomic_store(seg_cnt(rz_s0), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (rz_s1 >= 0) __hip_atomic_store(seg_cnt(rz_s1), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template __global__ void paged_decode_kernel<false>(DecodeArgs);
template __global__ void paged_decode_kernel<true>(DecodeArgs);

// Zero n words (arrival counters).  A kernel rather than a memset, so that a
// captured graph holds no memset node.
__global__ __launch_bounds__(256) void zero_words_kernel(int32_t* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

}  // namespace dpool_hip

namespace {

using namespace dpool_hip;

constexpr int kMaxBatchInLds = 4096;  // the unit prefix of the batch is kept in LDS
constexpr int kMaxWorkgroupsPerCu = 8;
constexpr size_t kLdsBytes = 160 * 1024;

// Compute units of the current device (cached per device); 256 when no device
// is visible, so that host-only callers still get a deterministic answer.
int device_cus(int* dev_out) {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    *dev_out = -1;
    return 256;
  }
  *dev_out = dev;
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

// Workgroups of the kernel one compute unit holds at once (register-limited;
// runtime occupancy query, cached).  Without a device: 1.
int resident_per_cu(int dev, bool fp8) {
  static std::mutex mu;
  static int cached[64][2] = {};
  if (dev < 0) return 1;
  std::lock_guard<std::mutex> lock(mu);
  int& occ = cached[dev][fp8 ? 1 : 0];
  if (!occ) {
    int n = 0;
    const void* fn = fp8 ? (const void*)paged_decode_kernel<true> : (const void*)paged_decode_kernel<false>;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kWaves * 64, 0) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      n = 1;
    }
    occ = n;
  }
  return occ;
}

struct Plan {
  int unit_tokens;  // tokens per unit (32 bf16, 64 fp8)
  int min_chunk;    // minimum units per slice
  int grid;         // workgroups
  size_t dyn_lds;   // dynamic LDS bytes
  size_t arrivals_off, rec_ml_off, rec_o_off, tile_cache_off, ws_bytes;
  int clear_words;  // arrival counters to zero before the launch (0 on the usual path)
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int validate(const dp_decode_shape* sh, Plan* plan) {
  using dpool::fail;
  if (!sh) return fail(DP_EINVAL, "paged_decode: null shape");
  if (sh->head_dim != kHeadDim) return fail(DP_ENOTSUP, "paged_decode: head_dim %d (only 128)", sh->head_dim);
  if (sh->block_size != kBlock) return fail(DP_ENOTSUP, "paged_decode: block_size %d (only 16)", sh->block_size);
  if (sh->kv_dtype != DP_KV_BF16 && sh->kv_dtype != DP_KV_FP8_E4M3)
    return fail(DP_ENOTSUP, "paged_decode: kv_dtype %d", sh->kv_dtype);
  if (sh->out_dtype != DP_OUT_BF16 && sh->out_dtype != DP_OUT_FP32)
    return fail(DP_ENOTSUP, "paged_decode: out_dtype %d", sh->out_dtype);
  if (sh->reserved != 0) return fail(DP_EINVAL, "paged_decode: reserved must be 0");
  if (sh->batch < 0) return fail(DP_EINVAL, "paged_decode: batch %d < 0", sh->batch);
  if (sh->batch > kMaxBatchInLds)
    return fail(DP_ENOTSUP, "paged_decode: batch %d > %d sequences per call", sh->batch, kMaxBatchInLds);
  if (sh->n_q_heads <= 0 || sh->n_kv_heads <= 0 || sh->n_kv_heads > 65535 || sh->n_q_heads % sh->n_kv_heads)
    return fail(DP_EINVAL, "paged_decode: n_q_heads %d must be a positive multiple of n_kv_heads %d",
                sh->n_q_heads, sh->n_kv_heads);
  if (sh->n_q_heads / sh->n_kv_heads > 16)
    return fail(DP_ENOTSUP, "paged_decode: GQA group %d > 16", sh->n_q_heads / sh->n_kv_heads);
  if (sh->max_blocks_per_seq <= 0 || sh->max_context_len < 0 ||
      (int64_t)sh->max_context_len > (int64_t)sh->max_blocks_per_seq * kBlock)
    return fail(DP_EINVAL, "paged_decode: max_context_len %d must be in [0, 16 * max_blocks_per_seq = %lld]",
                sh->max_context_len, (long long)sh->max_blocks_per_seq * kBlock);
  if (sh->num_blocks <= 0 || sh->num_blocks * (int64_t)sh->n_kv_heads > INT32_MAX)
    return fail(DP_EINVAL, "paged_decode: num_blocks %lld (num_blocks * n_kv_heads must fit int32)",
                (long long)sh->num_blocks);
  const bool fp8 = sh->kv_dtype == DP_KV_FP8_E4M3;
  const int unit = fp8 ? 64 : 32;
  const int P = sh->partition_tokens;
  if (P < 0 || P % unit || P / unit > kMaxUnitsPerWave)
    return fail(DP_EINVAL, "paged_decode: partition_tokens %d must be a multiple of %d in [0, %d]", P, unit,
                unit * kMaxUnitsPerWave);
  const int wpc = sh->workgroups_per_cu;
  if (wpc < 0 || wpc > kMaxWorkgroupsPerCu)
    return fail(DP_EINVAL, "paged_decode: workgroups_per_cu %d outside [0, %d]", wpc, kMaxWorkgroupsPerCu);
  const int64_t units_per_seq = ((int64_t)sh->max_context_len + unit - 1) / unit;
  const int64_t max_units = units_per_seq * sh->batch * sh->n_kv_heads;
  if (max_units > INT32_MAX) return fail(DP_ENOTSUP, "paged_decode: %lld units exceed int32", (long long)max_units);
  plan->unit_tokens = unit;
  plan->min_chunk = P ? P / unit : 1;
  // LDS per workgroup: the kernel's static arrays (tile lists, wave sums,
  // each wave's two records, the workgroup's merge counters, with 256 bytes
  // for alignment) +
  // unit prefix, context lengths and fp8 scales (dynamic)
  const size_t stat = (size_t)kWaves * kMaxUnitsPerWave * (fp8 ? 4 : 2) * sizeof(int) + kWaves * sizeof(int) +
                      (size_t)kWaves * 2 * kRecBytes + (size_t)4 * kWaves * sizeof(int) + 256;
  plan->dyn_lds = (size_t)(2 * sh->batch + 1 + 2 * sh->n_kv_heads) * 4;
  if (stat + plan->dyn_lds > kLdsBytes)
    return fail(DP_ENOTSUP, "paged_decode: %zu bytes of LDS per workgroup", stat + plan->dyn_lds);
  int dev = -1;
  const int cus = device_cus(&dev);
  const int per_cu = wpc ? std::min(wpc, resident_per_cu(dev, fp8)) : 1;
  // persistent grid (every workgroup resident at once), grown only if some
  // slice would exceed kMaxUnitsPerWave, shrunk when slices would be shorter
  // than the minimum
  int64_t grid = (int64_t)cus * per_cu;
  const int64_t need = (max_units + (int64_t)kWaves * kMaxUnitsPerWave - 1) / ((int64_t)kWaves * kMaxUnitsPerWave);
  const int64_t useful = (max_units + (int64_t)kWaves * plan->min_chunk - 1) / ((int64_t)kWaves * plan->min_chunk);
  grid = std::max<int64_t>(1, std::max(need, std::min(grid, useful)));
  plan->grid = (int)grid;
  const int G = sh->n_q_heads / sh->n_kv_heads;
  const size_t waves = (size_t)grid * kWaves;
  // The arrival counters open the workspace, and every call returns the ones
  // it used to zero.  Their region has the same size for every grid up to
  // kMaxWorkgroupsPerCu workgroups per compute unit, so the records of one
  // call never land where a later call of another shape expects a zero
  // counter.  A grid wider than that (only when some slice would otherwise
  // exceed kMaxUnitsPerWave) extends the region over what may be records of
  // an earlier call; that launch zeroes its counters first.
  const size_t cap_waves = (size_t)cus * kMaxWorkgroupsPerCu * kWaves;
  const size_t counter_waves = std::max(waves, cap_waves);
  plan->clear_words = waves > cap_waves ? (int)(2 * waves) : 0;
  plan->arrivals_off = 0;
  plan->rec_ml_off = align256(2 * counter_waves * sizeof(int32_t));
  // records: two workgroup pieces and one group record per workgroup
  plan->rec_o_off = plan->rec_ml_off + align256(3 * (size_t)grid * G * 2 * sizeof(float));
  plan->tile_cache_off = plan->rec_o_off + align256(3 * (size_t)grid * G * kHeadDim * sizeof(float));
  // each wave's first-unit tiles, kept for the next call (any content is safe)
  plan->ws_bytes = plan->tile_cache_off + align256(waves * 4 * sizeof(int32_t));
  return DP_OK;
}

}  // namespace

int dpool::decode_workspace_bytes(const dp_decode_shape* shape, size_t* bytes) {
  Plan plan;
  const int rc = validate(shape, &plan);
  if (rc == DP_OK) *bytes = plan.ws_bytes;
  return rc;
}

extern "C" size_t paged_decode_workspace_size(const dp_decode_shape* shape) {
  size_t bytes = 0;
  return dpool::decode_workspace_bytes(shape, &bytes) == DP_OK ? bytes : 0;
}

extern "C" int32_t paged_decode_partition_tokens(const dp_decode_shape* shape) {
  Plan plan;
  if (validate(shape, &plan) != DP_OK) return 0;
  return plan.min_chunk * plan.unit_tokens;
}

extern "C" int paged_decode_attention(const void* q, const void* k_blocks, const void* v_blocks,
                                      const int32_t* block_tables, const int32_t* context_lens, float scale,
                                      const float* k_scale, const float* v_scale, void* out,
                                      const dp_decode_shape* shape, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  using dpool::fail;
  Plan plan;
  int rc = validate(shape, &plan);
  if (rc != DP_OK) return rc;
  if (shape->batch == 0) return DP_OK;
  if (!q || !k_blocks || !v_blocks || !block_tables || !context_lens || !out)
    return fail(DP_EINVAL, "paged_decode: null tensor pointer");
  const bool fp8 = shape->kv_dtype == DP_KV_FP8_E4M3;
  if (fp8 && (!k_scale || !v_scale)) return fail(DP_EINVAL, "paged_decode: fp8 KV needs k_scale and v_scale");
  if (!fp8 && (k_scale || v_scale)) return fail(DP_EINVAL, "paged_decode: k_scale/v_scale must be NULL for bf16 KV");
  if (((uintptr_t)q | (uintptr_t)k_blocks | (uintptr_t)v_blocks | (uintptr_t)out) & 15)
    return fail(DP_EINVAL, "paged_decode: q, k_blocks, v_blocks and out must be 16-byte aligned");
  if (((uintptr_t)block_tables | (uintptr_t)context_lens) & 3)
    return fail(DP_EINVAL, "paged_decode: block_tables and context_lens must be 4-byte aligned");
  if (!std::isfinite(scale)) return fail(DP_EINVAL, "paged_decode: scale is not finite");
  if (!workspace || workspace_bytes < plan.ws_bytes)
    return fail(DP_ENOMEM, "paged_decode: workspace needs %zu bytes, got %zu", plan.ws_bytes, workspace_bytes);
  if ((uintptr_t)workspace & 255) return fail(DP_EINVAL, "paged_decode: workspace must be 256-byte aligned");
  DecodeArgs a;
  a.q = (const uint16_t*)q;
  a.k = (const char*)k_blocks;
  a.v = (const char*)v_blocks;
  a.block_tables = block_tables;
  a.context_lens = context_lens;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.out = out;
  a.arrivals = (int32_t*)((char*)workspace + plan.arrivals_off);
  a.rec_ml = (float*)((char*)workspace + plan.rec_ml_off);
  a.rec_o = (float*)((char*)workspace + plan.rec_o_off);
  a.tile_cache = (int32_t*)((char*)workspace + plan.tile_cache_off);
  a.qk_scale_log2 = scale * kLog2e;
  a.batch = shape->batch;
  a.hq = shape->n_q_heads;
  a.hkv = shape->n_kv_heads;
  a.group = shape->n_q_heads / shape->n_kv_heads;
  a.max_blocks_per_seq = shape->max_blocks_per_seq;
  a.max_ctx = shape->max_context_len;
  a.num_blocks_m1 = (int32_t)(shape->num_blocks - 1);
  a.out_fp32 = shape->out_dtype == DP_OUT_FP32;
  a.min_chunk = plan.min_chunk;
  (void)hipGetLastError();  // clear a stale error left by earlier work
  if (plan.clear_words)
    hipLaunchKernelGGL(zero_words_kernel, dim3(std::min((plan.clear_words + 255) / 256, 1024)), dim3(256), 0,
                       (hipStream_t)stream, a.arrivals, plan.clear_words);
  if (fp8)
    hipLaunchKernelGGL(paged_decode_kernel<true>, dim3(plan.grid), dim3(kWaves * 64), plan.dyn_lds,
                       (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(paged_decode_kernel<false>, dim3(plan.grid), dim3(kWaves * 64), plan.dyn_lds,
                       (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DP_EIO, "paged_decode: kernel launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}
