// Paged decode attention for gfx950 (MI355X).
//
// What it computes: one new query token per sequence attends over that
// sequence's block-paged KV cache - the per-step KV read the paper's cost
// model names as the memory-bandwidth-bound phase (Sec. 3 effect 4, Sec. 4.4
// "Why TPOT also improves"), over 16-token PagedAttention blocks (Sec. 3
// effect 3).  Definition: for sequence s (T = context_lens[s] tokens) and
// query head h with KV head g = h / G,
//     out[s,h] = sum_t softmax_t(scale * q[s,h] . K_t) V_t,
//     K_t / V_t = row t%16 of tile (block_tables[s][t/16], g), times the
//     per-head fp8 scale when the cache is e4m3.
//
// Design (one launch of the partition kernel, plus one merge launch when a
// sequence spans several partitions):
//   * one workgroup per (partition, KV head, sequence); a partition is P
//     consecutive tokens, so long contexts are split across workgroups
//     ("split-K") and merged afterwards with log-sum-exp weights;
//   * the workgroup's NW waves stream disjoint "units" of the partition (one
//     16-token block for bf16, two blocks for fp8) through private LDS stages
//     with gfx950's direct-to-LDS 128-bit loads (global_load_lds_dwordx4), so
//     NSTAGE-1 units per wave stay in flight with no VGPR cost;
//   * every K/V tile of a (block, KV head) is one contiguous 4 KiB (bf16) or
//     2 KiB (fp8) region and is read exactly once; all G query heads of the
//     GQA group use it from LDS;
//   * S^T = K Q^T runs on MFMA (v_mfma_f32_16x16x32_bf16: 16 tokens x 16
//     heads, query heads past G are zero padding).  Its accumulator layout is
//     exactly the B operand of O^T = V^T P, so the probabilities never move
//     between lanes; V^T comes straight out of LDS through the transposing
//     reads ds_read_b64_tr_b16 / ds_read_b64_tr_b8;
//   * the online softmax runs in base 2 (scale * log2 e folded into one
//     multiply), with the per-head max reduced across the four 16-lane rows
//     by cross-lane swizzles; O^T keeps each head in one lane column, so the
//     running-max rescale is lane-local;
//   * fp8 e4m3 tiles are widened to bf16 exactly (v_cvt_scalef32_pk_bf16_fp8
//     with scale 1) and the per-head K scale is folded into the score
//     multiplier, the V scale into the final normalisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "common.h"

// Kernels live in a named namespace: hipcc does not emit the host-side launch
// stubs of templated kernels declared in an anonymous namespace.
namespace dpool_hip {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

#define LDS_AS __attribute__((address_space(3)))

constexpr int kHeadDim = 128;
constexpr int kBlock = 16;
constexpr float kLog2e = 1.4426950408889634f;

struct DecodeArgs {
  const uint16_t* q;          // [B, Hq, 128] bf16
  const char* k;              // [num_blocks, Hkv, 16, 128] bf16 or e4m3
  const char* v;
  const int32_t* block_tables;  // [B, max_blocks_per_seq]
  const int32_t* context_lens;  // [B]
  const float* k_scale;       // [Hkv] (fp8)
  const float* v_scale;
  void* out;                  // [B, Hq, 128] bf16 or fp32
  float* part_o;              // [B, Hq, max_parts, 128]
  float* part_ml;             // [B, Hq, max_parts, 2]  (max in log2 units, sum)
  float qk_scale_log2;        // scale * log2(e)
  int32_t batch, hq, hkv, group;
  int32_t max_blocks_per_seq, max_ctx, part_tokens, max_parts;
  int32_t num_blocks_m1;      // num_blocks - 1 (block ids are clamped into range)
  int32_t out_fp32;
};

// ----- LDS swizzles: 16-byte chunk permutations per row, chosen so that the
// MFMA-layout reads (16 rows, same logical chunk) and the transposing reads
// (4 or 8 rows, adjacent chunks) hit distinct banks.
__device__ __forceinline__ int swz_bf16(int row) {  // 16 chunks per 256-byte row
  return ((row & 3) << 1) | ((row >> 2) & 1) | (row & 8);
}
__device__ __forceinline__ int swz_fp8(int row) {  // 8 chunks per 128-byte row
  return (row & 3) | ((((row >> 2) ^ (row >> 3)) & 1) << 2);
}

__device__ __forceinline__ void wait_vmcnt(int n) {
  // s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
  // vmcnt[3:0] | expcnt[6:4]=7 | lgkmcnt[11:8]=15 | vmcnt[5:4] in [15:14]).
  switch (n) {
#define WV(N) \
  case N: __builtin_amdgcn_s_waitcnt(((N) & 15) | (7 << 4) | (15 << 8) | (((N) >> 4) << 14)); break;
    WV(0) WV(1) WV(2) WV(3) WV(4) WV(5) WV(6) WV(7) WV(8) WV(9) WV(10) WV(11) WV(12) WV(13) WV(14) WV(15)
    WV(16) WV(17) WV(18) WV(19) WV(20) WV(21) WV(22) WV(23) WV(24) WV(25) WV(26) WV(27) WV(28)
#undef WV
    default: __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); break;
  }
}

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

// Transposing LDS reads, issued as inline asm: through the builtins the
// compiler cannot tell them apart from the in-flight direct-to-LDS loads and
// waits for every outstanding global load first.  The caller waits for
// completion with lds_wait_*(), which also carries the data dependency.
__device__ __forceinline__ i32x2 ds_read_tr16(uint32_t lds_addr) {
  i32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(lds_addr) : "memory");
  return r;
}
__device__ __forceinline__ i32x2 ds_read_tr8(uint32_t lds_addr) {
  i32x2 r;
  asm volatile("ds_read_b64_tr_b8 %0, %1" : "=v"(r) : "v"(lds_addr) : "memory");
  return r;
}
__device__ __forceinline__ void lds_wait_8(i32x2 (&v)[8]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7])
               :
               : "memory");
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

// Enqueue the direct-to-LDS loads of one unit (its K tiles, then its V tiles)
// into stage ui % NSTAGE of the wave's LDS region.  Each lane moves 16 bytes
// per instruction; goff holds its swizzled source offsets inside a tile.
template <bool FP8, int NSTAGE>
__device__ __forceinline__ void issue_unit(char* wbase, int my_ids, int ui, const char* kpool, const char* vpool,
                                           size_t block_stride, size_t head_tile, const int* goff) {
  constexpr int UB = FP8 ? 2 : 1;
  constexpr int TILE = FP8 ? 2048 : 4096;
  constexpr int STAGE = 2 * UB * TILE;
  constexpr int DMA_PER_TILE = TILE / 1024;
  char* st = wbase + (ui % NSTAGE) * STAGE;
  for (int b = 0; b < UB; ++b) {
    const int id = __builtin_amdgcn_readlane(my_ids, ui * UB + b);
    const char* kt = kpool + (size_t)id * block_stride + head_tile;
    for (int k = 0; k < DMA_PER_TILE; ++k)
      __builtin_amdgcn_global_load_lds(kt + goff[k], (LDS_AS void*)(st + b * TILE + k * 1024), 16, 0, 0);
  }
  for (int b = 0; b < UB; ++b) {
    const int id = __builtin_amdgcn_readlane(my_ids, ui * UB + b);
    const char* vt = vpool + (size_t)id * block_stride + head_tile;
    for (int k = 0; k < DMA_PER_TILE; ++k)
      __builtin_amdgcn_global_load_lds(vt + goff[k], (LDS_AS void*)(st + UB * TILE + b * TILE + k * 1024), 16, 0,
                                       0);
  }
}

template <bool FP8, int NW, int NSTAGE>
__global__ __launch_bounds__(NW * 64) void paged_decode_partition_kernel(DecodeArgs a) {
  constexpr int UB = FP8 ? 2 : 1;                // blocks per unit
  constexpr int TILE = FP8 ? 2048 : 4096;        // bytes of one (block, head) tile
  constexpr int STAGE = 2 * UB * TILE;           // K tiles then V tiles
  constexpr int DMA_PER_TILE = TILE / 1024;      // 64 lanes x 16 B per instruction
  constexpr int LOADS_PER_UNIT = 2 * UB * DMA_PER_TILE;
  constexpr int LOADS_V = UB * DMA_PER_TILE;
  constexpr int MERGE_STRIDE = kHeadDim + 4;     // floats per head row in the merge area
  static_assert(NW * NSTAGE * STAGE >= NW * 16 * 2 * 4 + NW * 16 * MERGE_STRIDE * 4, "merge area fits");
  __shared__ __attribute__((aligned(1024))) char smem[NW * NSTAGE * STAGE];

  const int p = blockIdx.x, g = blockIdx.y, s = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int G = a.group;
  const int li = lane & 15;  // MFMA column (head) / row index
  const int lj = lane >> 4;  // 16-lane row of the wave

  int ctx = a.context_lens[s];
  ctx = ctx < 0 ? 0 : (ctx > a.max_ctx ? a.max_ctx : ctx);
  const int P = a.part_tokens;
  if (ctx == 0) {
    if (p == 0) {  // empty sequence: zero output rows of this KV head's query heads
      for (int idx = threadIdx.x; idx < G * kHeadDim; idx += NW * 64) {
        const size_t o = ((size_t)s * a.hq + (size_t)g * G) * kHeadDim + idx;
        if (a.out_fp32) ((float*)a.out)[o] = 0.f;
        else ((uint16_t*)a.out)[o] = 0;
      }
    }
    return;
  }
  const int n_parts = (ctx + P - 1) / P;
  if (p >= n_parts) return;
  const int tok_begin = p * P;
  const int tok_end = min(ctx, tok_begin + P);
  const int kb0 = tok_begin / kBlock;
  const int nb = (tok_end - tok_begin + kBlock - 1) / kBlock;
  const int n_units = (nb + UB - 1) / UB;
  const int my_units = n_units > w ? (n_units - w + NW - 1) / NW : 0;

  // Block ids of this wave's units, one per lane: lane L <-> (unit L / UB, block L % UB).
  int my_ids = 0;
  {
    const int L = lane;
    if (L < my_units * UB) {
      int bi = kb0 + (w + NW * (L / UB)) * UB + (L % UB);
      if (bi >= kb0 + nb) bi -= 1;  // absent second block of a unit: reload the first (masked later)
      int id = a.block_tables[(size_t)s * a.max_blocks_per_seq + bi];
      my_ids = id < 0 ? 0 : (id > a.num_blocks_m1 ? a.num_blocks_m1 : id);
    }
  }

  // Q as the MFMA B operand: lane (li, lj) holds head li, 8 head-dim values per chunk c.
  bf16x8 qop[4];
  {
    const int h = g * G + li;
    for (int c = 0; c < 4; ++c) {
      const int d = FP8 ? 64 * (c >> 1) + 16 * lj + 8 * (c & 1) : 32 * c + 8 * lj;
      if (li < G) {
        qop[c] = *(const bf16x8*)(a.q + ((size_t)s * a.hq + h) * kHeadDim + d);
      } else {
        for (int e = 0; e < 8; ++e) qop[c][e] = (__bf16)0.f;
      }
    }
  }
  float cs = a.qk_scale_log2;
  if constexpr (FP8) cs *= a.k_scale[g];

  // Per-lane byte offsets: global (inside a tile) for each DMA instruction, and
  // LDS (inside a stage) for the MFMA-layout K reads and the transposing V reads.
  int goff[DMA_PER_TILE];
  for (int k = 0; k < DMA_PER_TILE; ++k) {
    if constexpr (FP8) {
      const int row = 8 * k + (lane >> 3);
      goff[k] = row * 128 + 16 * ((lane & 7) ^ swz_fp8(row));
    } else {
      const int row = 4 * k + (lane >> 4);
      goff[k] = row * 256 + 16 * ((lane & 15) ^ swz_bf16(row));
    }
  }
  int koff[4];  // bf16: chunk c ; fp8: (group q, half h) -> index 2q + h
  int voff[8];
  if constexpr (FP8) {
    for (int qg = 0; qg < 2; ++qg)
      for (int hh = 0; hh < 2; ++hh) {
        const int tau = 8 * (li >> 2) + 4 * qg + (li & 3);
        const int b = tau >> 4, r = tau & 15;
        koff[2 * qg + hh] = b * TILE + r * 128 + 16 * ((4 * hh + lj) ^ swz_fp8(r));
      }
    for (int n = 0; n < 8; ++n) {
      const int tau = 8 * lj + (li >> 1);
      const int b = tau >> 4, r = tau & 15;
      voff[n] = UB * TILE + b * TILE + r * 128 + 16 * (n ^ swz_fp8(r)) + 8 * (lane & 1);
    }
  } else {
    for (int c = 0; c < 4; ++c) koff[c] = li * 256 + 16 * ((4 * c + lj) ^ swz_bf16(li));
    for (int n = 0; n < 8; ++n) {
      const int row = 4 * lj + (li >> 2);
      voff[n] = TILE + row * 256 + 16 * ((2 * n + ((lane & 3) >> 1)) ^ swz_bf16(row)) + 8 * (lane & 1);
    }
  }

  char* const wbase = smem + w * NSTAGE * STAGE;
  const size_t head_tile = (size_t)g * TILE;
  const size_t block_stride = (size_t)a.hkv * TILE;

  float m_run = -INFINITY;  // running max (log2 units) of head li
  float l_part = 0.f;       // this lane's share of the running sum of head li
  f32x4 acc[8];
  for (int n = 0; n < 8; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int pro = min(NSTAGE - 1, my_units);
  for (int ui = 0; ui < pro; ++ui)
    issue_unit<FP8, NSTAGE>(wbase, my_ids, ui, a.k, a.v, block_stride, head_tile, goff);

  for (int ui = 0; ui < my_units; ++ui) {
    if (ui + NSTAGE - 1 < my_units) {
      __builtin_amdgcn_s_waitcnt((7 << 4) | (0 << 8) | (15) | (3 << 14));  // lgkmcnt(0): stage reads done
      issue_unit<FP8, NSTAGE>(wbase, my_ids, ui + NSTAGE - 1, a.k, a.v, block_stride, head_tile, goff);
    }
    const int younger = min(NSTAGE - 1, my_units - 1 - ui);
    const char* st = wbase + (ui % NSTAGE) * STAGE;
    const uint32_t st_lds = (uint32_t)(uintptr_t)(const LDS_AS char*)st;
    const int unit_tok0 = (kb0 + (w + NW * ui) * UB) * kBlock;
    const bool ragged = unit_tok0 + UB * kBlock > tok_end;

    wait_vmcnt(younger * LOADS_PER_UNIT + LOADS_V);  // K tiles of this unit have landed

    float z[2 * UB * 2];  // bf16: 4 scores (tokens 4lj+r); fp8: 8 scores (tokens 8lj+e)
    if constexpr (FP8) {
      for (int qg = 0; qg < 2; ++qg) {
        f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
        for (int hh = 0; hh < 2; ++hh) {
          const i32x4 raw = *(const LDS_AS i32x4*)(st + koff[2 * qg + hh]);
          const bf16x8 k0 = fp8x8_to_bf16(raw[0], raw[1]);
          const bf16x8 k1 = fp8x8_to_bf16(raw[2], raw[3]);
          sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qop[2 * hh], sacc, 0, 0, 0);
          sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qop[2 * hh + 1], sacc, 0, 0, 0);
        }
        for (int r = 0; r < 4; ++r) z[4 * qg + r] = sacc[r] * cs;
      }
      if (ragged)
        for (int e = 0; e < 8; ++e)
          if (unit_tok0 + 8 * lj + e >= tok_end) z[e] = -INFINITY;
    } else {
      f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
      for (int c = 0; c < 4; ++c) {
        const bf16x8 kop = *(const LDS_AS bf16x8*)(st + koff[c]);
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[c], sacc, 0, 0, 0);
      }
      for (int r = 0; r < 4; ++r) z[r] = sacc[r] * cs;
      if (ragged)
        for (int r = 0; r < 4; ++r)
          if (unit_tok0 + 4 * lj + r >= tok_end) z[r] = -INFINITY;
    }

    // online softmax (base 2) for head li over this unit's tokens
    constexpr int NZ = FP8 ? 8 : 4;
    float bmax = z[0];
    for (int e = 1; e < NZ; ++e) bmax = fmaxf(bmax, z[e]);
    bmax = xor_max(bmax);
    const float m_new = fmaxf(m_run, bmax);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    __bf16 pb[NZ];
    float psum = 0.f;
    for (int e = 0; e < NZ; ++e) {
      pb[e] = (__bf16)__builtin_amdgcn_exp2f(z[e] - m_new);
      psum += (float)pb[e];
    }
    l_part = l_part * alpha + psum;
    for (int n = 0; n < 8; ++n) acc[n] *= alpha;

    wait_vmcnt(younger * LOADS_PER_UNIT);  // V tiles of this unit have landed

    if constexpr (FP8) {
      bf16x8 pop;
      for (int e = 0; e < 8; ++e) pop[e] = pb[e];
      i32x2 raw[8];
      for (int n = 0; n < 8; ++n) raw[n] = ds_read_tr8(st_lds + voff[n]);
      lds_wait_8(raw);
      for (int n = 0; n < 8; ++n) {
        bf16x8 vop = fp8x8_to_bf16(raw[n][0], raw[n][1]);
        if (ragged)
          for (int e = 0; e < 8; ++e)
            if (unit_tok0 + 8 * lj + e >= tok_end) vop[e] = (__bf16)0.f;
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop, acc[n], 0, 0, 0);
      }
    } else {
      bf16x4 pop;
      for (int e = 0; e < 4; ++e) pop[e] = pb[e];
      i32x2 raw[8];
      for (int n = 0; n < 8; ++n) raw[n] = ds_read_tr16(st_lds + voff[n]);
      lds_wait_8(raw);
      for (int n = 0; n < 8; ++n) {
        bf16x4 vop = __builtin_bit_cast(bf16x4, raw[n]);
        if (ragged)
          for (int e = 0; e < 4; ++e)
            if (unit_tok0 + 4 * lj + e >= tok_end) vop[e] = (__bf16)0.f;
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, pop, acc[n], 0, 0, 0);
      }
    }
  }

  // ---- merge the NW waves of this workgroup through LDS ----
  const float l_wave = xor_sum(l_part);
  __syncthreads();  // every wave is done with its stages
  float* ml = (float*)smem;                      // [NW][16][2]
  float* oacc = (float*)smem + NW * 16 * 2;      // [NW][16][MERGE_STRIDE]
  if (lj == 0) {
    ml[(w * 16 + li) * 2 + 0] = m_run;
    ml[(w * 16 + li) * 2 + 1] = l_wave;
  }
  __syncthreads();
  float M = -INFINITY;
  for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, ml[(ww * 16 + li) * 2]);
  const float f_self = my_units > 0 ? __builtin_amdgcn_exp2f(m_run - M) : 0.f;
  for (int n = 0; n < 8; ++n) {
    f32x4 o = acc[n] * f_self;
    *(f32x4*)(oacc + (w * 16 + li) * MERGE_STRIDE + 16 * n + 4 * lj) = o;
  }
  __syncthreads();

  float vsc = 1.0f;
  if constexpr (FP8) vsc = a.v_scale[g];
  const bool single = n_parts == 1;
  for (int idx = threadIdx.x; idx < G * 32; idx += NW * 64) {
    const int i = idx >> 5;
    const int d = (idx & 31) * 4;
    float Mi = -INFINITY;
    for (int ww = 0; ww < NW; ++ww) Mi = fmaxf(Mi, ml[(ww * 16 + i) * 2]);
    float Li = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int ww = 0; ww < NW; ++ww) {
      const float mw = ml[(ww * 16 + i) * 2];
      const float f = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - Mi);
      Li += ml[(ww * 16 + i) * 2 + 1] * f;
      o += *(const f32x4*)(oacc + (ww * 16 + i) * MERGE_STRIDE + d);
    }
    const float inv = vsc / Li;
    o *= inv;
    const int h = g * G + i;
    if (single) {
      const size_t off = ((size_t)s * a.hq + h) * kHeadDim + d;
      if (a.out_fp32) {
        *(f32x4*)((float*)a.out + off) = o;
      } else {
        u16x4 ob;
        for (int e = 0; e < 4; ++e) ob[e] = f32_to_bf16_bits(o[e]);
        *(u16x4*)((uint16_t*)a.out + off) = ob;
      }
    } else {
      const size_t row = ((size_t)s * a.hq + h) * a.max_parts + p;
      *(f32x4*)(a.part_o + row * kHeadDim + d) = o;
      if (d == 0) {
        a.part_ml[row * 2 + 0] = Mi;
        a.part_ml[row * 2 + 1] = Li;
      }
    }
  }
}

// Log-sum-exp merge of the partition partials of each (sequence, KV head):
// M = max_p m_p, w_p = l_p 2^(m_p - M), out = sum_p w_p o_p / sum_p w_p.
__global__ __launch_bounds__(256) void paged_decode_merge_kernel(DecodeArgs a) {
  const int g = blockIdx.x, s = blockIdx.y;
  int ctx = a.context_lens[s];
  ctx = ctx < 0 ? 0 : (ctx > a.max_ctx ? a.max_ctx : ctx);
  const int n_parts = (ctx + a.part_tokens - 1) / a.part_tokens;
  if (n_parts <= 1) return;  // written directly by the partition kernel
  const int G = a.group;
  for (int idx = threadIdx.x; idx < G * 32; idx += 256) {
    const int i = idx >> 5;
    const int d = (idx & 31) * 4;
    const int h = g * G + i;
    const size_t row0 = ((size_t)s * a.hq + h) * a.max_parts;
    float M = -INFINITY;
    for (int pp = 0; pp < n_parts; ++pp) M = fmaxf(M, a.part_ml[(row0 + pp) * 2]);
    float L = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int pp = 0; pp < n_parts; ++pp) {
      const float wgt = a.part_ml[(row0 + pp) * 2 + 1] * __builtin_amdgcn_exp2f(a.part_ml[(row0 + pp) * 2] - M);
      L += wgt;
      o += wgt * *(const f32x4*)(a.part_o + (row0 + pp) * kHeadDim + d);
    }
    o *= 1.0f / L;
    const size_t off = ((size_t)s * a.hq + h) * kHeadDim + d;
    if (a.out_fp32) {
      *(f32x4*)((float*)a.out + off) = o;
    } else {
      u16x4 ob;
      for (int e = 0; e < 4; ++e) ob[e] = f32_to_bf16_bits(o[e]);
      *(u16x4*)((uint16_t*)a.out + off) = ob;
    }
  }
}

// The instantiations the launcher dispatches to (bf16 / fp8 KV, 2-4 stages).
template __global__ void paged_decode_partition_kernel<false, 4, 2>(DecodeArgs);
template __global__ void paged_decode_partition_kernel<true, 4, 2>(DecodeArgs);
template __global__ void paged_decode_partition_kernel<false, 4, 3>(DecodeArgs);
template __global__ void paged_decode_partition_kernel<true, 4, 3>(DecodeArgs);
template __global__ void paged_decode_partition_kernel<false, 4, 4>(DecodeArgs);
template __global__ void paged_decode_partition_kernel<true, 4, 4>(DecodeArgs);

}  // namespace dpool_hip

namespace {

using namespace dpool_hip;

constexpr int kWaves = 4;

int default_partition(const dp_decode_shape* sh) {
  const int unit = sh->kv_dtype == DP_KV_FP8_E4M3 ? 32 : 16;
  int P = 512;
  const int need = ((sh->max_context_len + unit - 1) / unit) * unit;
  if (need > 0 && need < P) P = need;  // one partition covers every sequence
  return std::max(P, unit);
}

int default_stages(const dp_decode_shape*) { return 2; }

struct Plan {
  int P, stages, max_parts;
  size_t ws_bytes;
};

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
  if (sh->batch < 0 || sh->batch > 65535) return fail(DP_EINVAL, "paged_decode: batch %d outside [0, 65535]", sh->batch);
  if (sh->n_q_heads <= 0 || sh->n_kv_heads <= 0 || sh->n_kv_heads > 65535 || sh->n_q_heads % sh->n_kv_heads)
    return fail(DP_EINVAL, "paged_decode: n_q_heads %d must be a positive multiple of n_kv_heads %d",
                sh->n_q_heads, sh->n_kv_heads);
  if (sh->n_q_heads / sh->n_kv_heads > 16)
    return fail(DP_ENOTSUP, "paged_decode: GQA group %d > 16", sh->n_q_heads / sh->n_kv_heads);
  if (sh->max_blocks_per_seq <= 0 || sh->max_context_len < 0 ||
      (int64_t)sh->max_context_len > (int64_t)sh->max_blocks_per_seq * kBlock)
    return fail(DP_EINVAL, "paged_decode: max_context_len %d must be in [0, 16 * max_blocks_per_seq = %lld]",
                sh->max_context_len, (long long)sh->max_blocks_per_seq * kBlock);
  if (sh->num_blocks <= 0 || sh->num_blocks > (int64_t)INT32_MAX + 1)
    return fail(DP_EINVAL, "paged_decode: num_blocks %lld", (long long)sh->num_blocks);
  const int unit = sh->kv_dtype == DP_KV_FP8_E4M3 ? 32 : 16;
  int P = sh->partition_tokens ? sh->partition_tokens : default_partition(sh);
  if (P <= 0 || P % unit || P / kBlock > 64 * kWaves)
    return fail(DP_EINVAL, "paged_decode: partition_tokens %d must be a positive multiple of %d and <= %d", P, unit,
                64 * kWaves * kBlock);
  int st = sh->pipeline_stages ? sh->pipeline_stages : default_stages(sh);
  if (st < 2 || st > 4) return fail(DP_EINVAL, "paged_decode: pipeline_stages %d outside [2, 4]", st);
  plan->P = P;
  plan->stages = st;
  plan->max_parts = sh->max_context_len > 0 ? (sh->max_context_len + P - 1) / P : 1;
  plan->ws_bytes = 0;
  if (plan->max_parts > 1) {
    const size_t rows = (size_t)sh->batch * sh->n_q_heads * plan->max_parts;
    size_t o_bytes = rows * kHeadDim * sizeof(float);
    o_bytes = (o_bytes + 255) & ~(size_t)255;
    plan->ws_bytes = o_bytes + rows * 2 * sizeof(float);
  }
  return DP_OK;
}

template <bool FP8, int ST>
void launch_partition(dim3 grid, hipStream_t stream, const DecodeArgs& args) {
  hipLaunchKernelGGL((paged_decode_partition_kernel<FP8, kWaves, ST>), grid, dim3(kWaves * 64), 0, stream, args);
}

}  // namespace

extern "C" size_t paged_decode_workspace_size(const dp_decode_shape* shape) {
  Plan plan;
  if (validate(shape, &plan) != DP_OK) return 0;
  return plan.ws_bytes;
}

extern "C" int32_t paged_decode_partition_tokens(const dp_decode_shape* shape) {
  Plan plan;
  if (validate(shape, &plan) != DP_OK) return 0;
  return plan.P;
}

namespace {

// Validate everything the host can check and fill the kernel arguments.
int prepare(const void* q, const void* k_blocks, const void* v_blocks, const int32_t* block_tables,
            const int32_t* context_lens, float scale, const float* k_scale, const float* v_scale, void* out,
            const dp_decode_shape* shape, void* workspace, size_t workspace_bytes, Plan* plan, DecodeArgs* args) {
  using dpool::fail;
  int rc = validate(shape, plan);
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
  if (plan->ws_bytes > 0) {
    if (!workspace || workspace_bytes < plan->ws_bytes)
      return fail(DP_ENOMEM, "paged_decode: workspace needs %zu bytes, got %zu", plan->ws_bytes, workspace_bytes);
    if ((uintptr_t)workspace & 255) return fail(DP_EINVAL, "paged_decode: workspace must be 256-byte aligned");
  }
  DecodeArgs& a = *args;
  a.q = (const uint16_t*)q;
  a.k = (const char*)k_blocks;
  a.v = (const char*)v_blocks;
  a.block_tables = block_tables;
  a.context_lens = context_lens;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.out = out;
  a.part_o = nullptr;
  a.part_ml = nullptr;
  if (plan->ws_bytes > 0) {
    const size_t rows = (size_t)shape->batch * shape->n_q_heads * plan->max_parts;
    const size_t o_bytes = (rows * kHeadDim * sizeof(float) + 255) & ~(size_t)255;
    a.part_o = (float*)workspace;
    a.part_ml = (float*)((char*)workspace + o_bytes);
  }
  a.qk_scale_log2 = scale * kLog2e;
  a.batch = shape->batch;
  a.hq = shape->n_q_heads;
  a.hkv = shape->n_kv_heads;
  a.group = shape->n_q_heads / shape->n_kv_heads;
  a.max_blocks_per_seq = shape->max_blocks_per_seq;
  a.max_ctx = shape->max_context_len;
  a.part_tokens = plan->P;
  a.max_parts = plan->max_parts;
  a.num_blocks_m1 = (int32_t)(shape->num_blocks - 1);
  a.out_fp32 = shape->out_dtype == DP_OUT_FP32;
  return DP_OK;
}

int launch_partition_phase(const dp_decode_shape* shape, const Plan& plan, const DecodeArgs& args, hipStream_t st) {
  const dim3 grid(plan.max_parts, shape->n_kv_heads, shape->batch);
  const bool fp8 = shape->kv_dtype == DP_KV_FP8_E4M3;
  (void)hipGetLastError();  // clear a stale error left by earlier work
  switch (plan.stages * 2 + (fp8 ? 1 : 0)) {
    case 4: launch_partition<false, 2>(grid, st, args); break;
    case 5: launch_partition<true, 2>(grid, st, args); break;
    case 6: launch_partition<false, 3>(grid, st, args); break;
    case 7: launch_partition<true, 3>(grid, st, args); break;
    case 8: launch_partition<false, 4>(grid, st, args); break;
    default: launch_partition<true, 4>(grid, st, args); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dpool::fail(DP_EIO, "paged_decode: partition launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}

int launch_merge_phase(const dp_decode_shape* shape, const Plan& plan, const DecodeArgs& args, hipStream_t st) {
  if (plan.max_parts <= 1) return DP_OK;
  (void)hipGetLastError();
  hipLaunchKernelGGL(paged_decode_merge_kernel, dim3(shape->n_kv_heads, shape->batch), dim3(256), 0, st, args);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dpool::fail(DP_EIO, "paged_decode: merge launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}

}  // namespace

extern "C" int paged_decode_attention(const void* q, const void* k_blocks, const void* v_blocks,
                                      const int32_t* block_tables, const int32_t* context_lens, float scale,
                                      const float* k_scale, const float* v_scale, void* out,
                                      const dp_decode_shape* shape, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  Plan plan;
  DecodeArgs args;
  int rc = prepare(q, k_blocks, v_blocks, block_tables, context_lens, scale, k_scale, v_scale, out, shape, workspace,
                   workspace_bytes, &plan, &args);
  if (rc != DP_OK || shape->batch == 0) return rc;
  rc = launch_partition_phase(shape, plan, args, (hipStream_t)stream);
  if (rc != DP_OK) return rc;
  return launch_merge_phase(shape, plan, args, (hipStream_t)stream);
}

extern "C" int paged_decode_partition(const void* q, const void* k_blocks, const void* v_blocks,
                                      const int32_t* block_tables, const int32_t* context_lens, float scale,
                                      const float* k_scale, const float* v_scale, void* out,
                                      const dp_decode_shape* shape, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  Plan plan;
  DecodeArgs args;
  int rc = prepare(q, k_blocks, v_blocks, block_tables, context_lens, scale, k_scale, v_scale, out, shape, workspace,
                   workspace_bytes, &plan, &args);
  if (rc != DP_OK || shape->batch == 0) return rc;
  return launch_partition_phase(shape, plan, args, (hipStream_t)stream);
}

extern "C" int paged_decode_merge(const int32_t* context_lens, void* out, const dp_decode_shape* shape,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  using dpool::fail;
  Plan plan;
  int rc = validate(shape, &plan);
  if (rc != DP_OK) return rc;
  if (shape->batch == 0 || plan.max_parts <= 1) return DP_OK;
  if (!context_lens || !out) return fail(DP_EINVAL, "paged_decode_merge: null tensor pointer");
  if (((uintptr_t)out & 15) || ((uintptr_t)context_lens & 3))
    return fail(DP_EINVAL, "paged_decode_merge: out must be 16-byte and context_lens 4-byte aligned");
  if (!workspace || workspace_bytes < plan.ws_bytes)
    return fail(DP_ENOMEM, "paged_decode_merge: workspace needs %zu bytes, got %zu", plan.ws_bytes, workspace_bytes);
  if ((uintptr_t)workspace & 255) return fail(DP_EINVAL, "paged_decode_merge: workspace must be 256-byte aligned");
  DecodeArgs a = {};
  const size_t rows = (size_t)shape->batch * shape->n_q_heads * plan.max_parts;
  const size_t o_bytes = (rows * kHeadDim * sizeof(float) + 255) & ~(size_t)255;
  a.part_o = (float*)workspace;
  a.part_ml = (float*)((char*)workspace + o_bytes);
  a.context_lens = context_lens;
  a.out = out;
  a.batch = shape->batch;
  a.hq = shape->n_q_heads;
  a.hkv = shape->n_kv_heads;
  a.group = shape->n_q_heads / shape->n_kv_heads;
  a.max_ctx = shape->max_context_len;
  a.part_tokens = plan.P;
  a.max_parts = plan.max_parts;
  a.out_fp32 = shape->out_dtype == DP_OUT_FP32;
  return launch_merge_phase(shape, plan, a, (hipStream_t)stream);
}
