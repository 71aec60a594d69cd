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
// Work decomposition (stream-K over the KV stream).  The cached tokens of
// every (sequence, KV head) "segment" form one flat stream of units (a unit
// is one 16-token block for bf16, two for fp8), segments in sequence-major,
// head-minor order.  A persistent grid sized to the device gives every wave
// one contiguous, equal-length slice of that stream, so the load is balanced
// to one unit however skewed the context lengths are, and no workgroup is
// launched without work.  A wave walks its slice across segment boundaries
// without draining its load pipeline.  A segment that lies wholly inside one
// slice is finished in registers and written to `out`; a segment cut by slice
// boundaries leaves one softmax partial per piece (each wave has at most two
// such pieces: its first and its last), merged afterwards with log-sum-exp
// weights by the merge kernel.
//
// Per wave, the hot loop:
//   * gfx950's direct-to-LDS loads (global_load_lds_dwordx4, 16 B per lane)
//     move each unit's K and V tiles into one of NSTAGE private LDS stages,
//     so NSTAGE-1 units stay in flight at no VGPR cost; a (block, head) tile
//     is one contiguous 4 KiB (bf16) / 2 KiB (fp8) region read exactly once;
//   * S^T = K Q^T on MFMA (v_mfma_f32_16x16x32_bf16: 16 tokens x 16 query
//     heads, heads past the GQA group are zero padding), so every query head
//     of the group reuses the tile from LDS;
//   * the score accumulator layout is exactly the B operand of O^T = V^T P,
//     so probabilities never move between lanes; V^T comes out of LDS
//     through the transposing reads ds_read_b64_tr_b16 / _b8;
//   * online softmax in base 2 (scale * log2 e folded into one multiply),
//     the per-head max crossing the four 16-lane rows by two swizzles; O^T
//     keeps each head in one lane column, so the running-max rescale is
//     lane-local;
//   * fp8 e4m3 tiles widen to bf16 exactly (v_cvt_scalef32_pk_bf16_fp8 with
//     scale 1); the per-head K scale folds into the score multiplier, the V
//     scale into the final normalisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>

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
constexpr int kWaves = 4;                 // waves per workgroup
constexpr int kMaxUnitsPerWave = 256;     // the host sizes the grid so that no slice is longer

struct StreamArgs {
  const uint16_t* q;            // [B, Hq, 128] bf16
  const char* k;                // [num_blocks, Hkv, 16, 128] bf16 or e4m3
  const char* v;
  const int32_t* block_tables;  // [B, max_blocks_per_seq]
  const int32_t* context_lens;  // [B]
  const float* k_scale;         // [Hkv] (fp8)
  const float* v_scale;
  void* out;                    // [B, Hq, 128] bf16 or fp32
  float* rec_o;                 // [waves, 2, G, 128]  partial outputs (normalised)
  float* rec_ml;                // [waves, 2, G, 2]    (max in log2 units, sum)
  int32_t* plan;                // [B + 2]: unit prefix over sequences, then the slice length
  int32_t* hdr;                 // [waves, 4]: (s, g, a0, nus) of the segment a wave terminates, nus = 0 if none
  float qk_scale_log2;          // scale * log2(e)
  int32_t batch, hq, hkv, group;
  int32_t max_blocks_per_seq, max_ctx;
  int32_t num_blocks_m1;        // num_blocks - 1 (block ids are clamped into range)
  int32_t out_fp32;
  int32_t min_chunk;            // minimum units per slice
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

// LDS reads of the V stages, issued as inline asm: through the builtins the
// compiler cannot tell them apart from the direct-to-LDS loads in flight
// into other stages and waits for every outstanding global load first.  Each
// asm block issues its reads and waits for them (lgkmcnt(0)) before it ends,
// so its outputs are complete when the compiler first sees them.
__device__ __forceinline__ void ds_read_tr16_x8(uint32_t base, const int* off, i32x2 (&r)[8]) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8\n\tds_read_b64_tr_b16 %1, %9\n\tds_read_b64_tr_b16 %2, %10\n\t"
      "ds_read_b64_tr_b16 %3, %11\n\tds_read_b64_tr_b16 %4, %12\n\tds_read_b64_tr_b16 %5, %13\n\t"
      "ds_read_b64_tr_b16 %6, %14\n\tds_read_b64_tr_b16 %7, %15\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
      : "v"(base + off[0]), "v"(base + off[1]), "v"(base + off[2]), "v"(base + off[3]), "v"(base + off[4]),
        "v"(base + off[5]), "v"(base + off[6]), "v"(base + off[7])
      : "memory");
}
__device__ __forceinline__ void ds_read_tr8_x8(uint32_t base, const int* off, i32x2 (&r)[8]) {
  asm volatile(
      "ds_read_b64_tr_b8 %0, %8\n\tds_read_b64_tr_b8 %1, %9\n\tds_read_b64_tr_b8 %2, %10\n\t"
      "ds_read_b64_tr_b8 %3, %11\n\tds_read_b64_tr_b8 %4, %12\n\tds_read_b64_tr_b8 %5, %13\n\t"
      "ds_read_b64_tr_b8 %6, %14\n\tds_read_b64_tr_b8 %7, %15\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
      : "v"(base + off[0]), "v"(base + off[1]), "v"(base + off[2]), "v"(base + off[3]), "v"(base + off[4]),
        "v"(base + off[5]), "v"(base + off[6]), "v"(base + off[7])
      : "memory");
}

__device__ __forceinline__ void ds_read_b128_x4(uint32_t base, const int* off, i32x4 (&r)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
      : "v"(base + off[0]), "v"(base + off[1]), "v"(base + off[2]), "v"(base + off[3])
      : "memory");
}
// Four 16-byte global loads and a wait for them (vmcnt(0), which also drains
// the wave's direct-to-LDS loads in flight) in one asm block.
__device__ __forceinline__ void global_load_b128_x4_wait(const char* p0, const char* p1, const char* p2,
                                                         const char* p3, i32x4 (&r)[4]) {
  asm volatile(
      "global_load_dwordx4 %0, %4, off\n\tglobal_load_dwordx4 %1, %5, off\n\t"
      "global_load_dwordx4 %2, %6, off\n\tglobal_load_dwordx4 %3, %7, off\n\ts_waitcnt vmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
      : "v"(p0), "v"(p1), "v"(p2), "v"(p3)
      : "memory");
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ __forceinline__ int clamp_ctx(int c, int max_ctx) { return c < 0 ? 0 : (c > max_ctx ? max_ctx : c); }

template <bool FP8>
__device__ __forceinline__ int units_of(int ctx) {
  const int nb = (ctx + kBlock - 1) / kBlock;
  return FP8 ? (nb + 1) >> 1 : nb;
}

template <int N>
__device__ __forceinline__ void vm_wait() {
  // s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
  // vmcnt[3:0] | expcnt[6:4]=7 | lgkmcnt[11:8]=15 | vmcnt[5:4] in [15:14]).
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// Wait for the direct-to-LDS loads of the unit being computed: `younger`
// later units (LPU instructions each) are in flight, plus `extra` of this
// unit's own loads issued after the ones waited for.
template <int D, int LPU, int EXTRA>
__device__ __forceinline__ void wait_unit(int younger) {
  if (D >= 3 && younger >= 3) vm_wait<(D >= 3 ? EXTRA + 3 * LPU : 0)>();
  else if (D >= 2 && younger == 2) vm_wait<(D >= 2 ? EXTRA + 2 * LPU : 0)>();
  else if (younger == 1) vm_wait<EXTRA + LPU>();
  else vm_wait<EXTRA>();
}

// Enqueue the direct-to-LDS loads of one unit (its K tiles, then its V
// tiles) into a stage.  Each lane moves 16 bytes per instruction; goff holds
// its swizzled source offsets inside a tile; tiles[] holds the flat tile
// index (block id * Hkv + head) of each block of each unit of the slice.
template <bool FP8>
__device__ __forceinline__ void issue_unit(const int* tiles, int ui, const char* kpool, const char* vpool,
                                           const int* goff, char* st) {
  constexpr int UB = FP8 ? 2 : 1;
  constexpr int TILE = FP8 ? 2048 : 4096;
  constexpr int DMA_PER_TILE = TILE / 1024;
  int t[UB];
  for (int b = 0; b < UB; ++b) t[b] = __builtin_amdgcn_readfirstlane(tiles[ui * UB + b]);
  for (int b = 0; b < UB; ++b) {
    const char* kt = kpool + (size_t)t[b] * TILE;
    for (int k = 0; k < DMA_PER_TILE; ++k)
      __builtin_amdgcn_global_load_lds(kt + goff[k], (LDS_AS void*)(st + b * TILE + k * 1024), 16, 0, 0);
  }
  for (int b = 0; b < UB; ++b) {
    const char* vt = vpool + (size_t)t[b] * TILE;
    for (int k = 0; k < DMA_PER_TILE; ++k)
      __builtin_amdgcn_global_load_lds(vt + goff[k], (LDS_AS void*)(st + (UB + b) * TILE + k * 1024), 16, 0, 0);
  }
}

// D = units in flight ahead of the one being computed (1..3); each wave owns
// D + 1 LDS stages of one unit's K and V tiles (8 KiB).
template <bool FP8, int D>
__global__ __launch_bounds__(kWaves * 64) void paged_decode_stream_kernel(StreamArgs a) {
  constexpr int NW = kWaves;
  constexpr int NS = D + 1;
  constexpr int UB = FP8 ? 2 : 1;                // blocks per unit
  constexpr int TILE = FP8 ? 2048 : 4096;        // bytes of one (block, head) tile
  constexpr int STAGE = 2 * UB * TILE;           // K tiles then V tiles of one unit
  constexpr int LPU = 2 * UB * (TILE / 1024);    // direct-to-LDS instructions per unit
  constexpr int VLD = UB * (TILE / 1024);        // of which V
  __shared__ __attribute__((aligned(1024))) char stages[NW * NS * STAGE];
  __shared__ int tiles_lds[NW][kMaxUnitsPerWave * UB];
  __shared__ int wave_sums[NW];
  extern __shared__ int dyn[];                   // pre[B + 1], ctxs[B], k_scale[Hkv], v_scale[Hkv]

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int B = a.batch, Hkv = a.hkv, G = a.group;
  const int li = lane & 15;  // MFMA column (head) / row index
  const int lj = lane >> 4;  // 16-lane row of the wave
  int* pre = dyn;
  int* ctxs = dyn + B + 1;
  float* kscl = (float*)(dyn + 2 * B + 1);
  float* vscl = kscl + Hkv;

  // ---- 1. prefix of units over sequences (every workgroup computes it) ----
  {
    const int T = NW * 64, tid = threadIdx.x;
    if constexpr (FP8) {
      for (int g = tid; g < Hkv; g += T) {
        kscl[g] = a.k_scale[g];
        vscl[g] = a.v_scale[g];
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
    int incl = local;
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off);
      if (lane >= off) incl += v;
    }
    if (lane == 63) wave_sums[w] = incl;
    __syncthreads();
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
    __syncthreads();
  }
  const int U = Hkv * pre[B];
  const int TW = gridDim.x * NW;
  int C = (U + TW - 1) / TW;
  if (C < a.min_chunk) C = a.min_chunk;
  if (blockIdx.x == 0) {  // the merge kernel needs the prefix and the slice length
    for (int s = threadIdx.x; s <= B; s += NW * 64) a.plan[s] = pre[s];
    if (threadIdx.x == 0) a.plan[B + 1] = C;
  }
  const int gw = blockIdx.x * NW + w;
  const int u0 = gw * C;
  const int u1 = min(u0 + C, U);
  if (u0 >= u1) {  // no work: no segment to terminate
    if (lane == 0) *(i32x4*)(a.hdr + 4 * gw) = i32x4{0, 0, 0, 0};
    return;  // no barrier follows: waves are independent from here on
  }
  const int n = u1 - u0;

  // ---- 2. tile indices of this wave's units into LDS ----
  int* tiles = tiles_lds[w];
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
    const int nb = (ctxs[s] + kBlock - 1) / kBlock;
    for (int b = 0; b < UB; ++b) {
      int blk = j * UB + b;
      if (blk >= nb) blk = j * UB;  // absent second block of an fp8 unit: reload the first (masked later)
      int id = a.block_tables[(size_t)s * a.max_blocks_per_seq + blk];
      id = id < 0 ? 0 : (id > a.num_blocks_m1 ? a.num_blocks_m1 : id);
      tiles[i * UB + b] = id * Hkv + g;
    }
  }

  // ---- 3. per-lane offsets ----
  int goff[TILE / 1024];  // source offset inside a tile for each direct-to-LDS instruction
  for (int k = 0; k < TILE / 1024; ++k) {
    if constexpr (FP8) {
      const int row = 8 * k + (lane >> 3);
      goff[k] = row * 128 + 16 * ((lane & 7) ^ swz_fp8(row));
    } else {
      const int row = 4 * k + (lane >> 4);
      goff[k] = row * 256 + 16 * ((lane & 15) ^ swz_bf16(row));
    }
  }
  int koff[4];  // K reads: bf16 chunk c ; fp8 (group q, half h) -> index 2q + h
  int voff[8];  // V transposing reads
  if constexpr (FP8) {
    for (int qg = 0; qg < 2; ++qg)
      for (int hh = 0; hh < 2; ++hh) {
        const int tau = 8 * (li >> 2) + 4 * qg + (li & 3);
        const int b = tau >> 4, r = tau & 15;
        koff[2 * qg + hh] = b * TILE + r * 128 + 16 * ((4 * hh + lj) ^ swz_fp8(r));
      }
    for (int nn = 0; nn < 8; ++nn) {
      const int tau = 8 * lj + (li >> 1);
      const int b = tau >> 4, r = tau & 15;
      voff[nn] = UB * TILE + b * TILE + r * 128 + 16 * (nn ^ swz_fp8(r)) + 8 * (lane & 1);
    }
  } else {
    for (int c = 0; c < 4; ++c) koff[c] = li * 256 + 16 * ((4 * c + lj) ^ swz_bf16(li));
    for (int nn = 0; nn < 8; ++nn) {
      const int row = 4 * lj + (li >> 2);
      voff[nn] = TILE + row * 256 + 16 * ((2 * nn + ((lane & 3) >> 1)) ^ swz_bf16(row)) + 8 * (lane & 1);
    }
  }
  int qoff[4];  // query reads: head li (padding heads re-read head 0 and are zeroed), chunk c
  for (int c = 0; c < 4; ++c)
    qoff[c] = ((li < G ? li : 0) * kHeadDim + (FP8 ? 64 * (c >> 1) + 16 * lj + 8 * (c & 1) : 32 * c + 8 * lj)) * 2;

  // ---- 4. walk the slice ----
  char* const wbase = stages + w * NS * STAGE;
  // compute-side position (uniform): segment (s, g), unit j inside it
  int cs_s, cs_g, cs_j, cs_nus;
  {
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (Hkv * pre[mid] <= u0) lo = mid;
      else hi = mid - 1;
    }
    cs_s = __builtin_amdgcn_readfirstlane(lo);
    cs_nus = __builtin_amdgcn_readfirstlane(pre[cs_s + 1] - pre[cs_s]);
    const int r = u0 - Hkv * pre[cs_s];
    cs_g = __builtin_amdgcn_readfirstlane(r / cs_nus);
    cs_j = __builtin_amdgcn_readfirstlane(r - cs_g * cs_nus);
    // this wave terminates a split segment when its first piece continues a
    // segment begun by an earlier wave and the segment ends inside this slice
    const bool term = cs_j > 0 && cs_nus - cs_j <= n;
    if (lane == 0) *(i32x4*)(a.hdr + 4 * gw) = term ? i32x4{cs_s, cs_g, u0 - cs_j, cs_nus} : i32x4{0, 0, 0, 0};
  }

  for (int ui = 0; ui < min(D, n); ++ui) issue_unit<FP8>(tiles, ui, a.k, a.v, goff, wbase + ui * STAGE);

  i32x4 qcur[4];
  float m_run = -INFINITY, l_part = 0.f, cscale = 0.f, vsc = 1.0f;
  f32x4 acc[8];
  int piece_j0 = 0, ctx_s = 0;
  bool piece_first = true;

  for (int ui = 0; ui < n; ++ui) {
    if (ui + D < n) {
      __builtin_amdgcn_s_waitcnt((7 << 4) | (0 << 8) | (15) | (3 << 14));  // lgkmcnt(0): stage reads done
      issue_unit<FP8>(tiles, ui + D, a.k, a.v, goff, wbase + ((ui + D) % NS) * STAGE);
    }
    if (ui == 0 || cs_j == 0) {  // a new piece starts: its query group, fresh softmax state
      piece_first = ui == 0;
      piece_j0 = cs_j;
      ctx_s = __builtin_amdgcn_readfirstlane(ctxs[cs_s]);
      const char* qrow = (const char*)(a.q + ((size_t)cs_s * a.hq + cs_g * G) * kHeadDim);
      global_load_b128_x4_wait(qrow + qoff[0], qrow + qoff[1], qrow + qoff[2], qrow + qoff[3], qcur);
      if (li >= G)  // padding heads contribute zero scores
        for (int c = 0; c < 4; ++c) qcur[c] = i32x4{0, 0, 0, 0};
      float ksc = 1.0f;
      if constexpr (FP8) {
        ksc = kscl[cs_g];
        vsc = vscl[cs_g];
      }
      cscale = a.qk_scale_log2 * ksc;
      m_run = -INFINITY;
      l_part = 0.f;
      for (int nn = 0; nn < 8; ++nn) acc[nn] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int younger = min(D, n - 1 - ui);
    const uint32_t st = (uint32_t)(uintptr_t)(const LDS_AS char*)(wbase + (ui % NS) * STAGE);
    const int unit_tok0 = cs_j * UB * kBlock;
    const bool ragged = unit_tok0 + UB * kBlock > ctx_s;

    wait_unit<D, LPU, VLD>(younger);  // K tiles of this unit have landed
    i32x4 kraw[4];
    ds_read_b128_x4(st, koff, kraw);

    constexpr int NZ = FP8 ? 8 : 4;  // scores per lane: bf16 tokens 4lj+r ; fp8 tokens 8lj+e
    float z[NZ];
    if constexpr (FP8) {
      for (int qg = 0; qg < 2; ++qg) {
        f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
        for (int hh = 0; hh < 2; ++hh) {
          const i32x4 raw = kraw[2 * qg + hh];
          const bf16x8 k0 = fp8x8_to_bf16(raw[0], raw[1]);
          const bf16x8 k1 = fp8x8_to_bf16(raw[2], raw[3]);
          sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, __builtin_bit_cast(bf16x8, qcur[2 * hh]), sacc, 0, 0,
                                                         0);
          sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, __builtin_bit_cast(bf16x8, qcur[2 * hh + 1]), sacc, 0,
                                                         0, 0);
        }
        for (int r = 0; r < 4; ++r) z[4 * qg + r] = sacc[r] * cscale;
      }
      if (ragged)
        for (int e = 0; e < 8; ++e)
          if (unit_tok0 + 8 * lj + e >= ctx_s) z[e] = -INFINITY;
    } else {
      f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
      for (int c = 0; c < 4; ++c)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kraw[c]),
                                                       __builtin_bit_cast(bf16x8, qcur[c]), sacc, 0, 0, 0);
      for (int r = 0; r < 4; ++r) z[r] = sacc[r] * cscale;
      if (ragged)
        for (int r = 0; r < 4; ++r)
          if (unit_tok0 + 4 * lj + r >= ctx_s) z[r] = -INFINITY;
    }

    // online softmax (base 2) for head li over this unit's tokens
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
    for (int nn = 0; nn < 8; ++nn) acc[nn] *= alpha;

    wait_unit<D, LPU, 0>(younger);  // V tiles of this unit have landed

    if constexpr (FP8) {
      bf16x8 pop;
      for (int e = 0; e < 8; ++e) pop[e] = pb[e];
      i32x2 raw[8];
      ds_read_tr8_x8(st, voff, raw);
      for (int nn = 0; nn < 8; ++nn) {
        bf16x8 vop = fp8x8_to_bf16(raw[nn][0], raw[nn][1]);
        if (ragged)
          for (int e = 0; e < 8; ++e)
            if (unit_tok0 + 8 * lj + e >= ctx_s) vop[e] = (__bf16)0.f;
        acc[nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop, acc[nn], 0, 0, 0);
      }
    } else {
      bf16x4 pop;
      for (int e = 0; e < 4; ++e) pop[e] = pb[e];
      i32x2 raw[8];
      ds_read_tr16_x8(st, voff, raw);
      for (int nn = 0; nn < 8; ++nn) {
        bf16x4 vop = __builtin_bit_cast(bf16x4, raw[nn]);
        if (ragged)
          for (int e = 0; e < 4; ++e)
            if (unit_tok0 + 4 * lj + e >= ctx_s) vop[e] = (__bf16)0.f;
        acc[nn] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, pop, acc[nn], 0, 0, 0);
      }
    }

    // ---- end of a piece: write the result or a partial record ----
    const bool seg_end = cs_j == cs_nus - 1;
    if (seg_end || ui == n - 1) {
      const float l_tot = xor_sum(l_part);
      const float inv = vsc / l_tot;
      if (li < G) {
        if (piece_j0 == 0 && seg_end) {  // the whole segment: final output
          const size_t row = ((size_t)cs_s * a.hq + cs_g * G + li) * kHeadDim;
          for (int nn = 0; nn < 8; ++nn) {
            const f32x4 o = acc[nn] * inv;
            const size_t off = row + 16 * nn + 4 * lj;
            if (a.out_fp32) {
              *(f32x4*)((float*)a.out + off) = o;
            } else {
              u16x4 ob;
              for (int e = 0; e < 4; ++e) ob[e] = f32_to_bf16_bits(o[e]);
              *(u16x4*)((uint16_t*)a.out + off) = ob;
            }
          }
        } else {  // a piece of a segment cut by slice boundaries
          const size_t rec = (size_t)gw * 2 + (piece_first ? 0 : 1);
          float* ro = a.rec_o + (rec * G + li) * kHeadDim;
          for (int nn = 0; nn < 8; ++nn) *(f32x4*)(ro + 16 * nn + 4 * lj) = acc[nn] * inv;
          if (lj == 0) {
            a.rec_ml[(rec * G + li) * 2 + 0] = m_run;
            a.rec_ml[(rec * G + li) * 2 + 1] = l_tot;
          }
        }
      }
    }
    // advance the compute-side position
    if (ui + 1 < n) {
      if (++cs_j == cs_nus) {
        cs_j = 0;
        if (++cs_g == Hkv) {
          cs_g = 0;
          do {
            ++cs_s;
          } while (cs_s < B - 1 && pre[cs_s + 1] == pre[cs_s]);  // skip empty sequences (bounded)
          cs_s = __builtin_amdgcn_readfirstlane(cs_s);
        }
        cs_nus = __builtin_amdgcn_readfirstlane(pre[cs_s + 1] - pre[cs_s]);
      }
    }
  }
}

// Log-sum-exp merge of the pieces of every segment cut by slice boundaries,
// and zero rows for empty sequences.  One workgroup per wave of the stream
// kernel: workgroup k merges the segment that wave k terminates (if any).
// That segment covers units [a0, a0 + nus); slices have length C, so its
// pieces come from waves k0 = a0 / C .. k: wave k0's last piece (record slot
// 1 if that wave began inside an earlier segment, else slot 0) and the first
// piece (slot 0) of every later wave.  256 threads = record groups x G heads
// x 8 lanes of 16 head-dim values; each group folds its records with a
// running log-sum-exp, and the groups are combined in LDS:
// M = max_p m_p, w_p = l_p 2^(m_p - M), out = sum_p w_p o_p / sum_p w_p.
__global__ __launch_bounds__(256) void paged_decode_merge_kernel(StreamArgs a) {
  const int k = blockIdx.x;
  const int G = a.group, B = a.batch;
  const int tid = threadIdx.x;
  // independent loads first: this wave's header, the slice length, and the
  // prefix entries that say whether sequence k is empty
  const i32x4 h = *(const i32x4*)(a.hdr + 4 * k);
  const int C = a.plan[B + 1];
  for (int s = k; s < B; s += gridDim.x) {  // empty sequences: zero rows
    if (a.plan[s + 1] == a.plan[s]) {
      for (int idx = tid; idx < a.hq * 32; idx += 256) {
        const size_t o = (size_t)s * a.hq * kHeadDim + (size_t)idx * 4;
        if (a.out_fp32) *(f32x4*)((float*)a.out + o) = f32x4{0.f, 0.f, 0.f, 0.f};
        else *(u16x4*)((uint16_t*)a.out + o) = u16x4{0, 0, 0, 0};
      }
    }
  }
  const int s = h[0], g = h[1], a0 = h[2], nus = h[3];
  if (nus == 0) return;  // wave k terminates no split segment
  const int k0 = a0 / C;
  const int first_slot = k0 * 2 + (a0 > k0 * C ? 1 : 0);
  const int nrec = k - k0 + 1;
  const int groups = 256 / (8 * G);             // G <= 16: at least 2 groups
  const int grp = tid / (8 * G);
  const int i = (tid >> 3) % G;                  // head inside the group
  const int d0 = (tid & 7) * 16;                 // 16 head-dim values per lane
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[4] = {};
  if (grp < groups) {
    constexpr int kBatch = 8;  // records whose loads are in flight together
    for (int r0 = grp; r0 < nrec; r0 += groups * kBatch) {
      float m[kBatch], l[kBatch];
      f32x4 o[kBatch][4];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int r = r0 + u * groups;
        if (r < nrec) {
          const size_t rec = r == 0 ? (size_t)first_slot : (size_t)(k0 + r) * 2;
          const float* ml = a.rec_ml + (rec * G + i) * 2;
          m[u] = ml[0];
          l[u] = ml[1];
          const f32x4* op = (const f32x4*)(a.rec_o + (rec * G + i) * kHeadDim + d0);
          for (int e = 0; e < 4; ++e) o[u][e] = op[e];
        } else {
          m[u] = -INFINITY;
          l[u] = 0.f;
          for (int e = 0; e < 4; ++e) o[u][e] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (m[u] == -INFINITY) continue;
        const float m_new = fmaxf(m_run, m[u]);
        const float c_old = __builtin_amdgcn_exp2f(m_run - m_new);
        const float c_new = l[u] * __builtin_amdgcn_exp2f(m[u] - m_new);
        for (int e = 0; e < 4; ++e) acc[e] = acc[e] * c_old + o[u][e] * c_new;
        l_run = l_run * c_old + c_new;
        m_run = m_new;
      }
    }
  }
  __shared__ float sm[32][16], sl[32][16];
  __shared__ f32x4 sacc[256][4];
  if (grp < groups) {
    if ((tid & 7) == 0) {
      sm[grp][i] = m_run;
      sl[grp][i] = l_run;
    }
    for (int e = 0; e < 4; ++e) sacc[tid][e] = acc[e];
  }
  __syncthreads();
  if (grp == 0) {
    float M = -INFINITY;
    for (int q = 0; q < groups; ++q) M = fmaxf(M, sm[q][i]);
    float L = 0.f;
    f32x4 o[4] = {};
    for (int q = 0; q < groups; ++q) {
      const float c = sm[q][i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sm[q][i] - M);
      L += sl[q][i] * c;
      for (int e = 0; e < 4; ++e) o[e] += sacc[q * 8 * G + tid][e] * c;
    }
    const float inv = 1.0f / L;
    const size_t orow = ((size_t)s * a.hq + (size_t)g * G + i) * kHeadDim + d0;
    for (int e = 0; e < 4; ++e) {
      const f32x4 v = o[e] * inv;
      if (a.out_fp32) {
        *(f32x4*)((float*)a.out + orow + 4 * e) = v;
      } else {
        u16x4 ob;
        for (int q = 0; q < 4; ++q) ob[q] = f32_to_bf16_bits(v[q]);
        *(u16x4*)((uint16_t*)a.out + orow + 4 * e) = ob;
      }
    }
  }
}

// The instantiations the launcher dispatches to (bf16 / fp8 KV, 1-3 units in flight).
template __global__ void paged_decode_stream_kernel<false, 1>(StreamArgs);
template __global__ void paged_decode_stream_kernel<true, 1>(StreamArgs);
template __global__ void paged_decode_stream_kernel<false, 2>(StreamArgs);
template __global__ void paged_decode_stream_kernel<true, 2>(StreamArgs);
template __global__ void paged_decode_stream_kernel<false, 3>(StreamArgs);
template __global__ void paged_decode_stream_kernel<true, 3>(StreamArgs);

}  // namespace dpool_hip

namespace {

using namespace dpool_hip;

constexpr int kMaxBatchInLds = 4096;  // the unit prefix of the batch is kept in LDS
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

const void* stream_kernel(bool fp8, int d) {
  switch (d * 2 + (fp8 ? 1 : 0)) {
    case 2: return (const void*)paged_decode_stream_kernel<false, 1>;
    case 3: return (const void*)paged_decode_stream_kernel<true, 1>;
    case 4: return (const void*)paged_decode_stream_kernel<false, 2>;
    case 5: return (const void*)paged_decode_stream_kernel<true, 2>;
    case 6: return (const void*)paged_decode_stream_kernel<false, 3>;
    default: return (const void*)paged_decode_stream_kernel<true, 3>;
  }
}

// Workgroups of the stream kernel one compute unit holds at once, limited by
// registers (runtime occupancy query, cached) and by LDS.  Without a device,
// only the LDS limit applies.
int blocks_per_cu(int dev, bool fp8, int d, size_t lds_bytes) {
  static std::mutex mu;
  static int cached[64][2][4] = {};
  int by_lds = (int)(kLdsBytes / lds_bytes);
  if (dev < 0) return std::max(1, std::min(by_lds, 2));
  int occ;
  {
    std::lock_guard<std::mutex> lock(mu);
    occ = cached[dev][fp8 ? 1 : 0][d];
    if (!occ) {
      int n = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, stream_kernel(fp8, d), kWaves * 64, 0) != hipSuccess ||
          n <= 0) {
        (void)hipGetLastError();
        n = 2;
      }
      occ = cached[dev][fp8 ? 1 : 0][d] = n;
    }
  }
  return std::max(1, std::min(occ, by_lds));
}

struct Plan {
  int unit_tokens;   // tokens per unit (16 bf16, 32 fp8)
  int min_chunk;     // minimum units per slice
  int stages;
  int grid;          // workgroups of the stream kernel
  size_t dyn_lds;    // dynamic LDS bytes
  size_t rec_o_off, rec_ml_off, plan_off, hdr_off, ws_bytes;
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
  if (sh->batch < 0 || sh->batch > 65535) return fail(DP_EINVAL, "paged_decode: batch %d outside [0, 65535]", sh->batch);
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
  const int unit = fp8 ? 32 : 16;
  const int P = sh->partition_tokens;
  if (P < 0 || P % unit || P / unit > kMaxUnitsPerWave)
    return fail(DP_EINVAL, "paged_decode: partition_tokens %d must be a multiple of %d in [0, %d]", P, unit,
                unit * kMaxUnitsPerWave);
  const int st = sh->pipeline_stages ? sh->pipeline_stages : 2;
  if (st < 2 || st > 4) return fail(DP_EINVAL, "paged_decode: pipeline_stages %d outside [2, 4]", st);
  const int64_t units_per_seq = ((int64_t)sh->max_context_len + unit - 1) / unit;
  const int64_t max_units = units_per_seq * sh->batch * sh->n_kv_heads;
  if (max_units > INT32_MAX) return fail(DP_ENOTSUP, "paged_decode: %lld units exceed int32", (long long)max_units);
  plan->unit_tokens = unit;
  plan->min_chunk = P ? P / unit : 8;
  plan->stages = st;
  // LDS per workgroup: K+V stages (8 KiB per unit) + tile indices + wave sums
  // (static) + unit prefix, context lengths and fp8 scales (dynamic)
  const size_t stat = (size_t)kWaves * st * 8192 + (size_t)kWaves * kMaxUnitsPerWave * (fp8 ? 2 : 1) * 4 + 64;
  plan->dyn_lds = (size_t)(2 * sh->batch + 1 + 2 * sh->n_kv_heads) * 4;
  const size_t lds = stat + plan->dyn_lds;
  if (lds > kLdsBytes) return fail(DP_ENOTSUP, "paged_decode: %zu bytes of LDS per workgroup", lds);
  int dev = -1;
  const int cus = device_cus(&dev);
  const int per_cu = blocks_per_cu(dev, fp8, st - 1, lds);
  // persistent grid: every workgroup resident at once, and no slice longer
  // than kMaxUnitsPerWave
  int64_t grid = (int64_t)cus * per_cu;
  const int64_t need = (max_units + (int64_t)kWaves * kMaxUnitsPerWave - 1) / ((int64_t)kWaves * kMaxUnitsPerWave);
  grid = std::max(grid, need);
  const int64_t useful = (max_units + (int64_t)kWaves * plan->min_chunk - 1) / ((int64_t)kWaves * plan->min_chunk);
  grid = std::max<int64_t>(1, std::min(grid, std::max(useful, need)));
  plan->grid = (int)grid;
  const int G = sh->n_q_heads / sh->n_kv_heads;
  const size_t recs = (size_t)grid * kWaves * 2 * G;
  plan->rec_o_off = 0;
  plan->rec_ml_off = align256(recs * kHeadDim * sizeof(float));
  plan->plan_off = plan->rec_ml_off + align256(recs * 2 * sizeof(float));
  plan->hdr_off = plan->plan_off + align256((size_t)(sh->batch + 2) * sizeof(int32_t));
  plan->ws_bytes = plan->hdr_off + align256((size_t)grid * kWaves * 4 * sizeof(int32_t));
  return DP_OK;
}

template <bool FP8, int ST>
void launch_stream(const Plan& plan, hipStream_t stream, const StreamArgs& args) {
  hipLaunchKernelGGL((paged_decode_stream_kernel<FP8, ST>), dim3(plan.grid), dim3(kWaves * 64), plan.dyn_lds,
                     stream, args);
}

// Validate everything the host can check and fill the kernel arguments.
int prepare(const void* q, const void* k_blocks, const void* v_blocks, const int32_t* block_tables,
            const int32_t* context_lens, float scale, const float* k_scale, const float* v_scale, void* out,
            const dp_decode_shape* shape, void* workspace, size_t workspace_bytes, Plan* plan, StreamArgs* args) {
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
  if (!workspace || workspace_bytes < plan->ws_bytes)
    return fail(DP_ENOMEM, "paged_decode: workspace needs %zu bytes, got %zu", plan->ws_bytes, workspace_bytes);
  if ((uintptr_t)workspace & 255) return fail(DP_EINVAL, "paged_decode: workspace must be 256-byte aligned");
  StreamArgs& a = *args;
  a.q = (const uint16_t*)q;
  a.k = (const char*)k_blocks;
  a.v = (const char*)v_blocks;
  a.block_tables = block_tables;
  a.context_lens = context_lens;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.out = out;
  a.rec_o = (float*)((char*)workspace + plan->rec_o_off);
  a.rec_ml = (float*)((char*)workspace + plan->rec_ml_off);
  a.plan = (int32_t*)((char*)workspace + plan->plan_off);
  a.hdr = (int32_t*)((char*)workspace + plan->hdr_off);
  a.qk_scale_log2 = scale * kLog2e;
  a.batch = shape->batch;
  a.hq = shape->n_q_heads;
  a.hkv = shape->n_kv_heads;
  a.group = shape->n_q_heads / shape->n_kv_heads;
  a.max_blocks_per_seq = shape->max_blocks_per_seq;
  a.max_ctx = shape->max_context_len;
  a.num_blocks_m1 = (int32_t)(shape->num_blocks - 1);
  a.out_fp32 = shape->out_dtype == DP_OUT_FP32;
  a.min_chunk = plan->min_chunk;
  return DP_OK;
}

int launch_partition_phase(const dp_decode_shape* shape, const Plan& plan, const StreamArgs& args, hipStream_t st) {
  const bool fp8 = shape->kv_dtype == DP_KV_FP8_E4M3;
  (void)hipGetLastError();  // clear a stale error left by earlier work
  switch ((plan.stages - 1) * 2 + (fp8 ? 1 : 0)) {
    case 2: launch_stream<false, 1>(plan, st, args); break;
    case 3: launch_stream<true, 1>(plan, st, args); break;
    case 4: launch_stream<false, 2>(plan, st, args); break;
    case 5: launch_stream<true, 2>(plan, st, args); break;
    case 6: launch_stream<false, 3>(plan, st, args); break;
    default: launch_stream<true, 3>(plan, st, args); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dpool::fail(DP_EIO, "paged_decode: stream kernel launch failed: %s", hipGetErrorString(e));
  return DP_OK;
}

int launch_merge_phase(const Plan& plan, const StreamArgs& args, hipStream_t st) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(paged_decode_merge_kernel, dim3(plan.grid * kWaves), dim3(256), 0, st, args);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return dpool::fail(DP_EIO, "paged_decode: merge launch failed: %s", hipGetErrorString(e));
  return DP_OK;
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
  return plan.min_chunk * plan.unit_tokens;
}

extern "C" int paged_decode_attention(const void* q, const void* k_blocks, const void* v_blocks,
                                      const int32_t* block_tables, const int32_t* context_lens, float scale,
                                      const float* k_scale, const float* v_scale, void* out,
                                      const dp_decode_shape* shape, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  Plan plan;
  StreamArgs args;
  int rc = prepare(q, k_blocks, v_blocks, block_tables, context_lens, scale, k_scale, v_scale, out, shape, workspace,
                   workspace_bytes, &plan, &args);
  if (rc != DP_OK || shape->batch == 0) return rc;
  rc = launch_partition_phase(shape, plan, args, (hipStream_t)stream);
  if (rc != DP_OK) return rc;
  return launch_merge_phase(plan, args, (hipStream_t)stream);
}

extern "C" int paged_decode_partition(const void* q, const void* k_blocks, const void* v_blocks,
                                      const int32_t* block_tables, const int32_t* context_lens, float scale,
                                      const float* k_scale, const float* v_scale, void* out,
                                      const dp_decode_shape* shape, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  Plan plan;
  StreamArgs args;
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
  if (shape->batch == 0) return DP_OK;
  if (!context_lens || !out) return fail(DP_EINVAL, "paged_decode_merge: null tensor pointer");
  if (((uintptr_t)out & 15) || ((uintptr_t)context_lens & 3))
    return fail(DP_EINVAL, "paged_decode_merge: out must be 16-byte and context_lens 4-byte aligned");
  if (!workspace || workspace_bytes < plan.ws_bytes)
    return fail(DP_ENOMEM, "paged_decode_merge: workspace needs %zu bytes, got %zu", plan.ws_bytes, workspace_bytes);
  if ((uintptr_t)workspace & 255) return fail(DP_EINVAL, "paged_decode_merge: workspace must be 256-byte aligned");
  StreamArgs a = {};
  a.rec_o = (float*)((char*)workspace + plan.rec_o_off);
  a.rec_ml = (float*)((char*)workspace + plan.rec_ml_off);
  a.plan = (int32_t*)((char*)workspace + plan.plan_off);
  a.hdr = (int32_t*)((char*)workspace + plan.hdr_off);
  a.context_lens = context_lens;
  a.out = out;
  a.batch = shape->batch;
  a.hq = shape->n_q_heads;
  a.hkv = shape->n_kv_heads;
  a.group = shape->n_q_heads / shape->n_kv_heads;
  a.max_ctx = shape->max_context_len;
  a.out_fp32 = shape->out_dtype == DP_OUT_FP32;
  a.min_chunk = plan.min_chunk;
  return launch_merge_phase(plan, a, (hipStream_t)stream);
}
