// Device helpers shared by the libad kernels: storage types, bf16 rounding, wave and
// block reductions, and the cache tile layouts.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ad {

constexpr int kHead = 64;        // head width
constexpr int kTile = 16;        // tokens per self-KV page / frames per cross-KV tile
constexpr int kTileElems = kTile * kHead;
constexpr int kWave = 64;

// ----------------------------------------------------------------- storage types

struct F32 {
  using T = float;
  static __device__ __forceinline__ float ld(const T* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void st(T* p, size_t i, float v) { p[i] = v; }
};

// bf16 kept as raw 16-bit words; conversion is a shift, rounding is nearest-even.
__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}
// gfx950 converts in hardware (v_cvt_pk_bf16_f32): round to nearest even, NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}
// two values in one conversion: a in the low half, b in the high half
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{a, b}), b2));
}

struct BF16 {
  using T = uint16_t;
  static __device__ __forceinline__ float ld(const T* p, size_t i) { return bf16_to_f32(p[i]); }
  static __device__ __forceinline__ void st(T* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// ----------------------------------------------------------------- reductions
// Combine a value across the four 16-lane rows of a wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48) with the gfx950 row-swap instructions; every lane gets the same result,
// combined in the same order.
__device__ __forceinline__ float rows4_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Fixed butterfly trees: the result depends only on the values, not on which other
// rows share the launch (the step is batch-invariant by construction).

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over a block of NW waves; every thread gets the total.  `red` holds NW floats.
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += red[i];
  return t;
}

// ----------------------------------------------------------------- cache layouts
// Self-KV pool: [layer][K|V][page][head][tile]; a 16-token x 64-lane tile holds keys
// token-major (t * 64 + j: a token's 64 lanes are one 128-byte line) and values
// lane-major (j * 16 + t: the 16 tokens of one lane are contiguous).
// Cross-KV: [layer][head][32-frame block][K|V], 2048 elements each for the keys and the
// values of a block, in the operand order of the attention products (see cross_off): a
// wave streams one contiguous range per key chunk and every load reads 1 KB contiguous.

constexpr int kCrossBlock = 32;                        // frames per cross-K/V block
constexpr int kCrossBlockElems = kCrossBlock * kHead;  // 2048

__device__ __forceinline__ size_t kv_tile_base(int layer, int kv, int page, int head,
                                               int num_pages, int H) {
  return ((((size_t)layer * 2 + kv) * num_pages + page) * H + head) * (size_t)kTileElems;
}
// start of one layer's, one head's cross K/V (keys and values of frames_cap frames)
__device__ __forceinline__ size_t cross_base(int layer, int head, int H, int frames_cap) {
  return ((size_t)layer * H + head) * (size_t)frames_cap * kHead * 2;
}
__device__ __forceinline__ int tile_off(int kv, int t, int j) {
  return kv == 0 ? t * kHead + j : j * kTile + t;
}
// Element (frame f, lane j) of one head's cross K (kv = 0) or V (kv = 1).  Within a
// 32-frame block the score product takes its 16 key rows in two passes tt, row c16
// holding frame 8 (c16 / 4) + 4 tt + c16 % 4, lane group g supplying lanes
// 16 g .. 16 g + 15 in two 8-lane halves: keys sit at (tt, half, g * 16 + c16, 8 lanes).
// The value product takes, per 16-lane tile dt, lane dt * 16 + c16 and frames
// 8 g .. 8 g + 7: values sit at (dt, g * 16 + c16, 8 frames).
__device__ __forceinline__ size_t cross_off(int kv, int f, int j) {
  const size_t o = ((size_t)(f / kCrossBlock) * 2 + kv) * kCrossBlockElems;
  const int t = f % kCrossBlock;
  if (kv == 0) {
    const int c16 = 4 * (t / 8) + (t & 3), tt = (t / 4) & 1;
    return o + ((tt * 2 + ((j / 8) & 1)) * 64 + (j / 16) * 16 + c16) * 8 + (j & 7);
  }
  return o + ((j / 16) * 64 + (t / 8) * 16 + (j & 15)) * 8 + (t & 7);
}

// ----------------------------------------------------------------- MFMA operands
// gfx950 v_mfma_f32_16x16x32_bf16: lane l supplies 8 bf16 of row (l % 16) of A and 8 of
// column (l % 16) of B for the same 8 reduction slots, and receives D rows
// 4 (l / 16) .. 4 (l / 16) + 3 of column l % 16.  Lane group g = l / 16 supplies
// reduction elements 8 g .. 8 g + 7 of each 32-wide block.

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Float32 activations enter bf16 products as a pair hi = bf16(v), lo = bf16(v - hi)
// (v - hi is exact in float32), which carries 16 significant bits into the product.
__device__ __forceinline__ void split_hilo(float v, uint16_t& hi, uint16_t& lo) {
  hi = f32_to_bf16(v);
  lo = f32_to_bf16(v - bf16_to_f32(hi));
}

// "A-fragment" order of an activation matrix X [M][K] (K a multiple of 32, RT row tiles):
// for every 32-wide K block kb and 16-row tile rt, two 1 KB runs (hi, lo) of 64 lanes x 8
// bf16 in the order the MFMA A operand is read; the RT tiles of one K block are
// contiguous, so a workgroup stages a block of rows with one contiguous copy.
__device__ __forceinline__ size_t afrag_index(int m, int k, int hilo, int RT) {
  const int kb = k >> 5, kk = k & 31, g = kk >> 3, j = kk & 7;
  const int rt = m >> 4, r = m & 15;
  return (((size_t)kb * RT + rt) * 2 + hilo) * 512 + (size_t)(g * 16 + r) * 8 + j;
}
__device__ __forceinline__ void afrag_store(uint16_t* base, int RT, int m, int k, float v) {
  uint16_t hi, lo;
  split_hilo(v, hi, lo);
  base[afrag_index(m, k, 0, RT)] = hi;
  base[afrag_index(m, k, 1, RT)] = lo;
}
// Four consecutive values v.x .. v.w at columns k .. k + 3 (k % 4 == 0) of row m: one
// 8-byte store each for hi and lo (the four lie in one run of eight).
__device__ __forceinline__ void afrag_store4(uint16_t* base, int RT, int m, int k, float4 v) {
  uint16_t h[4], l[4];
  split_hilo(v.x, h[0], l[0]);
  split_hilo(v.y, h[1], l[1]);
  split_hilo(v.z, h[2], l[2]);
  split_hilo(v.w, h[3], l[3]);
  *(uint2*)(base + afrag_index(m, k, 0, RT)) =
      make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
  *(uint2*)(base + afrag_index(m, k, 1, RT)) =
      make_uint2((uint32_t)l[0] | ((uint32_t)l[1] << 16), (uint32_t)l[2] | ((uint32_t)l[3] << 16));
}

// Direct global -> LDS copy of 16 bytes per lane: lane l's bytes land at lds_wave + 16 l
// (lds_wave must be the same for the whole wave).
__device__ __forceinline__ void dma16(const void* g, void* lds_wave) {
  __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)g,
                                   (void __attribute__((address_space(3)))*)lds_wave, 16, 0, 0);
}

// ----------------------------------------------------------------- split-K sums
// v[u] = sum over splits t of P[t][e], in split order; the loads of eight splits are
// issued before their sums.
__device__ __forceinline__ float4 split_sum4(const float* P, size_t plane, size_t e, int nsplit) {
  float4 acc = *(const float4*)(P + e);
  for (int t0 = 1; t0 < nsplit; t0 += 8) {
    float4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = *(const float4*)(P + (size_t)min(t0 + u, nsplit - 1) * plane + e);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (t0 + u < nsplit) { acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w; }
  }
  return acc;
}

// ----------------------------------------------------------------- step descriptors
// Built by the prep kernel from the caller's device arrays, after validation.

struct SeqDesc {
  int row0;     // first row of the sequence
  int k;        // drafts (rows - 1)
  int n;        // committed KV length
  int T;        // encoder frames
  int enc_off;  // first cross-KV slot
  int valid;    // 0 -> skipped (error bits were raised)
  int wlo, whi; // cross-attention frames [wlo, whi) (0, T unless a window is given)
};

struct RowDesc {
  int seq;      // owning sequence, or -1 for a padding row
  int i;        // index inside the block (0 = pending token)
  int pos;      // decoder position: n + i, or n + depth in a draft tree
  int token;    // token id (clamped into the vocabulary)
  int slot;     // cache slot of the row's keys / values: n + i
};

// A row of a draft-tree block: its depth below the root and its ancestor mask (bit j:
// block row j is the row itself or one of its ancestors).
struct RowTree {
  unsigned long long mask;
  int depth, pad;
};

}  // namespace ad
