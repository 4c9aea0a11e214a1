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
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))  // NaN stays a quiet NaN
    return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

struct BF16 {
  using T = uint16_t;
  static __device__ __forceinline__ float ld(const T* p, size_t i) { return bf16_to_f32(p[i]); }
  static __device__ __forceinline__ void st(T* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// ----------------------------------------------------------------- reductions
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
// Self-KV pool: [layer][K|V][page][head][tile]; cross-KV: [layer][K|V][head][frame].
// Inside a 16 x 64 tile element (token t, lane j) sits at t * 64 + j.

__device__ __forceinline__ size_t kv_tile_base(int layer, int kv, int page, int head,
                                               int num_pages, int H) {
  return ((((size_t)layer * 2 + kv) * num_pages + page) * H + head) * (size_t)kTileElems;
}
__device__ __forceinline__ size_t cross_base(int layer, int kv, int head, int H, int frames_cap) {
  return (((size_t)layer * 2 + kv) * H + head) * (size_t)frames_cap * kHead;
}
__device__ __forceinline__ int tile_off(int t, int j) { return t * kHead + j; }

// ----------------------------------------------------------------- step descriptors
// Built by the prep kernel from the caller's device arrays, after validation.

struct SeqDesc {
  int row0;     // first row of the sequence
  int k;        // drafts (rows - 1)
  int n;        // committed KV length
  int T;        // encoder frames
  int enc_off;  // first cross-KV slot
  int valid;    // 0 -> skipped (error bits were raised)
  int pad0, pad1;
};

struct RowDesc {
  int seq;      // owning sequence, or -1 for a padding row
  int i;        // index inside the block (0 = pending token)
  int pos;      // decoder position n + i
  int token;    // token id (clamped into the vocabulary)
};

}  // namespace ad
