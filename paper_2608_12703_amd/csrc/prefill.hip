// Encoder keys / values of every decoder layer on the gfx950 matrix cores (bf16 models).
//
// Setup, once per utterance: C[f][n] = sum_k enc[f][k] W_xkv[n][k] + b_xkv[n], with
// enc bf16 [frames_cap][d] and W_xkv bf16 [2d][d] row-major; columns n < d are the keys,
// the rest the values, written as bf16 into the cross-K/V cache layout (cross_off).  This
// is a large dense contraction (frames_cap x 2d x d per layer), so it is tiled the
// plain way: a workgroup owns 256 frames x 128 columns, its eight waves 64 x 64 each
// (4 x 4 tiles of v_mfma_f32_16x16x32_bf16).  Both operands move in 32-wide K steps
// through four-stage LDS rings filled by direct global->LDS loads three steps ahead: a
// row-major bf16 row segment of 8 values is exactly one lane's MFMA operand, so every
// load is one 16-byte piece per lane and lands in the order the products read it.  The
// encoder states are bf16 already, so no low half is needed (one product per tile).
#include "common.h"
#include "launch.h"

namespace ad {

namespace {

constexpr int kXM = 256;   // frames per workgroup (16 row tiles)
constexpr int kXN = 128;   // output columns per workgroup (8 column tiles)

// the s_waitcnt immediate: vmcnt in bits 3:0 and 15:14, no wait on exports, lgkmcnt 0
constexpr int xkv_waitcnt(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0070; }

// One K step of a wave: 4 row tiles (row group rg) x 4 column tiles (half ch).
__device__ __forceinline__ void xkv_step(f32x4 (&acc)[4][4], const uint4* sa, const uint4* sb, int rg,
                                         int ch, int lane) {
  bf16x8 b[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) b[ct] = as_bf16x8(sb[(ch * 4 + ct) * 64 + lane]);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const bf16x8 a = as_bf16x8(sa[(rg * 4 + r) * 64 + lane]);
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[r][ct] = mfma_bf16(a, b[ct], acc[r][ct]);
  }
}

}  // namespace

__global__ void __launch_bounds__(512) xkv_mfma_kernel(int M, int N, int K, const uint16_t* A,
                                                       const uint16_t* W, const uint16_t* bias,
                                                       uint16_t* cache, int layer, int H, int d,
                                                       int frames_cap) {
  // distinct LDS objects per ring stage, so the compiler can tell a read of one stage from
  // the direct loads still filling another
  __shared__ uint4 sa0[16 * 64], sa1[16 * 64], sa2[16 * 64], sa3[16 * 64];
  __shared__ uint4 sb0[8 * 64], sb1[8 * 64], sb2[8 * 64], sb3[8 * 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int rg = w & 3, ch = w >> 2;
  const int c16 = lane & 15, grp = lane >> 4;
  const int n0 = blockIdx.x * kXN, m0 = blockIdx.y * kXM;
  const int KB = K / 32;
  // wave w stages row tiles w and w + 8 and column tile w; rows / columns past the matrix
  // read its last row / column (valid addresses; those results are never stored)
  const uint16_t* pa0 = A + (size_t)min(m0 + w * 16 + c16, M - 1) * K + grp * 8;
  const uint16_t* pa1 = A + (size_t)min(m0 + (w + 8) * 16 + c16, M - 1) * K + grp * 8;
  const uint16_t* pb = W + (size_t)min(n0 + w * 16 + c16, N - 1) * K + grp * 8;
  auto issue = [&](uint4* sa, uint4* sb, int kb) {   // stage kb (clamped): three loads per wave
    const int k = min(kb, KB - 1) * 32;
    dma16(pa0 + k, sa + w * 64);
    dma16(pa1 + k, sa + (w + 8) * 64);
    dma16(pb + k, sb + w * 64);
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  issue(sa0, sb0, 0);
  issue(sa1, sb1, 1);
  issue(sa2, sb2, 2);
  int kb = 0;
  // Step j: wait until stage j has landed (stages j + 1 and j + 2, six loads, may still be
  // in flight) and every wave is past step j - 1, refill step j - 1's slot with stage
  // j + 3, multiply stage j.
#define XKV_STEP(SA, SB, NA, NB)                              \
  {                                                           \
    __builtin_amdgcn_s_waitcnt(xkv_waitcnt(6));               \
    __builtin_amdgcn_s_barrier();                             \
    asm volatile("" ::: "memory");                            \
    issue(NA, NB, kb + 3);                                    \
    xkv_step(acc, SA, SB, rg, ch, lane);                      \
    ++kb;                                                     \
  }
  for (int it = 0; it < KB / 4; ++it) {
    XKV_STEP(sa0, sb0, sa3, sb3)
    XKV_STEP(sa1, sb1, sa0, sb0)
    XKV_STEP(sa2, sb2, sa1, sb1)
    XKV_STEP(sa3, sb3, sa2, sb2)
  }
  const int rem = KB % 4;
  if (rem >= 1) XKV_STEP(sa0, sb0, sa3, sb3)
  if (rem >= 2) XKV_STEP(sa1, sb1, sa0, sb0)
  if (rem >= 3) XKV_STEP(sa2, sb2, sa1, sb1)
#undef XKV_STEP
  __builtin_amdgcn_s_waitcnt(xkv_waitcnt(0));

  // epilogue: bias, bf16 rounding, the cross-K/V layout (keys for n < d, values after)
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    const int n = n0 + (ch * 4 + ct) * 16 + c16;
    if (n >= N) continue;
    const float bn = bf16_to_f32(bias[n]);
    const int kv = n / d, h = (n % d) / kHead, j = n % kHead;
    uint16_t* base = cache + cross_base(layer, h, H, frames_cap);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + (rg * 4 + r) * 16 + grp * 4 + i;
        if (m < M) base[cross_off(kv, m, j)] = f32_to_bf16(acc[r][ct][i] + bn);
      }
  }
}

void launch_xkv_mfma(int M, int N, int K, const uint16_t* A, const uint16_t* W, const uint16_t* bias,
                     uint16_t* cache, int layer, int H, int d, int frames_cap, hipStream_t st) {
  const dim3 grid((N + kXN - 1) / kXN, (M + kXM - 1) / kXM), block(512);
  hipLaunchKernelGGL(xkv_mfma_kernel, grid, block, 0, st, M, N, K, A, W, bias, cache, layer, H, d,
                     frames_cap);
}

}  // namespace ad
