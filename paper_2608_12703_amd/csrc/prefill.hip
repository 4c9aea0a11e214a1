// Encoder keys / values of every decoder layer on the gfx950 matrix cores (bf16 models).
//
// Setup, once per utterance: C[f][n] = sum_k enc[f][k] W_xkv[n][k] + b_xkv[n], with
// enc bf16 [frames_cap][d] and W_xkv bf16 [2d][d] row-major; columns n < d are the keys,
// the rest the values, written as bf16 into the cross-K/V cache layout (cross_off).  This
// is a large dense contraction (frames_cap x 2d x d per layer), so it is tiled the
// plain way: a workgroup owns 256 frames x 256 columns, its eight waves 128 x 64 each
// (8 x 4 tiles of v_mfma_f32_16x16x32_bf16: 12 operand reads per 32 products).  Both
// operands move in 32-wide K steps through four-stage LDS rings (32 KB a stage) filled
// by direct global->LDS loads three steps ahead: a bf16 row segment of 8 values is
// exactly one lane's MFMA operand, so every load is one 16-byte piece per lane and lands
// in the order the products read it.  The encoder states are bf16 already, so no low
// half is needed (one product per tile).
//
// Operand layouts.  Row-major operands make each 1 KB load gather 16 rows x 64 bytes,
// which streams at a quarter of the rate of a contiguous 1 KB (measured: about 15-28
// against 60 bytes per clock per CU from L2).  So both operands are read in "fragment
// order" when they are available that way: the weights as tiled by ad_model_pack (the
// 128-column x 32-wide K blocks of pack_weight_kernel), the encoder states as copied by
// pack_rows_kernel (for each 32-wide K step and 16-row tile, the 1 KB the products read,
// in lane order).  Row-major operands remain supported.
//
// Stores.  In the cache layout four consecutive frames of one value lane, and four
// consecutive lanes of one key frame, are contiguous.  A value tile keeps the usual
// operand order (a lane's four accumulators are four consecutive frames); a key tile
// swaps the two operands of every product, so a lane's four accumulators are four
// consecutive key lanes.  Either way a lane stores 8 bytes at a time, and a wave's
// stores cover whole runs of the block.
//
// Workgroup order.  Workgroups are dealt round-robin over the 8 XCDs; each XCD takes a
// contiguous range of tiles, ordered column group (two halves of the columns), then
// frame block, then column tile, so an XCD's concurrent workgroups share their frame
// blocks and half of the weight matrix through its L2.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace ad {

namespace {

constexpr int kXM = 256;   // frames per workgroup (16 row tiles)
constexpr int kXN = 256;   // output columns per workgroup (16 column tiles)
constexpr int kPackN = 128;   // columns per tile of the packed weights (pack_weight_kernel)

// the s_waitcnt immediate: vmcnt in bits 3:0 and 15:14, no wait on exports, lgkmcnt 0
constexpr int xkv_waitcnt(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0070; }

// One K step of a wave: 8 row tiles (row half wr) x 4 column tiles (quarter wc).  TR: the
// operands swap places (accumulator element i then runs along the columns).
template <bool TR>
__device__ __forceinline__ void xkv_step(f32x4 (&acc)[8][4], const uint4* sa, const uint4* sb, int wr,
                                         int wc, int lane) {
  bf16x8 b[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) b[ct] = as_bf16x8(sb[(wc * 4 + ct) * 64 + lane]);
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const bf16x8 a = as_bf16x8(sa[(wr * 8 + r) * 64 + lane]);
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[r][ct] = TR ? mfma_bf16(b[ct], a, acc[r][ct]) : mfma_bf16(a, b[ct], acc[r][ct]);
  }
}

// The K loop and the stores of one tile (TR: a key tile with swapped operands; APK / WPK:
// encoder states / weights in fragment order).
template <bool TR, bool APK, bool WPK>
__device__ __forceinline__ void xkv_tile(int M, int N, int K, const uint16_t* A, const uint16_t* W,
                                         const uint16_t* bias, uint16_t* cache, int layer, int H, int d,
                                         int frames_cap, int m0, int n0, uint4* const (&sa)[4],
                                         uint4* const (&sb)[4]) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wr = w >> 2, wc = w & 3;
  const int c16 = lane & 15, grp = lane >> 4;
  const int KB = K / 32;
  // Wave w stages row tiles w and w + 8 and column tiles w and w + 8.  Rows / columns past
  // the matrix read its last row / column (valid addresses; those results are never
  // stored).  Per K step the source advances by `as` / `ws` elements.
  const int RT = M / 16, CT = (N + kPackN - 1) / kPackN;   // 16-row tiles, 128-column tiles
  const uint16_t *pa0, *pa1, *pb0, *pb1;
  size_t as, ws;
  if (APK) {
    pa0 = A + ((size_t)min(m0 / 16 + w, RT - 1) * 64 + lane) * 8;
    pa1 = A + ((size_t)min(m0 / 16 + w + 8, RT - 1) * 64 + lane) * 8;
    as = (size_t)RT * 512;
  } else {
    pa0 = A + (size_t)min(m0 + w * 16 + c16, M - 1) * K + grp * 8;
    pa1 = A + (size_t)min(m0 + (w + 8) * 16 + c16, M - 1) * K + grp * 8;
    as = 32;
  }
  if (WPK) {
    // column tile c of the workgroup: 128-column tile (n0 / 16 + c) / 8, 16-column tile
    // (n0 / 16 + c) % 8 inside it
    const int c0 = n0 / 16 + w, c1 = n0 / 16 + w + 8;
    pb0 = W + (((size_t)min(c0 / 8, CT - 1) * KB) * 512 + (c0 % 8) * 64 + lane) * 8;
    pb1 = W + (((size_t)min(c1 / 8, CT - 1) * KB) * 512 + (c1 % 8) * 64 + lane) * 8;
    ws = 512 * 8;
  } else {
    pb0 = W + (size_t)min(n0 + w * 16 + c16, N - 1) * K + grp * 8;
    pb1 = W + (size_t)min(n0 + (w + 8) * 16 + c16, N - 1) * K + grp * 8;
    ws = 32;
  }
  auto issue = [&](int s, int kb) {   // stage kb (clamped) into ring slot s: four loads per wave
    const size_t k = min(kb, KB - 1);
    dma16(pa0 + k * as, sa[s] + w * 64);
    dma16(pa1 + k * as, sa[s] + (w + 8) * 64);
    dma16(pb0 + k * ws, sb[s] + w * 64);
    dma16(pb1 + k * ws, sb[s] + (w + 8) * 64);
  };
  f32x4 acc[8][4];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  issue(0, 0);
  issue(1, 1);
  issue(2, 2);
  int kb = 0;
  // Step j: wait until stage j has landed (stages j + 1 and j + 2, eight loads, may still
  // be in flight) and every wave is past step j - 1, refill step j - 1's slot with stage
  // j + 3, multiply stage j.  The loop is unrolled over the ring, so every slot is a
  // compile-time choice.
#define XKV_STEP(S)                                           \
  {                                                           \
    __builtin_amdgcn_s_waitcnt(xkv_waitcnt(8));               \
    __builtin_amdgcn_s_barrier();                             \
    asm volatile("" ::: "memory");                            \
    issue(((S) + 3) % 4, kb + 3);                             \
    xkv_step<TR>(acc, sa[S], sb[S], wr, wc, lane);            \
    ++kb;                                                     \
  }
  for (int it = 0; it < KB / 4; ++it) {
    XKV_STEP(0)
    XKV_STEP(1)
    XKV_STEP(2)
    XKV_STEP(3)
  }
  const int rem = KB % 4;
  if (rem >= 1) XKV_STEP(0)
  if (rem >= 2) XKV_STEP(1)
  if (rem >= 3) XKV_STEP(2)
#undef XKV_STEP
  __builtin_amdgcn_s_waitcnt(xkv_waitcnt(0));

  // epilogue: bias, bf16 rounding, the cross-K/V layout (keys for n < d, values after).
  // Accumulator (r, ct, i) of this lane is frame m0 + 16 (8 wr + r) + {4 grp + i | c16}
  // and column n0 + 16 (4 wc + ct) + {c16 | 4 grp + i} (value | key tile).
  // (a tile that holds both keys and values keeps the usual order, in which a lane's four
  // key frames are not contiguous: it stores element by element)
  const bool whole = m0 + kXM <= M && n0 + kXN <= N && (TR || n0 >= d);
  if (whole) {
    // four contiguous elements per store
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const int nb = n0 + (wc * 4 + ct) * 16 + (TR ? grp * 4 : c16);
      const int kv = nb / d, h = (nb % d) / kHead, j = nb % kHead;
      uint16_t* base = cache + cross_base(layer, h, H, frames_cap);
      float bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) bv[i] = bf16_to_f32(bias[TR ? nb + i : nb]);
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int m = m0 + (wr * 8 + r) * 16 + (TR ? c16 : grp * 4);
        const f32x4 v = acc[r][ct];
        const uint2 pk = make_uint2(f32x2_to_bf16x2(v[0] + bv[0], v[1] + bv[1]),
                                    f32x2_to_bf16x2(v[2] + bv[2], v[3] + bv[3]));
        *(uint2*)(base + cross_off(kv, m, j)) = pk;
      }
    }
    return;
  }
  // a tile past the last frame or column, or across the key / value boundary: one
  // element at a time
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int n = n0 + (wc * 4 + ct) * 16 + (TR ? grp * 4 + i : c16);
        const int m = m0 + (wr * 8 + r) * 16 + (TR ? c16 : grp * 4 + i);
        if (n >= N || m >= M) continue;
        const int kv = n / d, h = (n % d) / kHead, j = n % kHead;
        cache[cross_base(layer, h, H, frames_cap) + cross_off(kv, m, j)] =
            f32_to_bf16(acc[r][ct][i] + bf16_to_f32(bias[n]));
      }
}

}  // namespace

template <bool APK, bool WPK>
__global__ void __launch_bounds__(512) xkv_mfma_kernel(int M, int N, int K, const uint16_t* A,
                                                       const uint16_t* W, const uint16_t* bias,
                                                       uint16_t* cache, int layer, int H, int d,
                                                       int frames_cap) {
  // distinct LDS objects per ring stage, so the compiler can tell a read of one stage from
  // the direct loads still filling another
  __shared__ uint4 sa0[16 * 64], sa1[16 * 64], sa2[16 * 64], sa3[16 * 64];
  __shared__ uint4 sb0[16 * 64], sb1[16 * 64], sb2[16 * 64], sb3[16 * 64];
  uint4* const sa[4] = {sa0, sa1, sa2, sa3};
  uint4* const sb[4] = {sb0, sb1, sb2, sb3};
  // tile of this workgroup (see the header: XCD ranges, column group, frame block, column)
  const int NT = (N + kXN - 1) / kXN, MB = (M + kXM - 1) / kXM;
  const int nwg = NT * MB, bid = blockIdx.x;
  const int x = bid & 7, q8 = nwg >> 3, r8 = nwg & 7;
  const int lin = x * q8 + min(x, r8) + (bid >> 3);
  const int gc = (NT + 1) / 2;
  const int g = lin / (MB * gc), rem = lin - g * MB * gc;
  const int gw = min(gc, NT - g * gc);
  const int m0 = (rem / gw) * kXM, n0 = (g * gc + rem % gw) * kXN;
  // a key tile (every column a key) swaps the product operands for its stores
  if (n0 + kXN <= d)
    xkv_tile<true, APK, WPK>(M, N, K, A, W, bias, cache, layer, H, d, frames_cap, m0, n0, sa, sb);
  else
    xkv_tile<false, APK, WPK>(M, N, K, A, W, bias, cache, layer, H, d, frames_cap, m0, n0, sa, sb);
}

// Encoder states [M][K] (M a multiple of 16) in fragment order: for 32-wide K step kb and
// 16-row tile rt, 64 lanes x 8 values at ((kb * RT + rt) * 64 + lane) * 8, lane l holding
// row 16 rt + l % 16, columns 32 kb + 8 (l / 16) .. + 7.  Each thread moves one 16-byte
// piece; consecutive threads read consecutive pieces of a row.
__global__ void __launch_bounds__(256) pack_rows_kernel(const uint16_t* A, int M, int K, uint16_t* P) {
  const int RT = M / 16;
  const size_t pieces = (size_t)M * K / 8;
  for (size_t q = (size_t)blockIdx.x * 256 + threadIdx.x; q < pieces; q += (size_t)gridDim.x * 256) {
    const int m = (int)(q / (K / 8)), k8 = (int)(q % (K / 8));
    const int kb = k8 / 4, g = k8 % 4, rt = m / 16, r = m % 16;
    const uint4 v = *(const uint4*)(A + q * 8);
    *(uint4*)(P + (((size_t)kb * RT + rt) * 64 + g * 16 + r) * 8) = v;
  }
}

void launch_xkv_mfma(int M, int N, int K, const uint16_t* A, bool a_packed, const uint16_t* W,
                     bool w_packed, const uint16_t* bias, uint16_t* cache, int layer, int H, int d,
                     int frames_cap, hipStream_t st) {
  const int tiles = ((N + kXN - 1) / kXN) * ((M + kXM - 1) / kXM);
  const dim3 grid(tiles), block(512);
  if (a_packed && w_packed)
    hipLaunchKernelGGL((xkv_mfma_kernel<true, true>), grid, block, 0, st, M, N, K, A, W, bias, cache, layer, H,
                       d, frames_cap);
  else if (a_packed)
    hipLaunchKernelGGL((xkv_mfma_kernel<true, false>), grid, block, 0, st, M, N, K, A, W, bias, cache, layer,
                       H, d, frames_cap);
  else if (w_packed)
    hipLaunchKernelGGL((xkv_mfma_kernel<false, true>), grid, block, 0, st, M, N, K, A, W, bias, cache, layer,
                       H, d, frames_cap);
  else
    hipLaunchKernelGGL((xkv_mfma_kernel<false, false>), grid, block, 0, st, M, N, K, A, W, bias, cache, layer,
                       H, d, frames_cap);
}

void launch_pack_rows(const uint16_t* A, int M, int K, uint16_t* P, hipStream_t st) {
  const size_t pieces = (size_t)M * K / 8;
  const dim3 grid((unsigned)std::min<size_t>((pieces + 255) / 256, 16384)), block(256);
  hipLaunchKernelGGL(pack_rows_kernel, grid, block, 0, st, A, M, K, P);
}

}  // namespace ad
