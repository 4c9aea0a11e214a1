// Projections and the LM head of the bf16 model on the gfx950 matrix cores.
//
// C[m][n] = sum_k X[m][k] W[n][k] with W bf16 [N][K] and X float32 activations stored as
// a hi/lo bf16 pair in A-fragment order.  A workgroup owns 128 output columns and up to
// RTC 16-row tiles; each of its four waves owns a quarter of the rows across all 128
// columns.  Operands move in 32-wide K steps through LDS rings filled by direct
// global->LDS loads: activations (L2-resident) two steps ahead, weights (streamed from
// HBM) five steps ahead.  The waits are explicit; the loop is unrolled over the ring
// stages so every buffer is a distinct LDS object.  Small-N products split K over several
// workgroups and the last one to finish a tile sums the partial tiles in split order.
// The split count depends on the weight shape only, so a row's result never depends
// on how many other rows share the launch.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace ad {

constexpr int kNT = 128;          // output columns per workgroup (8 tiles of 16)

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

struct Top2s {
  float v1;
  int i1;
  float v2;
  int bad;
};
__device__ __forceinline__ Top2s t2_merge(Top2s a, Top2s b) {
  const bool a_wins = (a.v1 > b.v1) || (a.v1 == b.v1 && a.i1 < b.i1);
  Top2s r;
  r.bad = a.bad | b.bad;
  if (a_wins) { r.v1 = a.v1; r.i1 = a.i1; r.v2 = fmaxf(a.v2, b.v1); }
  else        { r.v1 = b.v1; r.i1 = b.i1; r.v2 = fmaxf(b.v2, a.v1); }
  return r;
}
__device__ __forceinline__ Top2s t2_shfl(Top2s t, int mask) {
  Top2s u;
  u.v1 = __shfl_xor(t.v1, mask, kWave);
  u.i1 = __shfl_xor(t.i1, mask, kWave);
  u.v2 = __shfl_xor(t.v2, mask, kWave);
  u.bad = __shfl_xor(t.bad, mask, kWave);
  return u;
}

// Wait until at most N vector-memory operations of this wave are outstanding (they
// complete in order) and its LDS operations are done, then barrier.  No memory fence.
#define BARRIER_VMCNT(N)                       \
  do {                                         \
    __builtin_amdgcn_s_waitcnt(0x0070 | (N));  \
    __builtin_amdgcn_s_barrier();              \
    asm volatile("" ::: "memory");             \
  } while (0)

template <int RTC>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[RTC / 4][8], const uint4* abuf,
                                         const uint4* wbuf, int w, int lane) {
  constexpr int RW = RTC / 4;
  bf16x8 b[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) b[ct] = as_bf16x8(wbuf[ct * 64 + lane]);
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int rt = w * RW + r;
    const bf16x8 ah = as_bf16x8(abuf[(rt * 2 + 0) * 64 + lane]);
    const bf16x8 al = as_bf16x8(abuf[(rt * 2 + 1) * 64 + lane]);
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      acc[r][ct] = mfma_bf16(ah, b[ct], acc[r][ct]);
      acc[r][ct] = mfma_bf16(al, b[ct], acc[r][ct]);
    }
  }
}

template <int EPI, int RTC>
__global__ void __launch_bounds__(256) gemm_mfma_kernel(GemmArgs g) {
  constexpr int RW = RTC / 4;            // row tiles per wave
  constexpr int NA = RTC / 2;            // direct loads per wave for one activation stage
  // Activation ring: 3 stages (requested 2 steps ahead); weight ring: 6 stages (requested
  // 5 steps ahead, covering HBM latency).  Distinct LDS objects, so the compiler can tell
  // a read of one stage from the direct loads still filling another.
  __shared__ uint4 sa0[RTC * 128], sa1[RTC * 128], sa2[RTC * 128];
  __shared__ uint4 sw0[512], sw1[512], sw2[512], sw3[512], sw4[512], sw5[512];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c16 = lane & 15, grp = lane >> 4;

  // (split, column tile, row chunk) of this workgroup.  Workgroups are dealt
  // round-robin over the 8 XCDs; renumbering them so each XCD holds a contiguous id
  // range keeps the row chunks of one weight tile, and the tiles of one K split, on one
  // L2.
  const int nwg = gridDim.x, bid = blockIdx.x;
  const int x = bid & 7, q8 = nwg >> 3, r8 = nwg & 7;
  const int lin = x * q8 + min(x, r8) + (bid >> 3);
  const int mc = lin % g.mchunks;
  const int s = (lin / g.mchunks) / g.ntiles, nt = (lin / g.mchunks) % g.ntiles;
  const int rt0 = mc * RTC, n0 = nt * kNT;
  const int kb0 = (s * g.KB) / g.S, kb1 = ((s + 1) * g.KB) / g.S;

  f32x4 acc[RW][8];
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = kb1 - kb0, kl = kb1 - 1;
  auto ia = [&](uint4* buf, int kb) {   // activation stage of step kb (clamped)
    const uint4* src = (const uint4*)g.A + ((size_t)min(kb, kl) * g.RT + rt0) * 128;
#pragma unroll
    for (int ii = 0; ii < NA; ++ii) {
      const int i = ii * 4 + w;
      dma16(src + i * 64 + lane, buf + i * 64);
    }
  };
  auto iw = [&](uint4* buf, int kb) {   // weight stage of step kb (clamped)
    const int k = min(kb, kl);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int ct = w * 2 + t;
      const int n = min(n0 + ct * 16 + (lane & 15), g.N - 1);
      dma16(g.W + (size_t)n * g.K + k * 32 + (lane >> 4) * 8, buf + ct * 64);
    }
  };
  // Step j requests activations j + 2 and weights j + 5, in that order; the prologue
  // plays virtual steps -5 .. -1 so the outstanding-load count is the same everywhere:
  // at the end of step j the loads issued after A(j+1) are W(j+4), A(j+2), W(j+5).
  constexpr int kWaitAfter = NA + 4;
  iw(sw0, kb0);
  iw(sw1, kb0 + 1);
  iw(sw2, kb0 + 2);
  ia(sa0, kb0);
  iw(sw3, kb0 + 3);
  ia(sa1, kb0 + 1);
  iw(sw4, kb0 + 4);
  BARRIER_VMCNT(kWaitAfter);
  int kb = kb0;
#define GEMM_STEP(CA, CW, NXA, NXW)        \
  {                                        \
    ia(NXA, kb + 2);                       \
    iw(NXW, kb + 5);                       \
    mma_step<RTC>(acc, CA, CW, w, lane);   \
    BARRIER_VMCNT(kWaitAfter);             \
    ++kb;                                  \
  }
  for (int it = 0; it < nk / 6; ++it) {
    GEMM_STEP(sa0, sw0, sa2, sw5)
    GEMM_STEP(sa1, sw1, sa0, sw0)
    GEMM_STEP(sa2, sw2, sa1, sw1)
    GEMM_STEP(sa0, sw3, sa2, sw2)
    GEMM_STEP(sa1, sw4, sa0, sw3)
    GEMM_STEP(sa2, sw5, sa1, sw4)
  }
  const int rem = nk % 6;
  if (rem >= 1) GEMM_STEP(sa0, sw0, sa2, sw5)
  if (rem >= 2) GEMM_STEP(sa1, sw1, sa0, sw0)
  if (rem >= 3) GEMM_STEP(sa2, sw2, sa1, sw1)
  if (rem >= 4) GEMM_STEP(sa0, sw3, sa2, sw2)
  if (rem >= 5) GEMM_STEP(sa1, sw4, sa0, sw3)
#undef GEMM_STEP
  BARRIER_VMCNT(0);

  // row / column of accumulator element (r, ct, i) of this lane
  const int row_base = (rt0 + w * RW) * 16 + grp * 4;   // + r * 16 + i
  const int col_base = n0 + c16;                        // + ct * 16

  // This kernel's LDS is also written by direct loads, so the compiler orders every LDS
  // access after outstanding global stores; epilogues therefore finish all their
  // cross-lane (LDS) work before the first store.
  if (EPI == EPI_ARGMAX) {
    // LM head: top-2 of this tile's 128 columns per row.  A row's columns sit in 16
    // lanes x 8 registers; registers are merged in column order, then the 16 lanes, so
    // ties keep the lower index.
    Top2s t[RW][4];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        t[r][i] = Top2s{-INFINITY, 0x7fffffff, -INFINITY, 0};
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
          const int n = col_base + ct * 16;
          const float v = acc[r][ct][i];
          Top2s u{v, n, -INFINITY, 0};
          if (!isfinite(v)) { u.v1 = -INFINITY; u.bad = 1; }
          if (n < g.N) t[r][i] = t2_merge(t[r][i], u);
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) t[r][i] = t2_merge(t[r][i], t2_shfl(t[r][i], o));
      }
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = row_base + r * 16 + i;
        if (c16 == 0 && m < g.M) {
          float4 rec{t[r][i].v1, __int_as_float(t[r][i].i1), t[r][i].v2, __int_as_float(t[r][i].bad)};
          ((float4*)g.e.am_part)[(size_t)m * g.ntiles + nt] = rec;
        }
      }
    if (g.e.out) {
#pragma unroll
      for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int ct = 0; ct < 8; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = row_base + r * 16 + i, n = col_base + ct * 16;
            if (m < g.M && n < g.N) g.e.out[(size_t)m * g.e.ldo + n] = acc[r][ct][i];
          }
    }
    return;
  }

  // EPI_PARTIAL: the raw split-K partial product straight from registers (16 lanes store
  // 64 contiguous bytes of a row); the consumer kernel sums the splits in split order.
  float* P = g.part + (size_t)s * g.M * g.N;
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = row_base + r * 16 + i;
      if (m >= g.M) continue;
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        const int n = col_base + ct * 16;
        if (n < g.N) P[(size_t)m * g.N + n] = acc[r][ct][i];
      }
    }
}

// FFN up-projection epilogue: sum the S partial products of each element in split
// order, add the bias, apply GELU and store the result as the next product's A operand.
// One thread per 4 consecutive columns; the loads of eight splits are issued before
// their sums.
__global__ void __launch_bounds__(256) gelu_reduce_kernel(GemmArgs g) {
  const int n4 = g.N / 4;
  const size_t total4 = (size_t)g.M * n4, plane = (size_t)g.M * g.N;
  for (size_t q = (size_t)blockIdx.x * 256 + threadIdx.x; q < total4; q += (size_t)gridDim.x * 256) {
    const int m = (int)(q / n4), n = (int)(q % n4) * 4;
    const size_t e = (size_t)m * g.N + n;
    float4 acc = *(const float4*)(g.part + e);
    for (int t0 = 1; t0 < g.S; t0 += 8) {
      float4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = *(const float4*)(g.part + (size_t)min(t0 + u, g.S - 1) * plane + e);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (t0 + u < g.S) { acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w; }
    }
    const uint2 bu = *(const uint2*)(g.bias + n);
    float y[4] = {gelu_erf(acc.x + bf16_to_f32(bu.x & 0xffff)), gelu_erf(acc.y + bf16_to_f32(bu.x >> 16)),
                  gelu_erf(acc.z + bf16_to_f32(bu.y & 0xffff)), gelu_erf(acc.w + bf16_to_f32(bu.y >> 16))};
    uint16_t h[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) split_hilo(y[i], h[i], l[i]);
    *(uint2*)(g.e.frag + afrag_index(m, n, 0, g.e.frag_RT)) =
        uint2{h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16)};
    *(uint2*)(g.e.frag + afrag_index(m, n, 1, g.e.frag_RT)) =
        uint2{l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16)};
  }
}

// Row-wise merge of the per-tile top-2 records of the LM head: greedy token (lowest
// index among equal maxima) and the top-1 minus top-2 margin.
__global__ void __launch_bounds__(64) argmax_final_kernel(int M, int ntiles, const float4* part,
                                                          const RowDesc* rows, int* greedy,
                                                          float* margin, int* err) {
  const int m = blockIdx.x, lane = threadIdx.x;
  Top2s t{-INFINITY, 0x7fffffff, -INFINITY, 0};
  for (int j = lane; j < ntiles; j += 64) {
    const float4 p = part[(size_t)m * ntiles + j];
    t = t2_merge(t, Top2s{p.x, __float_as_int(p.y), p.z, __float_as_int(p.w)});
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) t = t2_merge(t, t2_shfl(t, o));
  if (lane == 0) {
    const bool valid_row = rows ? rows[m].seq >= 0 : true;
    if (t.bad && valid_row && err) atomicOr(err, 16);
    greedy[m] = (t.bad && valid_row) ? -1 : t.i1;
    if (margin) margin[m] = t.v1 - t.v2;
  }
}

// Row tiles per workgroup for an M-row product (the activation buffer holds a multiple
// of 16 row tiles, so every staged block lies inside it).
int gemm_rtc(int M) {
  const int rt = (M + 15) / 16;
  return rt <= 4 ? 4 : (rt <= 8 ? 8 : 16);
}

int gemm_splits(int N, int K) {
  const int ntiles = (N + kNT - 1) / kNT, KB = K / 32;
  int s = 240 / ntiles;
  s = min(s, KB);
  s = min(s, max(1, K / 256));
  return max(1, s);
}

static int gemm_mchunks(int M) {
  const int rtc = gemm_rtc(M);
  return ((M + 15) / 16 + rtc - 1) / rtc;
}

size_t gemm_part_floats(int M, int N, int K) { return (size_t)gemm_splits(N, K) * M * N; }

int lm_tiles(int V) { return (V + kNT - 1) / kNT; }

template <int EPI>
static void launch_one(GemmArgs g, hipStream_t st) {
  const int rtc = gemm_rtc(g.M);
  g.mchunks = gemm_mchunks(g.M);
  const dim3 grid(g.ntiles * g.S * g.mchunks), block(256);
  if (rtc == 4) hipLaunchKernelGGL((gemm_mfma_kernel<EPI, 4>), grid, block, 0, st, g);
  else if (rtc == 8) hipLaunchKernelGGL((gemm_mfma_kernel<EPI, 8>), grid, block, 0, st, g);
  else hipLaunchKernelGGL((gemm_mfma_kernel<EPI, 16>), grid, block, 0, st, g);
}

int gemm_launch_splits(int epi, int N, int K) { return epi == EPI_ARGMAX ? 1 : gemm_splits(N, K); }

void launch_gemm_mfma(int epi, GemmArgs g, hipStream_t st) {
  g.ntiles = (g.N + kNT - 1) / kNT;
  g.KB = g.K / 32;
  g.S = gemm_launch_splits(epi, g.N, g.K);
  if (epi == EPI_ARGMAX) launch_one<EPI_ARGMAX>(g, st);
  else launch_one<EPI_PARTIAL>(g, st);
}

void launch_gelu_reduce(GemmArgs g, hipStream_t st) {
  g.S = gemm_splits(g.N, g.K);
  const size_t total4 = (size_t)g.M * g.N / 4;
  const dim3 grid((unsigned)std::min<size_t>((total4 + 255) / 256, 4096)), block(256);
  hipLaunchKernelGGL(gelu_reduce_kernel, grid, block, 0, st, g);
}

void launch_argmax_final(int M, int ntiles, const void* part, const RowDesc* rows, int* greedy,
                         float* margin, int* err, hipStream_t st) {
  hipLaunchKernelGGL(argmax_final_kernel, dim3(M), dim3(64), 0, st, M, ntiles, (const float4*)part,
                     rows, greedy, margin, err);
}

}  // namespace ad
