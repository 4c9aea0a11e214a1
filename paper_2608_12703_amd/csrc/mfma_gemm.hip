// Projections and the LM head of the bf16 model on the gfx950 matrix cores.
//
// C[m][n] = sum_k X[m][k] W[n][k] with W bf16 [N][K] and X float32 activations stored as
// a hi/lo bf16 pair in A-fragment order.  A workgroup owns 128 output columns and up to
// RTC 16-row tiles; its eight waves (two per SIMD, so one wave's LDS reads overlap the
// other's matrix instructions) each own a quarter of the rows and half of the columns
// (with 8 row tiles: one row tile and all the columns each).
// Weights (streamed from HBM) move in 32-wide K steps through an LDS ring filled by
// direct global->LDS loads three to five steps ahead.  Activations (L2-resident) go
// straight into a register ring as far ahead for tiles of up to 8 row tiles (the
// A-fragment order is the matrix instruction's lane order, so each is one coalesced
// 16-byte load per lane; keeping them out of LDS removes a third of the step's LDS
// traffic), and through a three-stage LDS ring for 16 row tiles.  Workgroups with long K ranges (the FFN
// products) take two K steps per barrier.  The waits are explicit; the loops are unrolled
// over the ring stages so every buffer is a distinct object.  Small-N products split K
// over several workgroups, each storing its raw partial tile; the kernel that consumes
// the product (attention, or residual + LayerNorm) sums the partials in split order.
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

// Running top-2 of a set of logits: largest value v1 at index i1 (lowest index among
// equal maxima), the runner-up value v2 (equal to v1 when the maximum repeats), and
// whether a non-finite value was seen.  The merge is associative and commutative, so any
// reduction order gives the same record.  Branch-free (selects only).
struct Top2s {
  float v1;
  int i1;
  float v2;
  int bad;
};
__device__ __forceinline__ Top2s t2_merge(Top2s a, Top2s b) {
  const bool aw = (a.v1 > b.v1) | ((a.v1 == b.v1) & (a.i1 < b.i1));
  Top2s r;
  r.v1 = aw ? a.v1 : b.v1;
  r.i1 = aw ? a.i1 : b.i1;
  r.v2 = fmaxf(aw ? a.v2 : b.v2, aw ? b.v1 : a.v1);
  r.bad = a.bad | b.bad;
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
// Rotate by N lanes inside each row of 16 lanes (DPP row_ror, no LDS round trip).
template <int N>
__device__ __forceinline__ int ror16(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x120 + N, 0xf, 0xf, false);
}
template <int N>
__device__ __forceinline__ Top2s t2_ror16(Top2s t) {
  Top2s u;
  u.v1 = __int_as_float(ror16<N>(__float_as_int(t.v1)));
  u.i1 = ror16<N>(t.i1);
  u.v2 = __int_as_float(ror16<N>(__float_as_int(t.v2)));
  u.bad = ror16<N>(t.bad);
  return u;
}
// Merge over the 16 lanes of a row: afterwards every lane holds the row's record.
__device__ __forceinline__ Top2s t2_row16(Top2s t) {
  t = t2_merge(t, t2_ror16<8>(t));
  t = t2_merge(t, t2_ror16<4>(t));
  t = t2_merge(t, t2_ror16<2>(t));
  t = t2_merge(t, t2_ror16<1>(t));
  return t;
}

// Wait until at most N vector-memory operations of this wave are outstanding (they
// complete in order) and its LDS operations are done, then barrier.  No memory fence.
// The gfx9 s_waitcnt immediate holds vmcnt in two fields: bits 3:0 and bits 15:14
// (expcnt 7 in bits 6:4 means no wait on exports; lgkmcnt 0 in bits 11:8).
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0070; }
#define BARRIER_VMCNT(N)                                     \
  do {                                                       \
    static_assert((N) >= 0 && (N) < 64, "vmcnt is 6 bits");  \
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(N));               \
    __builtin_amdgcn_s_barrier();                            \
    asm volatile("" ::: "memory");                           \
  } while (0)

// Product order of one accumulator tile: SW computes the transposed tile (weights as the
// first operand), so a lane holds four consecutive columns of one row instead of four
// rows of one column; each element's sum is the same.
template <bool SW>
__device__ __forceinline__ f32x4 mma_tile(bf16x8 a, bf16x8 w, f32x4 c) {
  return SW ? mfma_bf16(w, a, c) : mfma_bf16(a, w, c);
}

// One 32-wide K step of a wave: RW row tiles (row group rg) x 4 column tiles (half ch).
template <int RTC, bool SW>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[RTC / 4][4], const uint4* abuf,
                                         const uint4* wbuf, int rg, int ch, int lane) {
  constexpr int RW = RTC / 4;
  bf16x8 b[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) b[ct] = as_bf16x8(wbuf[(ch * 4 + ct) * 64 + lane]);
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int rt = rg * RW + r;
    const bf16x8 ah = as_bf16x8(abuf[(rt * 2 + 0) * 64 + lane]);
    const bf16x8 al = as_bf16x8(abuf[(rt * 2 + 1) * 64 + lane]);
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      acc[r][ct] = mma_tile<SW>(ah, b[ct], acc[r][ct]);
      acc[r][ct] = mma_tile<SW>(al, b[ct], acc[r][ct]);
    }
  }
}

// The activation operand of one K step for the RW row tiles of one wave, in registers.
template <int RW>
struct AFrag {
  uint4 h[RW], l[RW];
};

// One 32-wide K step with the activations from registers: RW row tiles x CT column
// tiles (column group ch).
template <int RW, int CT, bool SW>
__device__ __forceinline__ void mma_step_reg(f32x4 (&acc)[RW][CT], const AFrag<RW>& a,
                                             const uint4* wbuf, int ch, int lane) {
  bf16x8 b[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) b[ct] = as_bf16x8(wbuf[(ch * CT + ct) * 64 + lane]);
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const bf16x8 ah = as_bf16x8(a.h[r]), al = as_bf16x8(a.l[r]);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      acc[r][ct] = mma_tile<SW>(ah, b[ct], acc[r][ct]);
      acc[r][ct] = mma_tile<SW>(al, b[ct], acc[r][ct]);
    }
  }
}

// WIDE (8 row tiles only): each wave owns one row tile and all 128 columns, so every
// activation fragment is loaded once per workgroup (the default layout loads each one
// twice, once per column half) and a K step does twice the matrix work for the same
// operand bytes.  The order of every output's sums is the same in both layouts.
template <int EPI, int RTC, bool PACKED, bool TWO = false, bool WIDE = false>
__global__ void __launch_bounds__(512) gemm_mfma_kernel(GemmArgs g) {
  static_assert(!WIDE || (RTC == 8 && EPI != EPI_ARGMAX), "the wide layout: 8 row tiles, no argmax");
  constexpr int RW = WIDE ? 1 : RTC / 4;  // row tiles per wave
  constexpr int CT = WIDE ? 8 : 4;        // 16-column tiles per wave
  constexpr int NA = RTC / 4;            // direct loads per wave for one activation stage
  // the up-projection keeps transposed tiles (four consecutive columns of a row per lane:
  // 8-byte hi / lo stores).  (Measured slower for the split-K partials: 16-byte
  // non-temporal stores of 16 rows per instruction against 4-byte stores of 4 rows.)
  constexpr bool kSw = EPI == EPI_GELU;
  // Activation ring: 3 stages (requested 2 steps ahead); weight ring: 6 stages (requested
  // 5 steps ahead, covering HBM latency).  Distinct LDS objects, so the compiler can tell
  // a read of one stage from the direct loads still filling another.  (Measured slower:
  // a 12-stage weight ring, and 6-stage rings for both operands; larger LDS footprints
  // cost more than the deeper prefetch gains.)
  __shared__ uint4 sa0[RTC * 128], sa1[RTC * 128], sa2[RTC * 128];
  __shared__ uint4 sw0[512], sw1[512], sw2[512], sw3[512], sw4[512], sw5[512];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int rg = WIDE ? w : (w & 3), ch = WIDE ? 0 : (w >> 2);   // row group, column group
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

  f32x4 acc[RW][CT];
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = kb1 - kb0, kl = kb1 - 1;
  auto ia = [&](uint4* buf, int kb) {   // activation stage of step kb (clamped)
    const uint4* src = (const uint4*)g.A + ((size_t)min(kb, kl) * g.RT + rt0) * 128;
#pragma unroll
    for (int ii = 0; ii < NA; ++ii) {
      const int i = ii * 8 + w;
      dma16(src + i * 64 + lane, buf + i * 64);
    }
  };
  auto iw = [&](uint4* buf, int kb) {   // weight stage of step kb (clamped)
    const int k = min(kb, kl);
    if constexpr (PACKED) {              // one contiguous 8 KB stage
      dma16(g.W + ((size_t)(nt * g.KB + k) * 512 + w * 64 + lane) * 8, buf + w * 64);
    } else {
      const int n = min(n0 + w * 16 + (lane & 15), g.N - 1);   // column tile w
      dma16(g.W + (size_t)n * g.K + k * 32 + (lane >> 4) * 8, buf + w * 64);
    }
  };
  int kb = kb0;
  if constexpr (RTC <= 8) {
    // Activations straight into registers (the A-fragment layout is the matrix
    // instruction's lane order, so each is one coalesced 16-byte load per lane), as far
    // ahead as the weights: only the weights pass through LDS, which halves the LDS
    // traffic of a step.  A step requests A then W; the barrier's wait counts whole
    // (A, W) pairs, so it also completes the activations of the next step and the
    // compiler needs no wait of its own for the registers.
    constexpr int kA = 2 * RW;                       // activation loads per step
    const uint4* abase = (const uint4*)g.A + ((size_t)rt0 + rg * RW) * 128 + lane;
    auto la = [&](AFrag<RW>& f, int k) {
      const uint4* src = abase + (size_t)min(k, kl) * g.RT * 128;
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        f.h[r] = src[(r * 2 + 0) * 64];
        f.l[r] = src[(r * 2 + 1) * 64];
      }
    };
    AFrag<RW> a0, a1, a2, a3, a4, a5;
    if constexpr (TWO) {
      // Long K ranges (TWO) take two K steps per barrier: iteration i (steps 2i, 2i + 1)
      // requests A and W of steps 2i + 4 and 2i + 5, multiplies, and ends with the
      // previous iteration's loads complete.  (Short ranges keep one step per barrier:
      // the first wait then covers one stage instead of two.)
      constexpr int kWait2 = 2 * (kA + 1);
      la(a0, kb0);
      iw(sw0, kb0);
      la(a1, kb0 + 1);
      iw(sw1, kb0 + 1);
      la(a2, kb0 + 2);
      iw(sw2, kb0 + 2);
      la(a3, kb0 + 3);
      iw(sw3, kb0 + 3);
      BARRIER_VMCNT(kWait2);
#define GEMM_ITER(CA0, CW0, CA1, CW1, NA0, NW0, NA1, NW1)         \
    {                                                             \
      la(NA0, kb + 4);                                            \
      iw(NW0, kb + 4);                                            \
      la(NA1, kb + 5);                                            \
      iw(NW1, kb + 5);                                            \
      mma_step_reg<RW, CT, kSw>(acc, CA0, CW0, ch, lane);                 \
      if (kb + 1 < kb1) mma_step_reg<RW, CT, kSw>(acc, CA1, CW1, ch, lane);\
      BARRIER_VMCNT(kWait2);                                      \
      kb += 2;                                                    \
    }
      const int iters = (nk + 1) >> 1;
      for (int it = 0; it < iters / 3; ++it) {
        GEMM_ITER(a0, sw0, a1, sw1, a4, sw4, a5, sw5)
        GEMM_ITER(a2, sw2, a3, sw3, a0, sw0, a1, sw1)
        GEMM_ITER(a4, sw4, a5, sw5, a2, sw2, a3, sw3)
      }
      const int rem = iters % 3;
      if (rem >= 1) GEMM_ITER(a0, sw0, a1, sw1, a4, sw4, a5, sw5)
      if (rem >= 2) GEMM_ITER(a2, sw2, a3, sw3, a0, sw0, a1, sw1)
#undef GEMM_ITER
    } else {
      // One step per barrier, operands three steps ahead (four ring slots): step j
      // requests A(j+3) then W(j+3) into the slots step j - 1 read and ends with step
      // j + 1 complete (two steps' loads still in flight).  (Five steps ahead measured
      // 0.16 us slower per launch in the verify step, two steps ahead slower still.)
      constexpr int kWait1 = 2 * (kA + 1);
      la(a0, kb0);
      iw(sw0, kb0);
      la(a1, kb0 + 1);
      iw(sw1, kb0 + 1);
      la(a2, kb0 + 2);
      iw(sw2, kb0 + 2);
      BARRIER_VMCNT(kWait1);
#define GEMM_STEP(CA, CW, NXA, NXW)                      \
    {                                                    \
      la(NXA, kb + 3);                                   \
      iw(NXW, kb + 3);                                   \
      mma_step_reg<RW, CT, kSw>(acc, CA, CW, ch, lane);  \
      BARRIER_VMCNT(kWait1);                             \
      ++kb;                                              \
    }
      for (int it = 0; it < nk / 4; ++it) {
        GEMM_STEP(a0, sw0, a3, sw3)
        GEMM_STEP(a1, sw1, a0, sw0)
        GEMM_STEP(a2, sw2, a1, sw1)
        GEMM_STEP(a3, sw3, a2, sw2)
      }
      const int rem = nk % 4;
      if (rem >= 1) GEMM_STEP(a0, sw0, a3, sw3)
      if (rem >= 2) GEMM_STEP(a1, sw1, a0, sw0)
      if (rem >= 3) GEMM_STEP(a2, sw2, a1, sw1)
#undef GEMM_STEP
    }
  } else {
    // Step j requests activations j + 2 and weights j + 5, in that order; the prologue
    // plays virtual steps -5 .. -1 so the outstanding-load count is the same everywhere:
    // at the end of step j the loads issued after A(j+1) are W(j+4), A(j+2), W(j+5).
    constexpr int kWait = NA + 2;
    iw(sw0, kb0);
    iw(sw1, kb0 + 1);
    iw(sw2, kb0 + 2);
    ia(sa0, kb0);
    iw(sw3, kb0 + 3);
    ia(sa1, kb0 + 1);
    iw(sw4, kb0 + 4);
    BARRIER_VMCNT(kWait);
#define GEMM_STEP(CA, CW, NXA, NXW)            \
  {                                            \
    ia(NXA, kb + 2);                           \
    iw(NXW, kb + 5);                           \
    mma_step<RTC, kSw>(acc, CA, CW, rg, ch, lane);  \
    BARRIER_VMCNT(kWait);                      \
    ++kb;                                      \
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
  }
  BARRIER_VMCNT(0);

  // row / column of accumulator element (r, ct, i) of this lane: row_base + r * 16 + i,
  // col_base + ct * 16; with transposed tiles row_base + r * 16, col_base + ct * 16 + i
  const int row_base = (rt0 + rg * RW) * 16 + (kSw ? c16 : grp * 4);
  const int col_base = n0 + ch * CT * 16 + (kSw ? grp * 4 : c16);

  // This kernel's LDS is also written by direct loads, so the compiler orders every LDS
  // access after outstanding global stores; epilogues therefore finish all their
  // cross-lane (LDS) work before the first store.
  if (EPI == EPI_ARGMAX) {
    // LM head: top-2 of this wave's 64 columns per row (one record per half tile).  A
    // row's columns sit in 16 lanes x 4 registers; the merge keeps the lowest index
    // among equal maxima whatever the order.
    Top2s t[RW][4];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        t[r][i] = Top2s{-INFINITY, 0x7fffffff, -INFINITY, 0};
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const int n = col_base + ct * 16;
          const float v = acc[r][ct][i];
          const bool fin = isfinite(v), in = n < g.N;
          // columns past V are neutral; a non-finite logit flags the row
          const Top2s u{(in & fin) ? v : -INFINITY, in ? n : 0x7fffffff, -INFINITY,
                        (in & !fin) ? 1 : 0};
          t[r][i] = t2_merge(t[r][i], u);
        }
        t[r][i] = t2_row16(t[r][i]);
      }
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = row_base + r * 16 + i;
        if (c16 == 0 && m < g.M) {
          float4 rec{t[r][i].v1, __int_as_float(t[r][i].i1), t[r][i].v2, __int_as_float(t[r][i].bad)};
          ((float4*)g.e.am_part)[(size_t)m * (2 * g.ntiles) + nt * 2 + ch] = rec;
        }
      }
    if (g.e.out) {
#pragma unroll
      for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = row_base + r * 16 + i, n = col_base + ct * 16;
            if (m < g.M && n < g.N) g.e.out[(size_t)m * g.e.ldo + n] = acc[r][ct][i];
          }
    }
    return;
  }

  if (EPI == EPI_GELU) {
    // FFN up-projection (unsplit): bias + GELU, stored straight from registers as the
    // next product's A operand (hi/lo bf16 pair in A-fragment order; four consecutive
    // columns of a row are one 8-byte store each for hi and lo)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const int n = col_base + ct * 16;
      float bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) bv[i] = bf16_to_f32(g.bias[min(n + i, g.N - 1)]);
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        const int m = row_base + r * 16;
        if (m >= g.M) continue;
        const float4 y{gelu_erf(acc[r][ct][0] + bv[0]), gelu_erf(acc[r][ct][1] + bv[1]),
                       gelu_erf(acc[r][ct][2] + bv[2]), gelu_erf(acc[r][ct][3] + bv[3])};
        if (n + 3 < g.N) {
          afrag_store4(g.e.frag, g.e.frag_RT, m, n, y);
        } else {
          const float yv[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n + i < g.N) afrag_store(g.e.frag, g.e.frag_RT, m, n + i, yv[i]);
        }
      }
    }
    return;
  }

  // EPI_PARTIAL: the raw split-K partial product straight from registers (16 lanes store
  // 64 contiguous bytes of a row, non-temporal: only the consumer kernel reads them); the
  // consumer kernel sums the splits in split order.
  float* P = g.part + (size_t)s * g.M * g.N;
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = row_base + r * 16 + i;
      if (m >= g.M) continue;
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const int n = col_base + ct * 16;
        if (n < g.N) __builtin_nontemporal_store(acc[r][ct][i], &P[(size_t)m * g.N + n]);
      }
    }
}

// LM head (argmax epilogue, unsplit) with 16 row tiles and 256 columns per workgroup:
// at the verify block's 224 rows the 406 column tiles of the vocabulary then fit one
// round of 203 workgroups (128 columns per workgroup take two rounds).  Eight waves, each
// with 4 row tiles x 8 column tiles; both operands through three-stage LDS rings filled
// by direct loads two steps ahead (144 KB).  Every output's sums run in the same order
// as in gemm_mfma_kernel, and the per-64-column top-2 records land in the same slots.
template <bool PACKED>
__global__ void __launch_bounds__(512) lm_head_kernel(GemmArgs g) {
  constexpr int RTC = 16, RW = 4, CT = 8, NA = RTC / 4;
  __shared__ uint4 sa0[RTC * 128], sa1[RTC * 128], sa2[RTC * 128];
  __shared__ uint4 sw0[2 * 512], sw1[2 * 512], sw2[2 * 512];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int rg = w & 3, ch = w >> 2;   // row group (4 row tiles), 128-column half
  const int c16 = lane & 15, grp = lane >> 4;

  // (column group of 256, row chunk), numbered so each XCD holds a contiguous id range
  const int nwg = gridDim.x, bid = blockIdx.x;
  const int x = bid & 7, q8 = nwg >> 3, r8 = nwg & 7;
  const int lin = x * q8 + min(x, r8) + (bid >> 3);
  const int mc = lin % g.mchunks, nt = lin / g.mchunks;
  const int rt0 = mc * RTC, n0 = nt * 2 * kNT;

  f32x4 acc[RW][CT];
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int kl = g.KB - 1;
  auto ia = [&](uint4* buf, int kb) {   // activation stage of step kb (clamped)
    const uint4* src = (const uint4*)g.A + ((size_t)min(kb, kl) * g.RT + rt0) * 128;
#pragma unroll
    for (int ii = 0; ii < NA; ++ii) {
      const int i = ii * 8 + w;
      dma16(src + i * 64 + lane, buf + i * 64);
    }
  };
  auto iw = [&](uint4* buf, int kb) {   // weight stage of step kb (clamped): two column tiles
    const int k = min(kb, kl);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (PACKED) {
        const int t = min(nt * 2 + h, g.ntiles - 1);
        dma16(g.W + ((size_t)(t * g.KB + k) * 512 + w * 64 + lane) * 8, buf + h * 512 + w * 64);
      } else {
        const int n = min(n0 + h * kNT + w * 16 + (lane & 15), g.N - 1);
        dma16(g.W + (size_t)n * g.K + k * 32 + (lane >> 4) * 8, buf + h * 512 + w * 64);
      }
    }
  };
  auto mma = [&](const uint4* abuf, const uint4* wbuf) __attribute__((always_inline)) {
    bf16x8 b[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) b[ct] = as_bf16x8(wbuf[ch * 512 + ct * 64 + lane]);
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const int rt = rg * RW + r;
      const bf16x8 ah = as_bf16x8(abuf[(rt * 2 + 0) * 64 + lane]);
      const bf16x8 al = as_bf16x8(abuf[(rt * 2 + 1) * 64 + lane]);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        acc[r][ct] = mfma_bf16(ah, b[ct], acc[r][ct]);
        acc[r][ct] = mfma_bf16(al, b[ct], acc[r][ct]);
      }
    }
  };
  // Step j requests A(j + 2) then W(j + 2) into the stages step j - 1 read; at the end of
  // step j the loads issued after W(j + 1) are A(j + 2) and W(j + 2).
  constexpr int kWait = NA + 2;
  ia(sa0, 0);
  iw(sw0, 0);
  ia(sa1, 1);
  iw(sw1, 1);
  BARRIER_VMCNT(kWait);
  int kb = 0;
#define LM_STEP(CA, CW, NXA, NXW) \
  {                               \
    ia(NXA, kb + 2);              \
    iw(NXW, kb + 2);              \
    mma(CA, CW);                  \
    BARRIER_VMCNT(kWait);         \
    ++kb;                         \
  }
  for (int it = 0; it < g.KB / 3; ++it) {
    LM_STEP(sa0, sw0, sa2, sw2)
    LM_STEP(sa1, sw1, sa0, sw0)
    LM_STEP(sa2, sw2, sa1, sw1)
  }
  const int rem = g.KB % 3;
  if (rem >= 1) LM_STEP(sa0, sw0, sa2, sw2)
  if (rem >= 2) LM_STEP(sa1, sw1, sa0, sw0)
#undef LM_STEP
  BARRIER_VMCNT(0);

  // top-2 of each 64-column half of this wave's 128 columns per row, stored in the slot
  // of that 64-column block (the slots gemm_mfma_kernel uses)
  const int row_base = (rt0 + rg * RW) * 16 + grp * 4;   // + r * 16 + i
  const int col_base = n0 + ch * kNT + c16;              // + ct * 16
#pragma unroll
  for (int r = 0; r < RW; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = row_base + r * 16 + i;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        Top2s t{-INFINITY, 0x7fffffff, -INFINITY, 0};
#pragma unroll
        for (int ct = 4 * q; ct < 4 * q + 4; ++ct) {
          const int n = col_base + ct * 16;
          const float v = acc[r][ct][i];
          const bool fin = isfinite(v), in = n < g.N;
          const Top2s u{(in & fin) ? v : -INFINITY, in ? n : 0x7fffffff, -INFINITY,
                        (in & !fin) ? 1 : 0};
          t = t2_merge(t, u);
        }
        t = t2_row16(t);
        const int slot = nt * 4 + ch * 2 + q;
        if (c16 == 0 && m < g.M && slot < 2 * g.ntiles) {
          float4 rec{t.v1, __int_as_float(t.i1), t.v2, __int_as_float(t.bad)};
          ((float4*)g.e.am_part)[(size_t)m * (2 * g.ntiles) + slot] = rec;
        }
      }
    }
  if (g.e.out) {
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = row_base + r * 16 + i, n = col_base + ct * 16;
          if (m < g.M && n < g.N) g.e.out[(size_t)m * g.e.ldo + n] = acc[r][ct][i];
        }
  }
}

// Tiled weight copy (see launch.h): one thread per 16-byte piece.
__global__ void __launch_bounds__(256) pack_weight_kernel(const uint16_t* W, int N, int K,
                                                          uint16_t* P, size_t pieces) {
  const int KB = K / 32;
  for (size_t q = (size_t)blockIdx.x * 256 + threadIdx.x; q < pieces; q += (size_t)gridDim.x * 256) {
    const size_t stage = q / 512;
    const int t = (int)(q % 512), ct = t / 64, lane = t % 64;
    const int nt = (int)(stage / KB), kb = (int)(stage % KB);
    const int n = nt * kNT + ct * 16 + (lane & 15), k = kb * 32 + (lane >> 4) * 8;
    const uint4 v = n < N ? *(const uint4*)(W + (size_t)n * K + k) : make_uint4(0, 0, 0, 0);
    *(uint4*)(P + q * 8) = v;
  }
}

// Row-wise merge of the per-tile top-2 records of the LM head: greedy token (lowest
// index among equal maxima) and the top-1 minus top-2 margin.
__global__ void __launch_bounds__(64) argmax_final_kernel(int M, int nrec, const float4* part,
                                                          const RowDesc* rows, int* greedy,
                                                          float* margin, int* err) {
  const int m = blockIdx.x, lane = threadIdx.x;
  Top2s t{-INFINITY, 0x7fffffff, -INFINITY, 0};
  for (int j = lane; j < nrec; j += 64) {
    const float4 p = part[(size_t)m * nrec + j];
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

// Launch planning.  A workgroup's time is dominated by fixed costs (first-load latency,
// the partial stores) plus its K steps, and a second round of workgroups costs a whole
// extra pass, so plans keep the grid within one workgroup per CU.  Per-step times for
// 4 / 8 / 16 row tiles: about 0.27 / 0.43 / 0.8 us.  (The wide 8-row-tile layout runs a
// step in about 0.38 us alone; priced that way, the 1280 x 5120 down-projection would
// take 12 splits instead of 6, which is faster alone (9.7 against 13.3 us) but slower
// inside the verify step (4.978 against 4.952 ms), where the consumer sums twice the
// partials.)
constexpr int kMaxWGs = 256;
constexpr int kRefRows = 224;   // reference block for the split choice (32 sequences x 7 rows)

static double step_us(int rtc) { return rtc == 4 ? 0.27 : (rtc == 8 ? 0.43 : 0.8); }
static int mchunks_of(int M, int rtc) { return ((M + 15) / 16 + rtc - 1) / rtc; }

// Split count of an N x K weight.  It depends on the weight shape only (never on the
// number of rows), so every row's sums run in the same order whatever the batch.
int gemm_splits(int N, int K) {
  const int ntiles = (N + kNT - 1) / kNT, KB = K / 32;
  double best = 1e30;
  int best_s = 1;
  for (int S = 1; S <= std::min(KB, 64); ++S)
    for (int rtc : {4, 8, 16}) {
      if (ntiles * mchunks_of(kRefRows, rtc) * S > kMaxWGs && S > 1) continue;
      const double partial_us = (double)S * kRefRows * N * 4 / 4e6;   // ~4 TB/s
      const double c = ((KB + S - 1) / S) * step_us(rtc) + partial_us;
      if (c < best - 1e-9) { best = c; best_s = S; }
    }
  return best_s;
}

// Row tiles per workgroup: the smallest tile whose grid stays within one workgroup per
// CU (the activation buffer holds a multiple of 16 row tiles, so every staged block lies
// in it).  With the wide 8-row-tile layout (twice the matrix work per K step for the
// same operand bytes) one round of 8-row-tile workgroups beats 4-row-tile ones sharing
// CUs: the 352-row block of an 11-node tree at batch 32 takes 5.31 ms per step against
// 5.86 ms with up to 1.5 four-row-tile workgroups per CU, the ragged 64-sequence batch
// 6.29 (packed) / 7.22 (padded) against 6.52 / 7.41 ms, the verify step unchanged.  The
// row tiling never changes a row's sums (same K order, same split order).
// When no tile fits (the LM head's 406 column tiles), 16 row tiles, or 4 when that
// needs no more row chunks (up to 64 rows, the draft block's 32): a 4-row-tile K step
// costs a third of a 16-row-tile one (draft step 198 -> 156 us at batch 32).
constexpr int kMaxWGsRows = 256;
int gemm_rtc(int M, int N, int S) {
  const int ntiles = (N + kNT - 1) / kNT;
  for (int rtc : {4, 8})
    if (ntiles * mchunks_of(M, rtc) * S <= kMaxWGsRows) return rtc;
  return mchunks_of(M, 4) == mchunks_of(M, 16) ? 4 : 16;
}

size_t gemm_part_floats(int M, int N, int K) { return (size_t)gemm_splits(N, K) * M * N; }

size_t packed_weight_elems(int N, int K) { return (size_t)((N + kNT - 1) / kNT) * kNT * K; }

void launch_pack_weight(const uint16_t* W, int N, int K, uint16_t* P, hipStream_t st) {
  const size_t pieces = packed_weight_elems(N, K) / 8;
  const dim3 grid((unsigned)std::min<size_t>((pieces + 255) / 256, 8192)), block(256);
  hipLaunchKernelGGL(pack_weight_kernel, grid, block, 0, st, W, N, K, P, pieces);
}

int lm_records(int V) { return 2 * ((V + kNT - 1) / kNT); }

// Workgroups with at least this many K steps take two steps per barrier (FFN up and
// down at d 1280: 40 and 26-27 steps; the down-projection measured 1.7 us faster alone
// and 0.2-0.5 us faster inside the verify step, while the 8-step d x d products are
// faster with one step per barrier).  The loop choice never changes the order of a
// tile's sums.
constexpr int kTwoStepMin = 24;

// Eight row tiles always take the wide wave layout, except for the LM head's argmax
// epilogue, which merges per column half.  Alone, the wide loop measured as fast or faster
// on every projection shape (the 1280 x 5120 down-projection at 224 rows, 12 splits: 9.7
// against 14.0 us); the 64-sequence ragged batch padded to 576 rows, whose projections
// take 8 row tiles, runs its verify step in 7.77 ms against 8.26 ms.
template <int EPI, int RTC, bool PACKED>
static void launch_rtc(const GemmArgs& g, dim3 grid, hipStream_t st) {
  constexpr bool kWide = RTC == 8 && EPI != EPI_ARGMAX;
  if (RTC <= 8 && g.KB / g.S >= kTwoStepMin)
    hipLaunchKernelGGL((gemm_mfma_kernel<EPI, RTC, PACKED, RTC <= 8, kWide>), grid, dim3(512), 0, st, g);
  else
    hipLaunchKernelGGL((gemm_mfma_kernel<EPI, RTC, PACKED, false, kWide>), grid, dim3(512), 0, st, g);
}

template <int EPI>
static void launch_one(GemmArgs g, hipStream_t st) {
  const int rtc = gemm_rtc(g.M, g.N, g.S);
  g.mchunks = mchunks_of(g.M, rtc);
  if (EPI == EPI_ARGMAX && rtc == 16 && g.ntiles * g.mchunks > kMaxWGs &&
      (g.ntiles + 1) / 2 * g.mchunks <= kMaxWGs) {
    const dim3 grid((g.ntiles + 1) / 2 * g.mchunks);
    if (g.packed) hipLaunchKernelGGL(lm_head_kernel<true>, grid, dim3(512), 0, st, g);
    else hipLaunchKernelGGL(lm_head_kernel<false>, grid, dim3(512), 0, st, g);
    return;
  }
  const dim3 grid(g.ntiles * g.S * g.mchunks);
  if (g.packed) {
    if (rtc == 4) launch_rtc<EPI, 4, true>(g, grid, st);
    else if (rtc == 8) launch_rtc<EPI, 8, true>(g, grid, st);
    else launch_rtc<EPI, 16, true>(g, grid, st);
  } else {
    if (rtc == 4) launch_rtc<EPI, 4, false>(g, grid, st);
    else if (rtc == 8) launch_rtc<EPI, 8, false>(g, grid, st);
    else launch_rtc<EPI, 16, false>(g, grid, st);
  }
}

// The fused epilogues (argmax, GELU) need the whole K sum in one workgroup.
int gemm_launch_splits(int epi, int N, int K) {
  return (epi == EPI_ARGMAX || epi == EPI_GELU) ? 1 : gemm_splits(N, K);
}

void launch_gemm_mfma(int epi, GemmArgs g, hipStream_t st) {
  g.ntiles = (g.N + kNT - 1) / kNT;
  g.KB = g.K / 32;
  g.S = gemm_launch_splits(epi, g.N, g.K);
  if (epi == EPI_ARGMAX) launch_one<EPI_ARGMAX>(g, st);
  else if (epi == EPI_GELU) launch_one<EPI_GELU>(g, st);
  else launch_one<EPI_PARTIAL>(g, st);
}


void launch_argmax_final(int M, int nrec, const void* part, const RowDesc* rows, int* greedy,
                         float* margin, int* err, hipStream_t st) {
  hipLaunchKernelGGL(argmax_final_kernel, dim3(M), dim3(64), 0, st, M, nrec, (const float4*)part,
                     rows, greedy, margin, err);
}

}  // namespace ad
