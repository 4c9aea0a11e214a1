// Vector-ALU matrix products and attention: the float32 model's path, and the
// reference-shaped path every optimised kernel must agree with.
//
// Every output element is reduced in a fixed order that does not depend on how many
// rows share the launch, so a row's result is the same alone or inside any batch.
#include "common.h"
#include "launch.h"

namespace ad {

// ---------------------------------------------------------------- GEMM
// C[m][n] = sum_k A[m][k] W[n][k] (+ bias[n]); 32 x 64 output tile per 256 threads, K in
// steps of 32 (K a multiple of 32).  Each output is one thread's fma chain over k in
// order.  A step's operands pass through LDS; every thread requests its slice of the
// operands kVStages steps ahead into registers, so a workgroup's K loop waits for memory
// once rather than once per step (with few rows, as in batch-1 decoding, the loop is
// otherwise a chain of dependent round trips).

constexpr int kVStages = 8;

// Workgroup barrier for LDS traffic only: this wave's LDS operations complete, its global
// loads stay in flight (__syncthreads would also wait for every outstanding load, which
// empties the prefetch rings below at every step).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt 0; vmcnt and expcnt not waited for
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One thread's slice of a K step: 4 activations of row ar; 8 weights (4 of rows wr and
// wr + 32 in float32, or 8 of row wb in bf16).
template <class S>
struct VStage;
template <>
struct VStage<F32> {
  float4 a, w0, w1;
};
template <>
struct VStage<BF16> {
  float4 a;
  uint4 w;
};

// Every load is issued unconditionally (rows and columns past the matrix read its last
// row or column, steps past K its last step), so the number of loads in flight is the
// same on every path and the compiler's waits count exactly; the values outside the
// matrix become zeros when the step is staged in LDS.
template <class S>
__device__ __forceinline__ void vstage_load(VStage<S>& st, int kb, int M, int N, int K, const float* A,
                                            const typename S::T* W, int m0, int n0, int tid) {
  const int k0 = min(kb * 32, K - 32);
  const int ar = tid >> 3, ak = (tid & 7) * 4;
  st.a = *(const float4*)(A + (size_t)min(m0 + ar, M - 1) * K + k0 + ak);
  if constexpr (sizeof(typename S::T) == 4) {
    const int wr = tid >> 3, wk = (tid & 7) * 4;
    st.w0 = *(const float4*)(W + (size_t)min(n0 + wr, N - 1) * K + k0 + wk);
    st.w1 = *(const float4*)(W + (size_t)min(n0 + wr + 32, N - 1) * K + k0 + wk);
  } else {
    const int wb = tid >> 2, wk = (tid & 3) * 8;
    st.w = *(const uint4*)(W + (size_t)min(n0 + wb, N - 1) * K + k0 + wk);
  }
}

// LDS layout of a step: activations transposed, At[k][row] (a row's 8 values of one k
// are one broadcast read pair), weights Ws[col][k]; rows of 36 floats keep every
// 16-byte read aligned and the weight reads of 16 lanes on distinct banks.
constexpr int kVLd = 36;

template <class S>
__device__ __forceinline__ void vstage_put(const VStage<S>& st, int M, int N, int m0, int n0,
                                           float (*At)[kVLd], float (*Ws)[kVLd], int tid) {
  const int ar = tid >> 3, ak = (tid & 7) * 4;
  const bool am = m0 + ar < M;
  At[ak + 0][ar] = am ? st.a.x : 0.f;
  At[ak + 1][ar] = am ? st.a.y : 0.f;
  At[ak + 2][ar] = am ? st.a.z : 0.f;
  At[ak + 3][ar] = am ? st.a.w : 0.f;
  if constexpr (sizeof(typename S::T) == 4) {
    const int wr = tid >> 3, wk = (tid & 7) * 4;
    const bool w0 = n0 + wr < N, w1 = n0 + wr + 32 < N;
    *(float4*)&Ws[wr][wk] = w0 ? st.w0 : float4{0.f, 0.f, 0.f, 0.f};
    *(float4*)&Ws[wr + 32][wk] = w1 ? st.w1 : float4{0.f, 0.f, 0.f, 0.f};
  } else {
    const int wb = tid >> 2, wk = (tid & 3) * 8;
    const bool wn = n0 + wb < N;
    const uint32_t u[4] = {st.w.x, st.w.y, st.w.z, st.w.w};
    float f[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f[2 * j] = wn ? bf16_to_f32(u[j] & 0xffff) : 0.f;
      f[2 * j + 1] = wn ? bf16_to_f32(u[j] >> 16) : 0.f;
    }
    *(float4*)&Ws[wb][wk] = float4{f[0], f[1], f[2], f[3]};
    *(float4*)&Ws[wb][wk + 4] = float4{f[4], f[5], f[6], f[7]};
  }
}

template <class S, class SA, int EPI>
__global__ void __launch_bounds__(256) gemm_valu_kernel(int M, int N, int K, const typename SA::T* A,
                                                        const typename S::T* W,
                                                        const typename S::T* bias, EpiArgs e) {
  static_assert(sizeof(typename SA::T) == 4, "float32 activations");
  __shared__ __align__(16) float At[32][kVLd];
  __shared__ __align__(16) float Ws[64][kVLd];
  const int tid = threadIdx.x, tx = tid & 63, ty = tid >> 6;
  const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 64;
  const int KB = K / 32;
  float acc[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) acc[r] = 0.f;
  VStage<S> s0, s1, s2, s3, s4, s5, s6, s7;
  vstage_load<S>(s0, 0, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s1, 1, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s2, 2, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s3, 3, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s4, 4, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s5, 5, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s6, 6, M, N, K, A, W, m0, n0, tid);
  vstage_load<S>(s7, 7, M, N, K, A, W, m0, n0, tid);
  // step kb: stage its operands in LDS, multiply, request step kb + kVStages into the
  // freed registers
#define VGEMM_STEP(ST, J)                                                 \
  {                                                                       \
    if (kb + (J) < KB) {                                                  \
      lds_barrier();                                                      \
      vstage_put<S>(ST, M, N, m0, n0, At, Ws, tid);                       \
      lds_barrier();                                                      \
      _Pragma("unroll") for (int k4 = 0; k4 < 32; k4 += 4) {              \
        const float4 w = *(const float4*)&Ws[tx][k4];                     \
        const float wv[4] = {w.x, w.y, w.z, w.w};                         \
        _Pragma("unroll") for (int u = 0; u < 4; ++u) {                   \
          const float4 a0 = *(const float4*)&At[k4 + u][ty * 8];          \
          const float4 a1 = *(const float4*)&At[k4 + u][ty * 8 + 4];      \
          const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w}; \
          _Pragma("unroll") for (int r = 0; r < 8; ++r) acc[r] = fmaf(av[r], wv[u], acc[r]); \
        }                                                                 \
      }                                                                   \
    }                                                                     \
    vstage_load<S>(ST, kb + (J) + kVStages, M, N, K, A, W, m0, n0, tid);  \
  }
  for (int kb = 0; kb < KB; kb += kVStages) {
    VGEMM_STEP(s0, 0)
    VGEMM_STEP(s1, 1)
    VGEMM_STEP(s2, 2)
    VGEMM_STEP(s3, 3)
    VGEMM_STEP(s4, 4)
    VGEMM_STEP(s5, 5)
    VGEMM_STEP(s6, 6)
    VGEMM_STEP(s7, 7)
  }
#undef VGEMM_STEP
  const int n = n0 + tx;
  if (n >= N) return;
  const float bn = bias ? S::ld(bias, n) : 0.f;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int m = m0 + ty * 8 + r;
    if (m >= M) continue;
    const float v = acc[r] + bn;
    if (EPI == EPI_STORE) {
      e.out[(size_t)m * e.ldo + n] = v;
    } else if (EPI == EPI_RESID) {
      e.out[(size_t)m * e.ldo + n] += v;
    } else if (EPI == EPI_GELU) {
      e.out[(size_t)m * e.ldo + n] = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
    } else if (EPI == EPI_QKV) {
      if (n < e.d) {
        e.out[(size_t)m * e.ldo + n] = v;
      } else {
        const RowDesc rd = e.rows[m];
        if (rd.seq >= 0) {
          const int c = n - e.d, kv = c / e.d, h = (c % e.d) / kHead, j = c % kHead;
          int pg = e.block_table[(size_t)rd.seq * e.pages_per_seq + rd.slot / kTile];
          pg = min(max(pg, 0), e.num_pages - 1);
          S::st((typename S::T*)e.cache,
                kv_tile_base(e.layer, kv, pg, h, e.num_pages, e.H) + tile_off(kv, rd.slot % kTile, j), v);
        }
      }
    } else if (EPI == EPI_XKV) {
      const int kv = n / e.d, h = (n % e.d) / kHead, j = n % kHead;
      S::st((typename S::T*)e.cache, cross_base(e.layer, h, e.H, e.frames_cap) + cross_off(kv, m, j), v);
    }
  }
}

template <class S, class SA>
static void gemm_valu_dispatch(int epi, int M, int N, int K, const void* A, const void* W,
                               const void* bias, const EpiArgs& e, hipStream_t st) {
  const dim3 grid((N + 63) / 64, (M + 31) / 32), block(256);
  const auto* a = (const typename SA::T*)A;
  const auto* w = (const typename S::T*)W;
  const auto* b = (const typename S::T*)bias;
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_valu_kernel<S, SA, EPI_STORE>), grid, block, 0, st, M, N, K, a, w, b, e); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_valu_kernel<S, SA, EPI_RESID>), grid, block, 0, st, M, N, K, a, w, b, e); break;
    case EPI_GELU: hipLaunchKernelGGL((gemm_valu_kernel<S, SA, EPI_GELU>), grid, block, 0, st, M, N, K, a, w, b, e); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm_valu_kernel<S, SA, EPI_QKV>), grid, block, 0, st, M, N, K, a, w, b, e); break;
    case EPI_XKV: hipLaunchKernelGGL((gemm_valu_kernel<S, SA, EPI_XKV>), grid, block, 0, st, M, N, K, a, w, b, e); break;
  }
}

template <class S>
void launch_gemm_valu(int epi, int M, int N, int K, const float* A, const void* W, const void* bias,
                      const EpiArgs& e, hipStream_t st) {
  gemm_valu_dispatch<S, F32>(epi, M, N, K, A, W, bias, e, st);
}
template void launch_gemm_valu<F32>(int, int, int, int, const float*, const void*, const void*, const EpiArgs&, hipStream_t);
template void launch_gemm_valu<BF16>(int, int, int, int, const float*, const void*, const void*, const EpiArgs&, hipStream_t);

// ---------------------------------------------------------------- attention
// One block per (head, sequence, group of kVGroupKeys keys at absolute positions 0, 128,
// 256, ...).  Queries are taken 16 at a time; a group's keys stream through LDS in
// chunks of 64 with an online softmax per query, which leaves a partial (max, sum,
// unnormalised output) per (row, head, group); a second kernel merges the groups in
// group order.  A key a query may not see contributes exp(-inf) = 0; keys past every query's
// range are staged as zeros so stale cache slots never reach the output.  Every thread
// requests its part of a chunk (two runs of 8 keys' lanes and two runs of 8 values of
// one lane, contiguous in both cache layouts) kAStages chunks ahead into registers.

constexpr int kAStages = 4;
constexpr int kVGroupKeys = 128;   // keys per workgroup
constexpr int kVPart = 2 + kHead;  // a partial: max, sum, 64 output lanes

template <class S>
struct AStage;
template <>
struct AStage<F32> {
  float4 k[2][2], v[2][2];
};
template <>
struct AStage<BF16> {
  uint4 k[2], v[2];
};

// Load chunk c0 (keys c0 .. c0 + 63): piece u of this thread is key run (key tid / 8 +
// 32 u, lanes 8 (tid % 8) ..) and value run (lane tid / 8 + 32 u, keys c0 + 8 (tid % 8) ..).
// Keys at or past n_keys read the last key's place (the values become zeros in LDS).
template <class S, bool CROSS>
__device__ __forceinline__ void astage_load(AStage<S>& st, int c0, int n_keys, int layer, int h, int H,
                                            int b, const SeqDesc& s, const typename S::T* kv,
                                            int num_pages, const int* block_table, int pages_per_seq,
                                            int frames_cap, int tid) {
  constexpr bool F = sizeof(typename S::T) == 4;
  const int last = max(n_keys - 1, 0);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int tk = c0 + (tid >> 3) + 32 * u, jk = (tid & 7) * 8;   // key run
    const int jv = (tid >> 3) + 32 * u, tv = c0 + (tid & 7) * 8;   // value run
    size_t bk = 0, bv = 0;
    if (CROSS) {
      bk = cross_base(layer, h, H, frames_cap) + cross_off(0, s.enc_off + min(tk, last), jk);
      bv = cross_base(layer, h, H, frames_cap) + cross_off(1, s.enc_off + min(tv, last) / 8 * 8, jv);
    } else {
      const int pk = min(max(block_table[(size_t)b * pages_per_seq + min(tk, last) / kTile], 0), num_pages - 1);
      const int pv = min(max(block_table[(size_t)b * pages_per_seq + min(tv, last) / kTile], 0), num_pages - 1);
      bk = kv_tile_base(layer, 0, pk, h, num_pages, H) + tile_off(0, min(tk, last) % kTile, jk);
      bv = kv_tile_base(layer, 1, pv, h, num_pages, H) + tile_off(1, min(tv, last) / 8 * 8 % kTile, jv);
    }
    if constexpr (F) {
      st.k[u][0] = *(const float4*)(kv + bk);
      st.k[u][1] = *(const float4*)(kv + bk + 4);
      st.v[u][0] = *(const float4*)(kv + bv);
      st.v[u][1] = *(const float4*)(kv + bv + 4);
    } else {
      st.k[u] = *(const uint4*)(kv + bk);
      st.v[u] = *(const uint4*)(kv + bv);
    }
  }
}

// Chunk c0's registers into LDS: ks[key][lane], vs[key][lane]; key and value slots at
// or past n_keys are zeroed.
template <class S>
__device__ __forceinline__ void astage_put(const AStage<S>& st, int c0, int n_keys, float (*ks)[65],
                                           float (*vs)[65], int tid) {
  constexpr bool F = sizeof(typename S::T) == 4;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int rk = (tid >> 3) + 32 * u, jk = (tid & 7) * 8;
    const int jv = (tid >> 3) + 32 * u, rv = (tid & 7) * 8;
    float kx[8], vx[8];
    if constexpr (F) {
      const float4 a = st.k[u][0], bq = st.k[u][1], c = st.v[u][0], dq = st.v[u][1];
      kx[0] = a.x; kx[1] = a.y; kx[2] = a.z; kx[3] = a.w; kx[4] = bq.x; kx[5] = bq.y; kx[6] = bq.z; kx[7] = bq.w;
      vx[0] = c.x; vx[1] = c.y; vx[2] = c.z; vx[3] = c.w; vx[4] = dq.x; vx[5] = dq.y; vx[6] = dq.z; vx[7] = dq.w;
    } else {
      const uint32_t ku[4] = {st.k[u].x, st.k[u].y, st.k[u].z, st.k[u].w};
      const uint32_t vu[4] = {st.v[u].x, st.v[u].y, st.v[u].z, st.v[u].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        kx[2 * j] = bf16_to_f32(ku[j] & 0xffff);
        kx[2 * j + 1] = bf16_to_f32(ku[j] >> 16);
        vx[2 * j] = bf16_to_f32(vu[j] & 0xffff);
        vx[2 * j + 1] = bf16_to_f32(vu[j] >> 16);
      }
    }
    const bool kin = c0 + rk < n_keys;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ks[rk][jk + e] = kin ? kx[e] : 0.f;
      vs[rv + e][jv] = (c0 + rv + e < n_keys) ? vx[e] : 0.f;
    }
  }
}

template <class S, bool CROSS>
__global__ void __launch_bounds__(256) attn_valu_kernel(int H, int d, int layer,
                                                        const SeqDesc* seqs, const float* q,
                                                        float* apart, int G, const typename S::T* kv,
                                                        int num_pages, const int* block_table,
                                                        int pages_per_seq, int frames_cap,
                                                        const RowTree* tree) {
  __shared__ float qs[16][65];
  __shared__ float ks[64][65];
  __shared__ float vs[64][65];
  __shared__ float ps[16][65];
  const int h = blockIdx.x, b = blockIdx.y, g = blockIdx.z, tid = threadIdx.x;
  const SeqDesc s = seqs[b];
  if (!s.valid) return;
  const int qi = tid >> 4, part = tid & 15;
  const int n_rows = s.k + 1;
  for (int qg = 0; qg < n_rows; qg += 16) {
    const int nq = min(16, n_rows - qg);
    lds_barrier();
    for (int i = tid; i < 16 * 64; i += 256) {
      const int r = i >> 6, j = i & 63;
      qs[r][j] = r < nq ? q[(size_t)(s.row0 + qg + r) * d + h * kHead + j] : 0.f;
    }
    // cross-attention sees frames [wlo, whi) (all frames unless a window was given);
    // self-attention every committed key and the block rows in the query's row mask
    const int lo = CROSS ? s.wlo : 0;
    const unsigned long long tm = (!CROSS && qi < nq) ? tree[s.row0 + qg + qi].mask : 0ull;
    const int n_keys = CROSS ? s.whi : s.n + qg + nq;
    float m_run = -INFINITY, l_run = 0.f, o[4] = {0.f, 0.f, 0.f, 0.f};
    // this group's chunks: keys [max(lo, 128 g), min(128 (g + 1), n_keys)), 64-aligned
    const int c_first = max(lo / 64 * 64, g * kVGroupKeys);
    const int c_end = min((g + 1) * kVGroupKeys, n_keys);
    const int nch = c_end > c_first ? (c_end - c_first + 63) / 64 : 0;
    AStage<S> st0, st1, st2, st3;
    // (chunks past the last one reread it; nch >= 1 whenever the loop runs)
    auto load = [&](AStage<S>& st, int ci) {
      astage_load<S, CROSS>(st, c_first + min(ci, max(nch - 1, 0)) * 64, n_keys, layer, h, H, b, s, kv,
                            num_pages, block_table, pages_per_seq, frames_cap, tid);
    };
    load(st0, 0);
    load(st1, 1);
    load(st2, 2);
    load(st3, 3);
    // the scores, the online-softmax update and the value product of chunk c0 (in LDS)
    auto attend = [&](int c0) __attribute__((always_inline)) {
      float sc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int key = part + 16 * u;
        float acc = 0.f;
#pragma unroll 16
        for (int j = 0; j < 64; ++j) acc = fmaf(qs[qi][j], ks[key][j], acc);
        const int t = c0 + key;
        const bool see = CROSS ? (t >= lo && t < n_keys)
                               : (t < s.n || (t < n_keys && ((tm >> (t - s.n)) & 1)));
        sc[u] = (see && qi < nq) ? acc * 0.125f : -INFINITY;
      }
      float cm = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, kWave));
      const float m_new = fmaxf(m_run, cm);
      const float scale = (m_new == -INFINITY) ? 1.f : expf(m_run - m_new);
      float ls = 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float p = (sc[u] == -INFINITY) ? 0.f : expf(sc[u] - m_new);
        ps[qi][part + 16 * u] = p;
        ls += p;
      }
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) ls += __shfl_xor(ls, off, kWave);
      l_run = l_run * scale + ls;
      m_run = m_new;
      lds_barrier();
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] *= scale;
      for (int key = 0; key < 64; ++key) {
        const float p = ps[qi][key];
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = fmaf(p, vs[key][part * 4 + r], o[r]);
      }
    };
    // chunk ci of the ring slot ST: stage it in LDS, request chunk ci + kAStages into the
    // freed registers, attend
#define VATT_CHUNK(ST, J)                                  \
  {                                                        \
    if (ci + (J) < nch) {                                  \
      const int c0 = c_first + (ci + (J)) * 64;            \
      lds_barrier();                                       \
      astage_put<S>(ST, c0, n_keys, ks, vs, tid);          \
      lds_barrier();                                       \
      attend(c0);                                          \
    }                                                      \
    load(ST, ci + (J) + kAStages);                         \
  }
    for (int ci = 0; ci < nch; ci += kAStages) {
      VATT_CHUNK(st0, 0)
      VATT_CHUNK(st1, 1)
      VATT_CHUNK(st2, 2)
      VATT_CHUNK(st3, 3)
    }
#undef VATT_CHUNK
    // the group's partial: (max, sum, unnormalised output); a group without keys leaves
    // (-inf, 0, 0)
    if (qi < nq) {
      float* pp = apart + (((size_t)(s.row0 + qg + qi) * H + h) * G + g) * kVPart;
      if (part == 0) {   // one of the row's 16 threads writes the statistics
        pp[0] = m_run;
        pp[1] = l_run;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) pp[2 + part * 4 + r] = o[r];
    }
  }
}

// Merge the G key groups of every (row, head) in group order: out = sum_g e^(m_g - M)
// o_g / sum_g e^(m_g - M) l_g with M = max_g m_g.  Rows of no sequence, or of a sequence
// the step skips, are left alone (as the attention kernel leaves them).
__global__ void __launch_bounds__(64) attn_merge_kernel(int H, int d, int G, const SeqDesc* seqs,
                                                        const RowDesc* rows, const float* part, float* out) {
  const int m = blockIdx.x, h = blockIdx.y, j = threadIdx.x;
  const int sq = rows[m].seq;
  if (sq < 0 || !seqs[sq].valid) return;
  const float* pp = part + ((size_t)m * H + h) * G * kVPart;
  float M = -INFINITY;
  for (int g = 0; g < G; ++g) M = fmaxf(M, pp[g * kVPart]);
  float L = 0.f, acc = 0.f;
  for (int g = 0; g < G; ++g) {
    const float mg = pp[g * kVPart];
    const float w = mg == -INFINITY ? 0.f : expf(mg - M);
    L += w * pp[g * kVPart + 1];
    acc += w * pp[g * kVPart + 2 + j];
  }
  out[(size_t)m * d + h * kHead + j] = acc / L;
}

int attn_valu_groups(int max_keys) { return (max_keys + kVGroupKeys - 1) / kVGroupKeys; }

template <class S>
void launch_self_attn_valu(int B, int M, int H, int d, int layer, const SeqDesc* seqs, const RowDesc* rows,
                           const float* q, float* part, int G, float* out, const void* pool, int num_pages,
                           const int* block_table, int pages_per_seq, const RowTree* tree, hipStream_t st) {
  hipLaunchKernelGGL((attn_valu_kernel<S, false>), dim3(H, B, G), dim3(256), 0, st, H, d, layer, seqs, q, part,
                     G, (const typename S::T*)pool, num_pages, block_table, pages_per_seq, 0, tree);
  hipLaunchKernelGGL(attn_merge_kernel, dim3(M, H), dim3(64), 0, st, H, d, G, seqs, rows, part, out);
}
template <class S>
void launch_cross_attn_valu(int B, int M, int H, int d, int layer, const SeqDesc* seqs, const RowDesc* rows,
                            const float* q, float* part, int G, float* out, const void* cross, int frames_cap,
                            hipStream_t st) {
  hipLaunchKernelGGL((attn_valu_kernel<S, true>), dim3(H, B, G), dim3(256), 0, st, H, d, layer, seqs, q, part,
                     G, (const typename S::T*)cross, 0, nullptr, 0, frames_cap, nullptr);
  hipLaunchKernelGGL(attn_merge_kernel, dim3(M, H), dim3(64), 0, st, H, d, G, seqs, rows, part, out);
}
template void launch_self_attn_valu<F32>(int, int, int, int, int, const SeqDesc*, const RowDesc*, const float*, float*, int, float*, const void*, int, const int*, int, const RowTree*, hipStream_t);
template void launch_self_attn_valu<BF16>(int, int, int, int, int, const SeqDesc*, const RowDesc*, const float*, float*, int, float*, const void*, int, const int*, int, const RowTree*, hipStream_t);
template void launch_cross_attn_valu<F32>(int, int, int, int, int, const SeqDesc*, const RowDesc*, const float*, float*, int, float*, const void*, int, hipStream_t);
template void launch_cross_attn_valu<BF16>(int, int, int, int, int, const SeqDesc*, const RowDesc*, const float*, float*, int, float*, const void*, int, hipStream_t);

}  // namespace ad
