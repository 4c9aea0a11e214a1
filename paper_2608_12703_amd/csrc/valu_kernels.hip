// Vector-ALU matrix products and attention: the float32 model's path, and the
// reference-shaped path every optimised kernel must agree with.
//
// Every output element is reduced in a fixed order that does not depend on how many
// rows share the launch, so a row's result is the same alone or inside any batch.
#include "common.h"
#include "launch.h"

namespace ad {

// ---------------------------------------------------------------- GEMM
// C[m][n] = sum_k A[m][k] W[n][k] (+ bias[n]); 32 x 64 output tile per 256 threads.

template <class S, class SA, int EPI>
__global__ void __launch_bounds__(256) gemm_valu_kernel(int M, int N, int K, const typename SA::T* A,
                                                        const typename S::T* W,
                                                        const typename S::T* bias, EpiArgs e) {
  __shared__ float As[32][33];
  __shared__ float Ws[64][33];
  const int tid = threadIdx.x, tx = tid & 63, ty = tid >> 6;
  const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 64;
  float acc[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) acc[r] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 32) {
    for (int i = tid; i < 32 * 32; i += 256) {
      const int r = i >> 5, c = i & 31, m = m0 + r, k = k0 + c;
      As[r][c] = (m < M && k < K) ? SA::ld(A, (size_t)m * K + k) : 0.f;
    }
    for (int i = tid; i < 64 * 32; i += 256) {
      const int r = i >> 5, c = i & 31, n = n0 + r, k = k0 + c;
      Ws[r][c] = (n < N && k < K) ? S::ld(W, (size_t)n * K + k) : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const float w = Ws[tx][kk];
#pragma unroll
      for (int r = 0; r < 8; ++r) acc[r] = fmaf(As[ty * 8 + r][kk], w, acc[r]);
    }
    __syncthreads();
  }
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
// One block per (head, sequence).  Queries are taken 16 at a time; keys stream through
// LDS in chunks of 64 at absolute positions 0, 64, 128, ... with an online softmax per
// query.  A key a query may not see contributes exp(-inf) = 0; keys past every query's
// range are staged as zeros so stale cache slots never reach the output.

template <class S, bool CROSS>
__global__ void __launch_bounds__(256) attn_valu_kernel(int H, int d, int layer,
                                                        const SeqDesc* seqs, const float* q,
                                                        float* out, const typename S::T* kv,
                                                        int num_pages, const int* block_table,
                                                        int pages_per_seq, int frames_cap,
                                                        const RowTree* tree) {
  __shared__ float qs[16][65];
  __shared__ float ks[64][65];
  __shared__ float vs[64][65];
  __shared__ float ps[16][65];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const SeqDesc s = seqs[b];
  if (!s.valid) return;
  const int qi = tid >> 4, part = tid & 15;
  const int n_rows = s.k + 1;
  for (int qg = 0; qg < n_rows; qg += 16) {
    const int nq = min(16, n_rows - qg);
    __syncthreads();
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
    for (int c0 = lo / 64 * 64; c0 < n_keys; c0 += 64) {
      __syncthreads();
      for (int i = tid; i < 64 * 64; i += 256) {
        const int key = i >> 6, j = i & 63, t = c0 + key;
        float kk = 0.f, vv = 0.f;
        if (t < n_keys) {
          size_t bk, bv;
          if (CROSS) {
            bk = cross_base(layer, h, H, frames_cap) + cross_off(0, s.enc_off + t, j);
            bv = cross_base(layer, h, H, frames_cap) + cross_off(1, s.enc_off + t, j);
          } else {
            int pg = block_table[(size_t)b * pages_per_seq + t / kTile];
            pg = min(max(pg, 0), num_pages - 1);
            bk = kv_tile_base(layer, 0, pg, h, num_pages, H) + tile_off(0, t % kTile, j);
            bv = kv_tile_base(layer, 1, pg, h, num_pages, H) + tile_off(1, t % kTile, j);
          }
          kk = S::ld(kv, bk);
          vv = S::ld(kv, bv);
        }
        ks[key][j] = kk;
        vs[key][j] = vv;
      }
      __syncthreads();
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
      __syncthreads();
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] *= scale;
      for (int key = 0; key < 64; ++key) {
        const float p = ps[qi][key];
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = fmaf(p, vs[key][part * 4 + r], o[r]);
      }
    }
    if (qi < nq) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        out[(size_t)(s.row0 + qg + qi) * d + h * kHead + part * 4 + r] = o[r] / l_run;
    }
  }
}

template <class S>
void launch_self_attn_valu(int B, int H, int d, int layer, const SeqDesc* seqs, const float* q,
                           float* out, const void* pool, int num_pages, const int* block_table,
                           int pages_per_seq, const RowTree* tree, hipStream_t st) {
  hipLaunchKernelGGL((attn_valu_kernel<S, false>), dim3(H, B), dim3(256), 0, st, H, d, layer, seqs, q, out,
                     (const typename S::T*)pool, num_pages, block_table, pages_per_seq, 0, tree);
}
template <class S>
void launch_cross_attn_valu(int B, int H, int d, int layer, const SeqDesc* seqs, const float* q,
                            float* out, const void* cross, int frames_cap, hipStream_t st) {
  hipLaunchKernelGGL((attn_valu_kernel<S, true>), dim3(H, B), dim3(256), 0, st, H, d, layer, seqs, q, out,
                     (const typename S::T*)cross, 0, nullptr, 0, frames_cap, nullptr);
}
template void launch_self_attn_valu<F32>(int, int, int, int, const SeqDesc*, const float*, float*, const void*, int, const int*, int, const RowTree*, hipStream_t);
template void launch_self_attn_valu<BF16>(int, int, int, int, const SeqDesc*, const float*, float*, const void*, int, const int*, int, const RowTree*, hipStream_t);
template void launch_cross_attn_valu<F32>(int, int, int, int, const SeqDesc*, const float*, float*, const void*, int, hipStream_t);
template void launch_cross_attn_valu<BF16>(int, int, int, int, const SeqDesc*, const float*, float*, const void*, int, hipStream_t);

}  // namespace ad
