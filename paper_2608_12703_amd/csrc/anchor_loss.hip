// The AnchorDraft training objective on the matrix cores (bf16 draft models).
//
// Paper, section "Correction and Cost", paragraph "AnchorDraft Training Objective", and
// appendix "Training Correction with AnchorDraft" (eq. anchordraft-supp):
//   Abar_t(j) = mean over heads of the first draft layer's cross-attention A_{t,hj}
//   q_t(j)    = Gaussian around the aligned frame c_t, normalised over the valid frames
//   L         = L_tok + 0.5 L_feat - lambda / |V| sum_t sum_j q_t(j) log Abar_t(j)
// Rows are padded per sequence: row t of sequence b is b * R + t.  The attention is
// recomputed from the layer's query rows and the cross-key cache (never stored):
//   stats   per (head, sequence, 16-row tile): softmax max / sum over all valid frames
//   abar    per (128-frame chunk, sequence, tile): every head's probabilities summed
//           into Abar (kept in workspace), the row's cross-entropy partial per chunk
//   dq      per (head, sequence, tile), optional: the gradient for the query rows,
//           d l_t / d x_{t,h} = (1/8) (X - c Y) with X = sum_j A_j g_j k_j,
//           Y = sum_j A_j k_j, c = sum_j A_j g_j, g_j = -q_t(j) / (H Abar_t(j))
// Scores use the transposed product of the attention kernels, S^T = K Q^T (keys on the
// MFMA rows, 16 query rows on the columns, queries as hi/lo bf16 pairs), so every lane
// holds 8 consecutive keys of one row; X^T and Y^T = K^T P^T take those 8 keys as their
// B operand directly and the keys, transposed through a per-wave LDS tile, as A.
// The token and feature terms are row kernels over the logits / features.
#include "common.h"
#include "launch.h"

namespace ad {

namespace {

constexpr int kLossThreads = 256;
constexpr int kLossChunk = 4 * kCrossBlock;   // frames per workgroup of the Abar kernel
constexpr int kKtStride = 68;                 // halfwords per key row of the LDS key tile

struct KTile {
  uint4 k00, k01, k10, k11;
};

// the sequence's frames, validated exactly as the prep kernel does
__device__ __forceinline__ bool seq_frames(const LossArgs& a, int b, int& T, int& off) {
  T = a.enc_len[b];
  off = a.enc_off[b];
  return T >= 1 && T <= a.max_frames && off >= 0 && off % kCrossBlock == 0 && off + T <= a.frames_cap;
}

// Q^T operand of query row `row`, head h: dims 16 grp .. 16 grp + 15 scaled by 1/8 (exact),
// as hi / lo bf16 pairs
__device__ __forceinline__ void load_q(const LossArgs& a, int row, int h, int grp, bf16x8 (&qh)[2],
                                       bf16x8 (&ql)[2]) {
  const float* p = a.xq + (size_t)row * a.d + h * kHead + grp * 16;
  float v[16];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float4 f = *(const float4*)(p + 4 * u);
    v[4 * u] = f.x * 0.125f;
    v[4 * u + 1] = f.y * 0.125f;
    v[4 * u + 2] = f.z * 0.125f;
    v[4 * u + 3] = f.w * 0.125f;
  }
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float x0 = v[8 * half + 2 * j], x1 = v[8 * half + 2 * j + 1];
      hw[j] = f32x2_to_bf16x2(x0, x1);
      lw[j] = f32x2_to_bf16x2(x0 - bf16_to_f32(hw[j] & 0xffff), x1 - bf16_to_f32(hw[j] >> 16));
    }
    qh[half] = as_bf16x8(make_uint4(hw[0], hw[1], hw[2], hw[3]));
    ql[half] = as_bf16x8(make_uint4(lw[0], lw[1], lw[2], lw[3]));
  }
}

// keys of 32-frame block blk of the sequence (head h), score-operand order
__device__ __forceinline__ void load_k(const LossArgs& a, int h, int off, int blk, int c16, int grp,
                                       KTile& t) {
  const uint16_t* kp = a.kv + cross_base(a.layer, h, a.H, a.frames_cap) +
                       (size_t)(off / kCrossBlock + blk) * 2 * kCrossBlockElems + (grp * 16 + c16) * 8;
  t.k00 = *(const uint4*)(kp + 0 * 512);
  t.k01 = *(const uint4*)(kp + 1 * 512);
  t.k10 = *(const uint4*)(kp + 2 * 512);
  t.k11 = *(const uint4*)(kp + 3 * 512);
}

// scores of keys blk*32 + 8 grp + 0..7 for this lane's row (-inf past T)
__device__ __forceinline__ void scores8(const KTile& t, const bf16x8 (&qh)[2], const bf16x8 (&ql)[2],
                                        int key0, int T, float (&sv)[8]) {
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 k0 = as_bf16x8(tt ? t.k10 : t.k00), k1 = as_bf16x8(tt ? t.k11 : t.k01);
    st = mfma_bf16(k0, qh[0], st);
    st = mfma_bf16(k1, qh[1], st);
    st = mfma_bf16(k0, ql[0], st);
    st = mfma_bf16(k1, ql[1], st);
#pragma unroll
    for (int i = 0; i < 4; ++i) sv[tt * 4 + i] = key0 + tt * 4 + i < T ? st[i] : -INFINITY;
  }
}

// q_t(j) for an aligned row (centre c, normaliser z)
__device__ __forceinline__ float gauss(int j, int c, float inv2s2, float z) {
  const float e = (float)(j - c);
  return expf(-e * e * inv2s2) / z;
}

__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    h[j] = f32x2_to_bf16x2(v[2 * j], v[2 * j + 1]);
    l[j] = f32x2_to_bf16x2(v[2 * j] - bf16_to_f32(h[j] & 0xffff), v[2 * j + 1] - bf16_to_f32(h[j] >> 16));
  }
  hi = as_bf16x8(make_uint4(h[0], h[1], h[2], h[3]));
  lo = as_bf16x8(make_uint4(l[0], l[1], l[2], l[3]));
}

}  // namespace

// Per row: validation, the Gaussian normaliser over the sequence's valid frames, the row
// flags (bit 0 aligned, bit 1 has a next token) and the counts |V|, |T|.  One wave per row.
__global__ void __launch_bounds__(kLossThreads) aloss_prep_kernel(LossArgs a) {
  const int row = blockIdx.x * (kLossThreads / kWave) + threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (row >= a.M) return;
  const int b = row / a.R;
  // (the alignment term only: frames and centres are read when query rows are given)
  int T = 0, off = 0;
  const bool seq_ok = a.xq && seq_frames(a, b, T, off);
  int err = (a.xq && !seq_ok) ? 8 : 0;
  const int c = a.xq ? a.center[row] : -1;
  if (c < -1 || (seq_ok && c >= T)) err |= 8;
  const bool av = seq_ok && c >= 0 && c < T;
  const int y = a.targets ? a.targets[row] : -1;
  if (y < -1 || y >= a.V) err |= 4;
  const bool tv = y >= 0 && y < a.V;
  float z = 0.f;
  if (av) {
    const float inv = 1.f / (2.f * a.sigma * a.sigma);
    for (int j = lane; j < T; j += kWave) {
      const float e = (float)(j - c);
      z += expf(-e * e * inv);
    }
    z = wave_sum(z);
  }
  if (lane == 0) {
    a.Z[row] = z;
    a.rowflag[row] = (av ? 1 : 0) | (tv ? 2 : 0);
    if (av) atomicAdd(&a.counts[0], 1);
    if (tv) atomicAdd(&a.counts[1], 1);
    if (err) atomicOr(a.err, err);
  }
}

// Softmax statistics (max, sum of exp(score - max)) of every (row, head) over all valid
// frames.  Four waves take interleaved 32-frame blocks; their partials merge in order.
__global__ void __launch_bounds__(kLossThreads) aloss_stats_kernel(LossArgs a) {
  __shared__ float2 part[4][kWave];
  const int h = blockIdx.x, b = blockIdx.y, tile = blockIdx.z;
  int T, off;
  if (!seq_frames(a, b, T, off)) return;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave, c16 = lane & 15, grp = lane >> 4;
  const int r = tile * 16 + c16;
  const int row = b * a.R + min(r, a.R - 1);
  bf16x8 qh[2], ql[2];
  load_q(a, row, h, grp, qh, ql);
  const int nblk = (T + kCrossBlock - 1) / kCrossBlock;
  float m = -INFINITY, l = 0.f;
  for (int blk = w; blk < nblk; blk += 4) {
    KTile t;
    load_k(a, h, off, blk, c16, grp, t);
    float sv[8];
    scores8(t, qh, ql, blk * kCrossBlock + grp * 8, T, sv);
    float bm = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) bm = fmaxf(bm, sv[i]);
    if (bm == -INFINITY) continue;
    const float mn = fmaxf(m, bm);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += sv[i] == -INFINITY ? 0.f : __expf(sv[i] - mn);
    l = (m == -INFINITY ? 0.f : l * __expf(m - mn)) + s;
    m = mn;
  }
  part[w][lane] = float2{m, l};
  __syncthreads();
  if (threadIdx.x < 16) {
    const int rr = tile * 16 + threadIdx.x;
    float M = -INFINITY;
    for (int ww = 0; ww < 4; ++ww)
      for (int g = 0; g < 4; ++g) M = fmaxf(M, part[ww][g * 16 + threadIdx.x].x);
    float L = 0.f;
    for (int ww = 0; ww < 4; ++ww)
      for (int g = 0; g < 4; ++g) {
        const float2 p = part[ww][g * 16 + threadIdx.x];
        if (p.x != -INFINITY) L += p.y * __expf(p.x - M);
      }
    if (rr < a.R) a.stats[(size_t)(b * a.R + rr) * a.H + h] = float2{M, L};
  }
}

// Head-averaged attention over one 128-frame chunk (one 32-frame block per wave, every
// head in turn), stored in workspace, and each row's cross-entropy partial over the chunk.
__global__ void __launch_bounds__(kLossThreads) aloss_abar_kernel(LossArgs a) {
  __shared__ float part[4][16];
  const int chunk = blockIdx.x, b = blockIdx.y, tile = blockIdx.z;
  int T, off;
  if (!seq_frames(a, b, T, off) || chunk * kLossChunk >= T) return;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave, c16 = lane & 15, grp = lane >> 4;
  const int r = tile * 16 + c16;
  const int row = b * a.R + min(r, a.R - 1);
  const int nblk = (T + kCrossBlock - 1) / kCrossBlock;
  const int blk = chunk * 4 + w;
  const bool active = blk < nblk;
  const int blk_ld = active ? blk : nblk - 1;   // idle waves reload a valid block
  const int key0 = blk * kCrossBlock + grp * 8;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int h = 0; h < a.H; ++h) {
    bf16x8 qh[2], ql[2];
    load_q(a, row, h, grp, qh, ql);
    KTile t;
    load_k(a, h, off, blk_ld, c16, grp, t);
    const float2 st = a.stats[(size_t)row * a.H + h];
    float sv[8];
    scores8(t, qh, ql, key0, active ? T : 0, sv);
    const float il = 1.f / st.y;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] += sv[i] == -INFINITY ? 0.f : __expf(sv[i] - st.x) * il;
  }
  const int flag = a.rowflag[row];
  const int c = a.center[row];
  const float z = a.Z[row];
  const float inv = 1.f / (2.f * a.sigma * a.sigma);
  float ell = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    acc[i] = acc[i] / (float)a.H;
    const int j = key0 + i;
    if (active && j < T && (flag & 1)) {
      const float q = gauss(j, c, inv, z);
      if (q > 0.f) ell -= q * logf(acc[i]);
    }
  }
  if (active && r < a.R) {
    float* dst = a.abar + (size_t)row * a.abar_ld + key0;
    if (key0 + 8 <= T) {
      *(float4*)dst = float4{acc[0], acc[1], acc[2], acc[3]};
      *(float4*)(dst + 4) = float4{acc[4], acc[5], acc[6], acc[7]};
    } else {
      for (int i = 0; i < 8; ++i)
        if (key0 + i < T) dst[i] = acc[i];
    }
  }
  ell = rows4_sum(ell);
  if (grp == 0) part[w][c16] = ell;
  __syncthreads();
  if (threadIdx.x < 16 && tile * 16 + (int)threadIdx.x < a.R) {
    const float s = part[0][threadIdx.x] + part[1][threadIdx.x] + part[2][threadIdx.x] + part[3][threadIdx.x];
    a.lpart[(size_t)(b * a.R + tile * 16 + threadIdx.x) * a.nchunk + chunk] = s;
  }
}

// Gradient of lambda L_anchor for the query rows (0 for rows without an alignment).
__global__ void __launch_bounds__(kLossThreads) aloss_dq_kernel(LossArgs a) {
  __shared__ uint16_t kt[4][kCrossBlock * kKtStride];   // per wave: one block's keys, [key][dim]
  __shared__ float xy[4][2][kHead][16];                  // per wave: X, Y partials [dim][row]
  __shared__ float cpart[4][16];
  const int h = blockIdx.x, b = blockIdx.y, tile = blockIdx.z;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave, c16 = lane & 15, grp = lane >> 4;
  int T, off;
  if (!seq_frames(a, b, T, off)) {
    for (int e = threadIdx.x; e < 16 * kHead; e += kLossThreads) {
      const int rr = tile * 16 + e / kHead;
      if (rr < a.R) a.out_dxq[(size_t)(b * a.R + rr) * a.d + h * kHead + e % kHead] = 0.f;
    }
    return;
  }
  const int r = tile * 16 + c16;
  const int row = b * a.R + min(r, a.R - 1);
  bf16x8 qh[2], ql[2];
  load_q(a, row, h, grp, qh, ql);
  const float2 st = a.stats[(size_t)row * a.H + h];
  const float il = 1.f / st.y;
  const int flag = a.rowflag[row];
  const int c = a.center[row];
  const float z = a.Z[row];
  const float inv = 1.f / (2.f * a.sigma * a.sigma);
  const float* abar_row = a.abar + (size_t)row * a.abar_ld;
  const int nblk = (T + kCrossBlock - 1) / kCrossBlock;
  f32x4 X[4], Y[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) X[dt] = Y[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float cs = 0.f;
  uint16_t* myk = kt[w];
  // this lane's two key rows of the tile (products tt = 0, 1) and its 16 dims
  const int kA = 8 * (c16 >> 2) + (c16 & 3);
  for (int blk = w; blk < nblk; blk += 4) {
    KTile t;
    load_k(a, h, off, blk, c16, grp, t);
    const int key0 = blk * kCrossBlock + grp * 8;
    float sv[8];
    scores8(t, qh, ql, key0, T, sv);
    float p0[8], p1[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = key0 + i;
      const bool in = j < T;
      const float A = in ? __expf(sv[i] - st.x) * il : 0.f;
      float g = 0.f;
      if (in && (flag & 1)) {
        const float q = gauss(j, c, inv, z);
        if (q > 0.f) g = -q / ((float)a.H * abar_row[j]);
      }
      p0[i] = A;
      p1[i] = A * g;
      cs += A * g;
    }
    // keys [key][dim] into the wave's LDS tile, then dim-major 8-key operands
    uint2* d0 = (uint2*)(myk + kA * kKtStride + grp * 16);
    uint2* d1 = (uint2*)(myk + (kA + 4) * kKtStride + grp * 16);
    d0[0] = make_uint2(t.k00.x, t.k00.y);
    d0[1] = make_uint2(t.k00.z, t.k00.w);
    d0[2] = make_uint2(t.k01.x, t.k01.y);
    d0[3] = make_uint2(t.k01.z, t.k01.w);
    d1[0] = make_uint2(t.k10.x, t.k10.y);
    d1[1] = make_uint2(t.k10.z, t.k10.w);
    d1[2] = make_uint2(t.k11.x, t.k11.y);
    d1[3] = make_uint2(t.k11.z, t.k11.w);
    bf16x8 a0h, a0l, a1h, a1l;
    split8(p0, a0h, a0l);
    split8(p1, a1h, a1l);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const uint16_t* src = myk + (grp * 8) * kKtStride + dt * 16 + c16;
      uint32_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        v[u] = (uint32_t)src[(2 * u) * kKtStride] | ((uint32_t)src[(2 * u + 1) * kKtStride] << 16);
      const bf16x8 kT = as_bf16x8(make_uint4(v[0], v[1], v[2], v[3]));
      Y[dt] = mfma_bf16(kT, a0h, Y[dt]);
      Y[dt] = mfma_bf16(kT, a0l, Y[dt]);
      X[dt] = mfma_bf16(kT, a1h, X[dt]);
      X[dt] = mfma_bf16(kT, a1l, X[dt]);
    }
  }
  cs = rows4_sum(cs);
  if (grp == 0) cpart[w][c16] = cs;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xy[w][0][dt * 16 + grp * 4 + i][c16] = X[dt][i];
      xy[w][1][dt * 16 + grp * 4 + i][c16] = Y[dt][i];
    }
  __syncthreads();
  const int nv = a.counts[0];
  const float scale = nv > 0 ? a.lam / (float)nv * 0.125f : 0.f;
  for (int e = threadIdx.x; e < 16 * kHead; e += kLossThreads) {
    const int rr = e / kHead, dim = e % kHead;
    const int gr = tile * 16 + rr;
    if (gr >= a.R) continue;
    const float cc = cpart[0][rr] + cpart[1][rr] + cpart[2][rr] + cpart[3][rr];
    const float Xs = xy[0][0][dim][rr] + xy[1][0][dim][rr] + xy[2][0][dim][rr] + xy[3][0][dim][rr];
    const float Ys = xy[0][1][dim][rr] + xy[1][1][dim][rr] + xy[2][1][dim][rr] + xy[3][1][dim][rr];
    const bool al = a.rowflag[b * a.R + gr] & 1;
    a.out_dxq[(size_t)(b * a.R + gr) * a.d + h * kHead + dim] = al ? scale * (Xs - cc * Ys) : 0.f;
  }
}

// Token cross-entropy of one row (and its gradient): logsumexp - z[y].
__global__ void __launch_bounds__(kLossThreads) aloss_token_kernel(LossArgs a) {
  __shared__ float red[2][kLossThreads / kWave];
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* z = a.logits + (size_t)row * a.V;
  float* dz = a.out_dlogits ? a.out_dlogits + (size_t)row * a.V : nullptr;
  if (!(a.rowflag[row] & 2)) {
    if (dz)
      for (int j = tid; j < a.V; j += kLossThreads) dz[j] = 0.f;
    if (tid == 0) a.tok_row[row] = 0.f;
    return;
  }
  float m = -INFINITY, s = 0.f;
  for (int j0 = tid; j0 < a.V; j0 += 4 * kLossThreads) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = j0 + u * kLossThreads;
      v[u] = j < a.V ? z[j] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (v[u] == -INFINITY) continue;
      if (v[u] > m) {
        s = s * expf(m - v[u]) + 1.f;
        m = v[u];
      } else {
        s += expf(v[u] - m);
      }
    }
  }
  // merge the threads' (max, sum) pairs: wave butterflies, then the waves in order
  float M = wave_max(m);
  const int w = tid / kWave, l = tid % kWave;
  float S = wave_sum(m == -INFINITY ? 0.f : s * expf(m - M));
  if (l == 0) {
    red[0][w] = M;
    red[1][w] = S;
  }
  __syncthreads();
  float MM = red[0][0];
  for (int i = 1; i < kLossThreads / kWave; ++i) MM = fmaxf(MM, red[0][i]);
  float SS = 0.f;
  for (int i = 0; i < kLossThreads / kWave; ++i) SS += red[1][i] * expf(red[0][i] - MM);
  const float lse = MM + logf(SS);
  const int y = a.targets[row];
  if (tid == 0) a.tok_row[row] = lse - z[y];
  if (dz) {
    const float inv_n = 1.f / (float)a.counts[1];
    for (int j = tid; j < a.V; j += kLossThreads) dz[j] = (expf(z[j] - lse) - (j == y ? 1.f : 0.f)) * inv_n;
  }
}

// Smooth-L1 (beta = 1) feature term of one row (and its gradient, weight 0.5 included).
__global__ void __launch_bounds__(kLossThreads) aloss_feature_kernel(LossArgs a) {
  __shared__ float red[kLossThreads / kWave];
  const int row = blockIdx.x, tid = threadIdx.x;
  const bool tv = a.rowflag[row] & 2;
  const float* p = a.feat + (size_t)row * a.d;
  const float* q = a.feat_target + (size_t)row * a.d;
  float* dp = a.out_dfeat ? a.out_dfeat + (size_t)row * a.d : nullptr;
  const float gscale = tv ? 0.5f / ((float)a.counts[1] * (float)a.d) : 0.f;
  float s = 0.f;
  for (int j = tid; j < a.d; j += kLossThreads) {
    const float e = p[j] - q[j];
    const float ae = fabsf(e);
    if (tv) s += ae < 1.f ? 0.5f * e * e : ae - 0.5f;
    if (dp) dp[j] = fminf(fmaxf(e, -1.f), 1.f) * gscale;
  }
  s = block_sum<kLossThreads / kWave>(s, red);
  if (tid == 0) a.feat_row[row] = s;
}

// Totals in a fixed order: out_row, and {L, L_tok, L_feat, L_anchor}.
__global__ void __launch_bounds__(kLossThreads) aloss_final_kernel(LossArgs a) {
  __shared__ float red[kLossThreads / kWave];
  const int tid = threadIdx.x;
  float sa = 0.f, stok = 0.f, sf = 0.f;
  for (int row = tid; row < a.M; row += kLossThreads) {
    const int flag = a.rowflag[row];
    float ell = 0.f;
    if (flag & 1) {
      const int T = a.enc_len[row / a.R];
      const int nch = (T + kLossChunk - 1) / kLossChunk;
      for (int c = 0; c < nch; ++c) ell += a.lpart[(size_t)row * a.nchunk + c];
    }
    if (a.out_row) a.out_row[row] = ell;
    sa += ell;
    if (a.logits) stok += a.tok_row[row];
    if (a.feat) sf += a.feat_row[row];
  }
  sa = block_sum<kLossThreads / kWave>(sa, red);
  stok = block_sum<kLossThreads / kWave>(stok, red);
  sf = block_sum<kLossThreads / kWave>(sf, red);
  if (tid == 0) {
    const int nv = a.counts[0], nt = a.counts[1];
    const float la = nv > 0 ? sa / (float)nv : 0.f;
    const float lt = nt > 0 ? stok / (float)nt : 0.f;
    const float lf = nt > 0 ? sf / ((float)nt * (float)a.d) : 0.f;
    a.out_terms[0] = lt + 0.5f * lf + a.lam * la;
    a.out_terms[1] = lt;
    a.out_terms[2] = lf;
    a.out_terms[3] = la;
  }
}

int loss_chunks(int max_frames) { return (max_frames + kLossChunk - 1) / kLossChunk; }

void launch_anchordraft_loss(const LossArgs& a, hipStream_t st) {
  launch_zero_i32(a.counts, 2, st);
  const int tiles = (a.R + 15) / 16;
  hipLaunchKernelGGL(aloss_prep_kernel, dim3((a.M + 3) / 4), dim3(kLossThreads), 0, st, a);
  if (a.xq) {
    hipLaunchKernelGGL(aloss_stats_kernel, dim3(a.H, a.B, tiles), dim3(kLossThreads), 0, st, a);
    hipLaunchKernelGGL(aloss_abar_kernel, dim3(a.nchunk, a.B, tiles), dim3(kLossThreads), 0, st, a);
    if (a.out_dxq)
      hipLaunchKernelGGL(aloss_dq_kernel, dim3(a.H, a.B, tiles), dim3(kLossThreads), 0, st, a);
  }
  if (a.logits) hipLaunchKernelGGL(aloss_token_kernel, dim3(a.M), dim3(kLossThreads), 0, st, a);
  if (a.feat) hipLaunchKernelGGL(aloss_feature_kernel, dim3(a.M), dim3(kLossThreads), 0, st, a);
  hipLaunchKernelGGL(aloss_final_kernel, dim3(1), dim3(kLossThreads), 0, st, a);
}

}  // namespace ad
