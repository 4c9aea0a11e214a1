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
//           into Abar, the row's cross-entropy partial per 32-frame block, and
//           g_j = -q_t(j) / (H Abar_t(j)) kept in workspace for the gradient
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

// Per row: validation, the Gaussian normaliser over the sequence's valid frames and the
// row flags (bit 0 aligned, bit 1 has a next token).  One wave per row.  Frames further
// than 14 sigma from the centre are left out of the normaliser: their terms are below
// e^-98, under float32's smallest normal number.
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
    const float reach = ceilf(14.f * a.sigma);
    const int j0 = reach < (float)T ? max(0, c - (int)reach) : 0;
    const int j1 = reach < (float)T ? min(T, c + (int)reach + 1) : T;
    for (int j = j0 + lane; j < j1; j += kWave) {
      const float e = (float)(j - c);
      z += expf(-e * e * inv);
    }
    z = wave_sum(z);
  }
  if (lane == 0) {
    a.Z[row] = z;
    a.rowflag[row] = (av ? 1 : 0) | (tv ? 2 : 0);
    if (err) atomicOr(a.err, err);
  }
}

// |V| and |T| from the row flags (one workgroup, fixed order).
__global__ void __launch_bounds__(1024) aloss_count_kernel(LossArgs a) {
  __shared__ float red[1024 / kWave];
  float nv = 0.f, nt = 0.f;
  for (int row = threadIdx.x; row < a.M; row += 1024) {
    const int f = a.rowflag[row];
    nv += (f & 1) ? 1.f : 0.f;
    nt += (f & 2) ? 1.f : 0.f;
  }
  nv = block_sum<1024 / kWave>(nv, red);
  nt = block_sum<1024 / kWave>(nt, red);
  if (threadIdx.x == 0) {
    a.counts[0] = (int)nv;
    a.counts[1] = (int)nt;
  }
}

// Raw loads of one (head, block) step, issued together and used later: the loads of the
// next step go out before the current one is computed (straight-line ping-pong; loads
// complete in order, so waiting for one step leaves the next one's in flight).
struct QRaw {
  float4 q[4];
};
__device__ __forceinline__ void load_q_raw(const LossArgs& a, int row, int h, int grp, QRaw& r) {
  const float* p = a.xq + (size_t)row * a.d + h * kHead + grp * 16;
#pragma unroll
  for (int u = 0; u < 4; ++u) r.q[u] = *(const float4*)(p + 4 * u);
}
__device__ __forceinline__ void q_operands(const QRaw& r, bf16x8 (&qh)[2], bf16x8 (&ql)[2]) {
  float v[16];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    v[4 * u] = r.q[u].x * 0.125f;
    v[4 * u + 1] = r.q[u].y * 0.125f;
    v[4 * u + 2] = r.q[u].z * 0.125f;
    v[4 * u + 3] = r.q[u].w * 0.125f;
  }
  split8(v, qh[0], ql[0]);
  split8(v + 8, qh[1], ql[1]);
}

// Softmax statistics (max, sum of exp(score - max)) of every (row, head) over all valid
// frames.  Four waves take interleaved 32-frame blocks, two blocks in flight per wave;
// their partials merge in order.
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
  auto step = [&](const KTile& t, int blk) __attribute__((always_inline)) {
    float sv[8];
    scores8(t, qh, ql, blk * kCrossBlock + grp * 8, T, sv);   // blocks past T: all -inf
    float bm = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) bm = fmaxf(bm, sv[i]);
    const float mn = fmaxf(m, bm);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += sv[i] == -INFINITY ? 0.f : __expf(sv[i] - mn);
    const float keep = m == -INFINITY ? 0.f : __expf(m - mn);
    l = bm == -INFINITY ? l : l * keep + s;
    m = bm == -INFINITY ? m : mn;
  };
  KTile ta, tb;
  load_k(a, h, off, min(w, nblk - 1), c16, grp, ta);
  load_k(a, h, off, min(w + 4, nblk - 1), c16, grp, tb);
  for (int blk = w; blk < nblk; blk += 8) {
    step(ta, blk);
    load_k(a, h, off, min(blk + 8, nblk - 1), c16, grp, ta);
    step(tb, blk + 4);
    load_k(a, h, off, min(blk + 12, nblk - 1), c16, grp, tb);
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

// Head-averaged attention over one 128-frame chunk: four waves take interleaved heads
// (two in flight per wave), each computing the chunk's four 32-frame blocks from one
// load of the head's query operands; the waves' sums merge in wave order and wave w
// finishes block w: each row's cross-entropy partial, and g = -q / (H Abar) into
// workspace (0 where q is 0 or the row has no alignment).
constexpr int kAbarBlocks = 4;
__global__ void __launch_bounds__(kLossThreads) aloss_abar_kernel(LossArgs a) {
  __shared__ float part[4][kAbarBlocks][8][kWave];
  const int chunk = blockIdx.x, b = blockIdx.y, tile = blockIdx.z;
  int T, off;
  if (!seq_frames(a, b, T, off) || chunk * kAbarBlocks * kCrossBlock >= T) return;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave, c16 = lane & 15, grp = lane >> 4;
  const int r = tile * 16 + c16;
  const int row = b * a.R + min(r, a.R - 1);
  const int nblk = (T + kCrossBlock - 1) / kCrossBlock;
  const int blk0 = chunk * kAbarBlocks;
  float acc[kAbarBlocks][8];
#pragma unroll
  for (int q = 0; q < kAbarBlocks; ++q)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[q][i] = 0.f;
  struct HeadRaw {
    QRaw q;
    KTile k[kAbarBlocks];
    float2 st;
  };
  const int H = a.H;
  auto load = [&](int h, HeadRaw& v) __attribute__((always_inline)) {
    const int hh = min(h, H - 1);
    load_q_raw(a, row, hh, grp, v.q);
#pragma unroll
    for (int q = 0; q < kAbarBlocks; ++q) load_k(a, hh, off, min(blk0 + q, nblk - 1), c16, grp, v.k[q]);
    v.st = a.stats[(size_t)row * H + hh];
  };
  auto step = [&](const HeadRaw& v, bool on) __attribute__((always_inline)) {
    bf16x8 qh[2], ql[2];
    q_operands(v.q, qh, ql);
    const float il = 1.f / v.st.y;
#pragma unroll
    for (int q = 0; q < kAbarBlocks; ++q) {
      float sv[8];
      scores8(v.k[q], qh, ql, (blk0 + q) * kCrossBlock + grp * 8, T, sv);   // past T: -inf
#pragma unroll
      for (int i = 0; i < 8; ++i)
        acc[q][i] += (on && sv[i] != -INFINITY) ? __expf(sv[i] - v.st.x) * il : 0.f;
    }
  };
  HeadRaw va, vb;
  load(w, va);
  load(w + 4, vb);
  for (int h = w; h < H; h += 8) {
    step(va, true);
    load(h + 8, va);
    step(vb, h + 4 < H);
    load(h + 12, vb);
  }
#pragma unroll
  for (int q = 0; q < kAbarBlocks; ++q)
#pragma unroll
    for (int i = 0; i < 8; ++i) part[w][q][i][lane] = acc[q][i];
  __syncthreads();
  // wave w finishes block blk0 + w
  const int blk = blk0 + w;
  if (blk >= nblk) return;
  const int key0 = blk * kCrossBlock + grp * 8;
  const int flag = a.rowflag[row];
  const int c = a.center[row];
  const float z = a.Z[row];
  const float inv = 1.f / (2.f * a.sigma * a.sigma);
  float gv[8];
  float ell = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float ab = (((part[0][w][i][lane] + part[1][w][i][lane]) + part[2][w][i][lane]) +
                      part[3][w][i][lane]) / (float)H;
    const int j = key0 + i;
    gv[i] = 0.f;
    if (j < T && (flag & 1)) {
      const float q = gauss(j, c, inv, z);
      if (q > 0.f) {
        ell -= q * logf(ab);
        gv[i] = -q / ((float)H * ab);
      }
    }
  }
  if (r < a.R) {
    float* dst = a.gq + (size_t)row * a.g_ld + key0;
    if (key0 + 8 <= T) {
      *(float4*)dst = float4{gv[0], gv[1], gv[2], gv[3]};
      *(float4*)(dst + 4) = float4{gv[4], gv[5], gv[6], gv[7]};
    } else {
      for (int i = 0; i < 8; ++i)
        if (key0 + i < T) dst[i] = gv[i];
    }
  }
  ell = rows4_sum(ell);
  if (grp == 0 && r < a.R) a.lpart[(size_t)(b * a.R + r) * a.nchunk + blk] = ell;
}

// Gradient of lambda L_anchor for the query rows (0 for rows without an alignment).
// Four waves take interleaved 32-frame blocks, two in flight per wave (keys and the
// row's Abar values of the block); partials merge in wave order.
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
  const float* g_row = a.gq + (size_t)row * a.g_ld;   // g_j of the row
  const int nblk = (T + kCrossBlock - 1) / kCrossBlock;
  f32x4 X[4], Y[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) X[dt] = Y[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float cs = 0.f;
  uint16_t* myk = kt[w];
  // this lane's two key rows of the tile (products tt = 0, 1) and its 16 dims
  const int kA = 8 * (c16 >> 2) + (c16 & 3);
  struct BlkRaw {
    KTile k;
    float4 g0, g1;   // g of the lane's 8 keys (rows of the workspace hold whole 32-frame blocks)
  };
  auto load = [&](int blk, BlkRaw& v) __attribute__((always_inline)) {
    const int bl = min(blk, nblk - 1);
    load_k(a, h, off, bl, c16, grp, v.k);
    const float* p = g_row + bl * kCrossBlock + grp * 8;
    v.g0 = *(const float4*)p;
    v.g1 = *(const float4*)(p + 4);
  };
  auto step = [&](const BlkRaw& v, int blk) __attribute__((always_inline)) {
    const int key0 = blk * kCrossBlock + grp * 8;
    float sv[8];
    scores8(v.k, qh, ql, key0, T, sv);
    const float gg[8] = {v.g0.x, v.g0.y, v.g0.z, v.g0.w, v.g1.x, v.g1.y, v.g1.z, v.g1.w};
    float p0[8], p1[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool in = key0 + i < T;
      const float A = in ? __expf(sv[i] - st.x) * il : 0.f;
      const float g = in ? gg[i] : 0.f;   // (workspace past T is never written)
      p0[i] = A;
      p1[i] = A * g;
      cs += A * g;
    }
    // keys [key][dim] into the wave's LDS tile, then dim-major 8-key operands
    uint2* d0 = (uint2*)(myk + kA * kKtStride + grp * 16);
    uint2* d1 = (uint2*)(myk + (kA + 4) * kKtStride + grp * 16);
    d0[0] = make_uint2(v.k.k00.x, v.k.k00.y);
    d0[1] = make_uint2(v.k.k00.z, v.k.k00.w);
    d0[2] = make_uint2(v.k.k01.x, v.k.k01.y);
    d0[3] = make_uint2(v.k.k01.z, v.k.k01.w);
    d1[0] = make_uint2(v.k.k10.x, v.k.k10.y);
    d1[1] = make_uint2(v.k.k10.z, v.k.k10.w);
    d1[2] = make_uint2(v.k.k11.x, v.k.k11.y);
    d1[3] = make_uint2(v.k.k11.z, v.k.k11.w);
    bf16x8 a0h, a0l, a1h, a1l;
    split8(p0, a0h, a0l);
    split8(p1, a1h, a1l);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const uint16_t* src = myk + (grp * 8) * kKtStride + dt * 16 + c16;
      uint32_t kv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        kv[u] = (uint32_t)src[(2 * u) * kKtStride] | ((uint32_t)src[(2 * u + 1) * kKtStride] << 16);
      const bf16x8 kT = as_bf16x8(make_uint4(kv[0], kv[1], kv[2], kv[3]));
      Y[dt] = mfma_bf16(kT, a0h, Y[dt]);
      Y[dt] = mfma_bf16(kT, a0l, Y[dt]);
      X[dt] = mfma_bf16(kT, a1h, X[dt]);
      X[dt] = mfma_bf16(kT, a1l, X[dt]);
    }
  };
  BlkRaw va, vb;
  load(w, va);
  load(w + 4, vb);
  for (int blk = w; blk < nblk; blk += 8) {
    step(va, blk);
    load(blk + 8, va);
    step(vb, blk + 4);   // past the last block: every key masked, adds nothing
    load(blk + 12, vb);
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

// Token cross-entropy of one row (and its gradient): logsumexp - z[y].  The row stays in
// registers (kTokThreads threads x kTokPer values): the logits are read once and the
// gradient written once.  Up to 52 Ki logits, 512 threads x 102 values, two workgroups
// share a CU (one's loads overlap the other's arithmetic); up to 64 Ki, 1024 x 64.
template <int VEC, int kTokThreads, int kTokPer>
__global__ void __launch_bounds__(kTokThreads) __attribute__((amdgpu_waves_per_eu(kTokThreads == 512 ? 4 : 1)))
aloss_token_reg_kernel(LossArgs a) {
  __shared__ float red[kTokThreads / kWave];
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* z = a.logits + (size_t)row * a.V;
  float* dz = a.out_dlogits ? a.out_dlogits + (size_t)row * a.V : nullptr;
  if (!(a.rowflag[row] & 2)) {
    if (dz)
      for (int j = tid; j < a.V; j += kTokThreads) dz[j] = 0.f;
    if (tid == 0) a.tok_row[row] = 0.f;
    return;
  }
  // element u of this thread: logit (u / VEC) * VEC * 1024 + VEC * tid + u % VEC
  auto col = [&](int u) { return (u / VEC) * VEC * kTokThreads + VEC * tid + u % VEC; };
  float v[kTokPer];
#pragma unroll
  for (int u = 0; u < kTokPer; u += VEC) {
    const int j = col(u);
    if (VEC == 2) {
      const float2 p = j < a.V ? *(const float2*)(z + j) : float2{-INFINITY, -INFINITY};
      v[u] = p.x;
      v[u + 1] = p.y;
    } else {
      v[u] = j < a.V ? z[j] : -INFINITY;
    }
  }
  float m = v[0];
#pragma unroll
  for (int u = 1; u < kTokPer; ++u) m = fmaxf(m, v[u]);
  m = wave_max(m);
  const int w = tid / kWave, l = tid % kWave;
  if (l == 0) red[w] = m;
  __syncthreads();
  float M = red[0];
  for (int i = 1; i < kTokThreads / kWave; ++i) M = fmaxf(M, red[i]);
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < kTokPer; ++u) {
    v[u] = v[u] == -INFINITY ? 0.f : __expf(v[u] - M);   // v now holds exp(z - M)
    s += v[u];
  }
  const float S = block_sum<kTokThreads / kWave>(s, red);
  const int y = a.targets[row];
  if (tid == 0) a.tok_row[row] = M + logf(S) - z[y];
  if (dz) {
    const float inv_s = 1.f / S, inv_n = 1.f / (float)a.counts[1];
#pragma unroll
    for (int u = 0; u < kTokPer; u += VEC) {
      const int j = col(u);
      if (j >= a.V) continue;
      if (VEC == 2) {
        *(float2*)(dz + j) = float2{(v[u] * inv_s - (j == y ? 1.f : 0.f)) * inv_n,
                                    (v[u + 1] * inv_s - (j + 1 == y ? 1.f : 0.f)) * inv_n};
      } else {
        dz[j] = (v[u] * inv_s - (j == y ? 1.f : 0.f)) * inv_n;
      }
    }
  }
}

// The same for larger vocabularies: two passes over the logits.
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

// Each row's alignment cross-entropy: the sum of its block partials (one wave per row,
// a fixed butterfly).
__global__ void __launch_bounds__(kLossThreads) aloss_rowsum_kernel(LossArgs a) {
  const int row = blockIdx.x * (kLossThreads / kWave) + threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (row >= a.M) return;
  float ell = 0.f;
  if (a.rowflag[row] & 1) {
    const int T = a.enc_len[row / a.R];
    const int nb = (T + kCrossBlock - 1) / kCrossBlock;
    const float* p = a.lpart + (size_t)row * a.nchunk;
    for (int c = lane; c < nb; c += kWave) ell += p[c];
    ell = wave_sum(ell);
  }
  if (lane == 0) {
    a.lrow[row] = ell;
    if (a.out_row) a.out_row[row] = ell;
  }
}

// Totals in a fixed order: {L, L_tok, L_feat, L_anchor}.
__global__ void __launch_bounds__(1024) aloss_final_kernel(LossArgs a) {
  __shared__ float red[1024 / kWave];
  const int tid = threadIdx.x;
  float sa = 0.f, stok = 0.f, sf = 0.f;
  for (int row = tid; row < a.M; row += 1024) {
    if (a.xq) sa += a.lrow[row];
    if (a.logits) stok += a.tok_row[row];
    if (a.feat) sf += a.feat_row[row];
  }
  sa = block_sum<1024 / kWave>(sa, red);
  stok = block_sum<1024 / kWave>(stok, red);
  sf = block_sum<1024 / kWave>(sf, red);
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

int loss_chunks(int max_frames) { return (max_frames + kCrossBlock - 1) / kCrossBlock; }

void launch_anchordraft_loss(const LossArgs& a, hipStream_t st) {
  const int tiles = (a.R + 15) / 16;
  hipLaunchKernelGGL(aloss_prep_kernel, dim3((a.M + 3) / 4), dim3(kLossThreads), 0, st, a);
  hipLaunchKernelGGL(aloss_count_kernel, dim3(1), dim3(1024), 0, st, a);
  if (a.xq) {
    hipLaunchKernelGGL(aloss_stats_kernel, dim3(a.H, a.B, tiles), dim3(kLossThreads), 0, st, a);
    hipLaunchKernelGGL(aloss_abar_kernel, dim3((a.nchunk + kAbarBlocks - 1) / kAbarBlocks, a.B, tiles),
                       dim3(kLossThreads), 0, st, a);
    if (a.out_dxq)
      hipLaunchKernelGGL(aloss_dq_kernel, dim3(a.H, a.B, tiles), dim3(kLossThreads), 0, st, a);
  }
  if (a.logits && a.V <= 512 * 102 && a.V % 2 == 0)
    hipLaunchKernelGGL((aloss_token_reg_kernel<2, 512, 102>), dim3(a.M), dim3(512), 0, st, a);
  else if (a.logits && a.V <= 1024 * 64 && a.V % 2 == 0)
    hipLaunchKernelGGL((aloss_token_reg_kernel<2, 1024, 64>), dim3(a.M), dim3(1024), 0, st, a);
  else if (a.logits && a.V <= 1024 * 64)
    hipLaunchKernelGGL((aloss_token_reg_kernel<1, 1024, 64>), dim3(a.M), dim3(1024), 0, st, a);
  else if (a.logits)
    hipLaunchKernelGGL(aloss_token_kernel, dim3(a.M), dim3(kLossThreads), 0, st, a);
  if (a.feat) hipLaunchKernelGGL(aloss_feature_kernel, dim3(a.M), dim3(kLossThreads), 0, st, a);
  if (a.xq) hipLaunchKernelGGL(aloss_rowsum_kernel, dim3((a.M + 3) / 4), dim3(kLossThreads), 0, st, a);
  hipLaunchKernelGGL(aloss_final_kernel, dim3(1), dim3(1024), 0, st, a);
}

}  // namespace ad
