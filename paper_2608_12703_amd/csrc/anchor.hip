// Verification-attention anchor readout (paper, section "Correction and Cost", paragraph
// "Verification-Attention Correction"; appendix "Runtime Correction"): the target's
// audio attention during verification, averaged over the heads of one decoder layer,
// peaks at the audio position of the next token, which centres the next draft window.
// Like the paper's runtime source, it is recomputed after verification from the layer's
// queries (kept by the cross-attention kernel of that layer) and its existing key cache;
// no extra decoder pass.  The row read is block row a_b, the last verified position,
// whose output is the bonus token.
//
// Two kernels after the accept scan:
//   scores: one workgroup per (head, sequence, 384-frame chunk) computes q.k / 8 for the
//           chunk's frames (float32) plus the chunk's (max, sum of exp(s - max));
//   pick:   one workgroup per sequence combines the chunk statistics into each head's
//           softmax normaliser (chunk order), averages the heads' weights per frame
//           (head order) and takes the frame with the largest average (lowest index on
//           ties).
// Keys are read once (the layer's K of every sequence, as the attention kernel does for
// one of its products); the scores round-trip through a small scratch buffer.
#include <algorithm>

#include "common.h"
#include "launch.h"

namespace ad {

template <class S>
__global__ void __launch_bounds__(256) anchor_scores_kernel(AnchorArgs a) {
  constexpr int kBlocks = kAnchorChunk / kCrossBlock;   // 12
  __shared__ float part[kBlocks][kCrossBlock][9];       // dot products of 8-dim pieces
  __shared__ float red[4];
  const int h = blockIdx.x, b = blockIdx.y, c = blockIdx.z;
  const SeqDesc s = a.seqs[b];
  const int acc = a.accept_len[b];
  if (!s.valid || acc < 0) return;
  const int f0 = c * kAnchorChunk;
  if (f0 >= s.T) return;
  const int f1 = min(f0 + kAnchorChunk, s.T);
  const int nblk = (f1 - f0 + kCrossBlock - 1) / kCrossBlock;
  const int tid = threadIdx.x;
  // this thread: frame t of every block of the chunk, dims j0 .. j0 + 7 (16 contiguous
  // bytes of the key layout)
  const int t = tid >> 3, g = tid & 7, j0 = g * 8;
  // the last verified row: row a_b of a chain, the accepted path's last node of a tree
  const int row = s.row0 + (a.path ? a.path[(size_t)b * a.path_stride + acc] : acc);
  const float* qp = a.q + (size_t)row * a.d + h * kHead + j0;
  const float4 qa = *(const float4*)qp, qb = *(const float4*)(qp + 4);
  const float q[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
  const typename S::T* kb = (const typename S::T*)a.kv + cross_base(a.layer, h, a.H, a.frames_cap);
  // every block's piece requested before any is used (blocks past the chunk reload its
  // last block; frames past T read valid slots of the sequence's 32-frame block)
  float kv[kBlocks][8];
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) {
    const int bi = i < nblk ? i : nblk - 1;
    const typename S::T* p = kb + cross_off(0, s.enc_off + f0 + bi * kCrossBlock + t, j0);
    if constexpr (sizeof(typename S::T) == 2) {   // 8 bf16 keys: one 16-byte load
      const uint4 v = *(const uint4*)p;
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kv[i][2 * e] = bf16_to_f32(w[e] & 0xffff);
        kv[i][2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[i][e] = S::ld(p, e);
    }
  }
#pragma unroll
  for (int i = 0; i < kBlocks; ++i) {
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) dot = fmaf(q[e], kv[i][e], dot);
    part[i][t][g] = dot;
  }
  __syncthreads();
  // frame scores (pieces summed in dim order; two frames per thread cover the chunk's
  // 384), then the chunk's max and sum
  float* sc = a.score + ((size_t)b * a.H + h) * a.max_frames;
  float sv[2];
  float m = -INFINITY;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int idx = tid + u * 256, i = idx / kCrossBlock, tt = idx % kCrossBlock;
    const int f = f0 + idx;
    sv[u] = -INFINITY;
    if (i < nblk && f < f1) {
      float d = 0.f;
#pragma unroll
      for (int gg = 0; gg < 8; ++gg) d += part[i][tt][gg];
      sv[u] = d * 0.125f;
      sc[f] = sv[u];
    }
    m = fmaxf(m, sv[u]);
  }
  m = wave_max(m);
  if ((tid & 63) == 0) red[tid >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float e = 0.f;
#pragma unroll
  for (int u = 0; u < 2; ++u)
    if (sv[u] != -INFINITY) e += expf(sv[u] - m);
  const float l = block_sum<4>(e, red);
  if (tid == 0) a.stats[((size_t)b * a.H + h) * a.nchunks + c] = make_float2(m, l);
}

constexpr int kPickThreads = 512;

__global__ void __launch_bounds__(kPickThreads) anchor_pick_kernel(AnchorArgs a) {
  constexpr int kHB = 8;                       // heads whose scores are loaded together
  constexpr int kNW = kPickThreads / kWave;
  __shared__ float Mh[64], Lh[64];
  __shared__ float bv[kNW];
  __shared__ int bi[kNW];
  const int b = blockIdx.x, tid = threadIdx.x;
  const SeqDesc s = a.seqs[b];
  const int acc = a.accept_len[b];
  if (!s.valid || acc < 0) {
    if (tid == 0) {
      a.out_anchor[b] = -1;
      if (a.out_peak) a.out_peak[b] = 0.f;
    }
    return;
  }
  const int T = s.T, H = a.H;
  // fused: the scores of every block row, one (max, sum) per head; else this sequence's
  // recomputed row, statistics per chunk
  const size_t base = a.fused ? (size_t)s.row0 + (a.path ? a.path[(size_t)b * a.path_stride + acc] : acc)
                              : (size_t)b;
  const int nch = a.fused ? 1 : (T + kAnchorChunk - 1) / kAnchorChunk;
  const int ld = a.fused ? a.score_ld : a.max_frames;
  // each head's softmax normaliser from its chunks, in chunk order
  for (int h = tid; h < H; h += kPickThreads) {
    const float2* st = a.stats + (base * H + h) * (a.fused ? 1 : a.nchunks);
    float M = -INFINITY;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, st[c].x);
    float L = 0.f;
    for (int c = 0; c < nch; ++c) L += st[c].y * expf(st[c].x - M);
    Mh[h] = M;
    Lh[h] = L;
  }
  __syncthreads();
  // head-averaged weight per frame (heads summed in order), two frames per pass and
  // eight heads' scores per round of loads; this thread's best (its frames rise, so
  // '>' keeps the lowest index among equal values)
  const float* sc = a.score + base * H * ld;
  float best = -1.f;
  int best_t = 0x7fffffff;
  for (int t0 = tid; t0 < T; t0 += 2 * kPickThreads) {
    float w[2] = {0.f, 0.f};
    for (int hb = 0; hb < H; hb += kHB) {
      float v[2][kHB];
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int e = 0; e < kHB; ++e) {
          const int h = min(hb + e, H - 1), t = min(t0 + f * kPickThreads, T - 1);
          v[f][e] = sc[(size_t)h * ld + t];
        }
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int e = 0; e < kHB; ++e)
          if (hb + e < H) w[f] += expf(v[f][e] - Mh[hb + e]) / Lh[hb + e];
    }
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int t = t0 + f * kPickThreads;
      const float wt = w[f] / (float)H;
      if (t < T && wt > best) {
        best = wt;
        best_t = t;
      }
    }
  }
  // block argmax: larger value, then lower frame
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(best, o, kWave);
    const int ot = __shfl_xor(best_t, o, kWave);
    const bool take = (ov > best) | ((ov == best) & (ot < best_t));
    best = take ? ov : best;
    best_t = take ? ot : best_t;
  }
  if ((tid & 63) == 0) {
    bv[tid >> 6] = best;
    bi[tid >> 6] = best_t;
  }
  __syncthreads();
  if (tid == 0) {
    float v = bv[0];
    int t = bi[0];
    for (int w = 1; w < kNW; ++w)
      if ((bv[w] > v) | ((bv[w] == v) & (bi[w] < t))) {
        v = bv[w];
        t = bi[w];
      }
    a.out_anchor[b] = t;
    if (a.out_peak) a.out_peak[b] = v;
  }
}

// Fused readout: the head-averaged weights of one block row, a slice of frames per
// workgroup (every frame's heads loaded at once), each slice's best (weight, lowest frame)
// merged with a 64-bit atomic max over (weight bits, ~frame): weights are >= 0, so their
// bits order like the values, and the result does not depend on the merge order.
constexpr int kPickSlices = 8, kSliceThreads = 256;
__global__ void __launch_bounds__(kSliceThreads) anchor_pick_slices_kernel(AnchorArgs a) {
  __shared__ float Mh[64], Lh[64];
  __shared__ unsigned long long red[kSliceThreads / kWave];
  const int b = blockIdx.x, slice = blockIdx.y, tid = threadIdx.x;
  const SeqDesc s = a.seqs[b];
  const int acc = a.accept_len[b];
  if (!s.valid || acc < 0) return;
  const int T = s.T, H = a.H, ld = a.score_ld;
  const size_t row = (size_t)s.row0 + (a.path ? a.path[(size_t)b * a.path_stride + acc] : acc);
  for (int h = tid; h < H; h += kSliceThreads) {
    const float2 st = a.stats[row * H + h];
    Mh[h] = st.x;
    Lh[h] = st.y;
  }
  __syncthreads();
  const int per = (T + kPickSlices - 1) / kPickSlices;
  const int t0 = slice * per, t1 = min(T, t0 + per);
  const float* sc = a.score + row * H * ld;
  unsigned long long best = 0;
  for (int t = t0 + tid; t < t1; t += kSliceThreads) {
    float w = 0.f;
    for (int h = 0; h < H; ++h) w += expf(sc[(size_t)h * ld + t] - Mh[h]) / Lh[h];
    w = w / (float)H;
    const unsigned long long key =
        ((unsigned long long)__float_as_uint(w) << 32) | (unsigned long long)(0xffffffffu - (unsigned)t);
    best = key > best ? key : best;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned long long other = __shfl_xor(best, o, kWave);
    best = other > best ? other : best;
  }
  if ((tid & 63) == 0) red[tid >> 6] = best;
  __syncthreads();
  if (tid == 0) {
    for (int i = 1; i < kSliceThreads / kWave; ++i) best = red[i] > best ? red[i] : best;
    if (best) atomicMax(a.best + b, best);
  }
}

// The merged best per sequence into the outputs; the slot is left at 0 for the next step.
__global__ void anchor_pick_final_kernel(AnchorArgs a, int B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const SeqDesc s = a.seqs[b];
  const bool ok = s.valid && a.accept_len[b] >= 0;
  const unsigned long long v = a.best[b];
  a.out_anchor[b] = ok ? (int)(0xffffffffu - (unsigned)(v & 0xffffffffu)) : -1;
  if (a.out_peak) a.out_peak[b] = ok ? __uint_as_float((unsigned)(v >> 32)) : 0.f;
  a.best[b] = 0;
}

int anchor_score_ld(int max_frames) { return (max_frames + kCrossBlock - 1) / kCrossBlock * kCrossBlock; }

size_t anchor_score_floats(int rows, int B, int H, int max_frames) {
  const size_t n = std::max((size_t)B * H * max_frames, (size_t)rows * H * anchor_score_ld(max_frames));
  return (n + 63) / 64 * 64;   // the statistics follow, aligned
}

size_t anchor_scratch_floats(int rows, int B, int H, int max_frames) {
  const int nch = (max_frames + kAnchorChunk - 1) / kAnchorChunk;
  return anchor_score_floats(rows, B, H, max_frames) +
         2 * std::max((size_t)B * H * nch, (size_t)rows * H);
}

template <class S>
void launch_anchor(const AnchorArgs& a, int B, hipStream_t st) {
  if (a.fused) {
    hipLaunchKernelGGL(anchor_pick_slices_kernel, dim3(B, kPickSlices), dim3(kSliceThreads), 0, st, a);
    hipLaunchKernelGGL(anchor_pick_final_kernel, dim3((B + 255) / 256), dim3(256), 0, st, a, B);
    return;
  }
  hipLaunchKernelGGL(anchor_scores_kernel<S>, dim3(a.H, B, a.nchunks), dim3(256), 0, st, a);
  hipLaunchKernelGGL(anchor_pick_kernel, dim3(B), dim3(kPickThreads), 0, st, a);
}
template void launch_anchor<F32>(const AnchorArgs&, int, hipStream_t);
template void launch_anchor<BF16>(const AnchorArgs&, int, hipStream_t);

}  // namespace ad
