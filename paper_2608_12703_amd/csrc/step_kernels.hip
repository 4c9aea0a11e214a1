// Small kernels of the verify step: descriptor preparation and validation, embedding,
// LayerNorm, argmax with top-2 margin, the prefix-accept scan, commit, prefix import and
// the draft-head helpers.
#include "common.h"
#include "launch.h"

namespace ad {

// ---------------------------------------------------------------- descriptors

__global__ void prep_seq_kernel(StepArgs a, SeqDesc* seqs, int* err) {
  for (int b = threadIdx.x + blockIdx.x * blockDim.x; b < a.B; b += blockDim.x * gridDim.x) {
    const int kb = a.k[b];
    const int n = a.kv_len[b];
    const int T = a.enc_len[b];
    const int off = a.enc_off[b];
    int row0 = a.layout == 0 ? b * (a.k_max + 1) : a.cu_rows[b];
    int e = 0;
    if (kb < 0 || kb > a.k_max || n < 0 || n + kb + 1 > a.max_pos) e |= 1;
    if (a.layout == 1) {
      const int r1 = a.cu_rows[b + 1];
      if (row0 < 0 || r1 > a.rows || r1 - row0 != kb + 1) e |= 1;
    }
    if (T < 1 || T > a.max_frames || off < 0 || (off % kCrossBlock) || off + T > a.frames_cap)
      e |= 8;
    int wlo = 0, whi = T;
    if (a.cross_window) {
      wlo = a.cross_window[2 * b];
      whi = a.cross_window[2 * b + 1];
      if (wlo < 0 || whi > T || wlo >= whi) e |= 8;
    }
    if (!(e & 1)) {
      const int last_page = (n + kb) / kTile;
      if (last_page >= a.pages_per_seq) {
        e |= 2;
      } else {
        for (int p = 0; p <= last_page; ++p) {
          const int pg = a.block_table[(size_t)b * a.pages_per_seq + p];
          if (pg < 0 || pg >= a.num_pages) e |= 2;
        }
      }
      for (int i = 0; i <= kb; ++i) {
        const int t = a.tokens[row0 + i];
        if (t < 0 || t >= a.V) e |= 4;
      }
      // depth and ancestor mask of every block row: a draft tree's parents must be earlier
      // rows; without a tree the rows form a chain (row i's parent is row i - 1)
      if (!(e & 1) && !a.parents) {
        for (int i = 0; i <= kb; ++i) a.tree[row0 + i] = RowTree{(2ull << i) - 1, i, 0};
      } else if (!(e & 1)) {
        for (int i = 0; i <= kb; ++i) {
          const int p = i == 0 ? -1 : a.parents[row0 + i];
          if (i > 0 && (p < 0 || p >= i)) {
            e |= 32;
            break;
          }
          RowTree r;
          r.depth = i == 0 ? 0 : a.tree[row0 + p].depth + 1;
          r.mask = (i == 0 ? 0ull : a.tree[row0 + p].mask) | (1ull << i);
          r.pad = 0;
          a.tree[row0 + i] = r;
        }
      }
    }
    if (e) atomicOr(err, e);
    if (e & 1) row0 = 0;
    seqs[b] = SeqDesc{row0, e ? 0 : kb, e ? 0 : n, e ? 1 : T, e ? 0 : off, e == 0, e ? 0 : wlo,
                      e ? 1 : whi};
  }
}

__global__ void prep_row_kernel(StepArgs a, const SeqDesc* seqs, RowDesc* rows) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= a.rows) return;
  int b, i;
  if (a.layout == 0) {
    b = m / (a.k_max + 1);
    i = m % (a.k_max + 1);
  } else {
    // last sequence whose first row is <= m (bounded binary search over cu_rows)
    int lo = 0, hi = a.B - 1;
    b = -1;
    while (lo <= hi) {
      const int mid = (lo + hi) >> 1;
      if (a.cu_rows[mid] <= m) { b = mid; lo = mid + 1; } else { hi = mid - 1; }
    }
    i = b >= 0 ? m - a.cu_rows[b] : 0;
  }
  RowDesc r{-1, 0, 0, 0, 0};
  if (b >= 0 && b < a.B) {
    const SeqDesc s = seqs[b];
    if (s.valid && i >= 0 && i <= s.k && s.row0 + i == m) {
      r.seq = b;
      r.i = i;
      r.pos = s.n + a.tree[m].depth;
      r.slot = s.n + i;
      r.token = a.tokens[m];
    }
  }
  rows[m] = r;
}

// ---------------------------------------------------------------- embedding

template <class S>
__global__ void embed_kernel(int d, const RowDesc* rows, const typename S::T* tok_emb,
                             const typename S::T* pos_emb, float* x, const float* in_rows) {
  const int m = blockIdx.x;
  const RowDesc r = rows[m];
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    x[(size_t)m * d + j] = (in_rows ? in_rows[(size_t)m * d + j] : S::ld(tok_emb, (size_t)r.token * d + j)) +
                           S::ld(pos_emb, (size_t)r.pos * d + j);
}

// ---------------------------------------------------------------- LayerNorm
// out = (x - mean) / sqrt(var + 1e-5) * g + b, biased variance, two passes over the row.

template <class S>
__global__ void __launch_bounds__(256) layernorm_kernel(int d, const float* x,
                                                        const typename S::T* g,
                                                        const typename S::T* b, float* out) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * d;
  float s = 0.f;
  for (int j = threadIdx.x; j < d; j += 256) s += xr[j];
  const float mean = block_sum<4>(s, red) / (float)d;
  float v = 0.f;
  for (int j = threadIdx.x; j < d; j += 256) {
    const float t = xr[j] - mean;
    v += t * t;
  }
  const float var = block_sum<4>(v, red) / (float)d;
  const float rstd = 1.0f / sqrtf(var + 1e-5f);
  for (int j = threadIdx.x; j < d; j += 256)
    out[(size_t)m * d + j] = (xr[j] - mean) * rstd * S::ld(g, j) + S::ld(b, j);
}

// Same normalisation, written as the hi/lo A operand of the next bf16 product.
template <class S>
__global__ void __launch_bounds__(256) layernorm_frag_kernel(int d, const float* x,
                                                             const typename S::T* g,
                                                             const typename S::T* b,
                                                             uint16_t* frag, int RT, float* out) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * d;
  float s = 0.f;
  for (int j = threadIdx.x; j < d; j += 256) s += xr[j];
  const float mean = block_sum<4>(s, red) / (float)d;
  float v = 0.f;
  for (int j = threadIdx.x; j < d; j += 256) {
    const float t = xr[j] - mean;
    v += t * t;
  }
  const float var = block_sum<4>(v, red) / (float)d;
  const float rstd = 1.0f / sqrtf(var + 1e-5f);
  for (int j = threadIdx.x; j < d; j += 256) {
    const float y = (xr[j] - mean) * rstd * S::ld(g, j) + S::ld(b, j);
    afrag_store(frag, RT, m, j, y);
    if (out) out[(size_t)m * d + j] = y;
  }
}

// Split-K epilogue of the residual-writing products fused with the next LayerNorm:
//   x[m] += sum_s P[s][m] + bias   (partials in split order)
//   frag[m] = LN(x[m]) in A-fragment order (and, when out is given, also as float32).
// One workgroup per row; the row is held in LDS.
// Sum over the block's waves in wave order; every thread gets the total.
__device__ __forceinline__ float row_block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// split_sum4 with the first eight planes as straight-line loads (planes past nsplit
// are clamped reads that add -0, which leaves every value, signed zeros included,
// unchanged): no loop, so loads issued before it stay in flight across it.  Further
// planes, if any, in a loop.
__device__ __forceinline__ float4 split_sum4_flat(const float* P, size_t plane, size_t e, int nsplit) {
  float4 p[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) p[u] = *(const float4*)(P + (size_t)min(u, nsplit - 1) * plane + e);
  float4 acc = p[0];
#pragma unroll
  for (int u = 1; u < 8; ++u) {
    const bool in = u < nsplit;
    acc.x += in ? p[u].x : -0.f;
    acc.y += in ? p[u].y : -0.f;
    acc.z += in ? p[u].z : -0.f;
    acc.w += in ? p[u].w : -0.f;
  }
  for (int t = 8; t < nsplit; ++t) {
    const float4 w = *(const float4*)(P + (size_t)t * plane + e);
    acc.x += w.x; acc.y += w.y; acc.z += w.z; acc.w += w.w;
  }
  return acc;
}

// The same for a `red` array that no other reduction of the kernel uses (no barrier
// needed before writing it).
__device__ __forceinline__ float row_block_sum_once(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

__device__ __forceinline__ float4 ld_bf16x4(const uint16_t* p, int j) {
  const uint2 u = *(const uint2*)(p + j);
  return float4{bf16_to_f32(u.x & 0xffff), bf16_to_f32(u.x >> 16), bf16_to_f32(u.y & 0xffff),
                bf16_to_f32(u.y >> 16)};
}

// Row of workgroup `bid` for the row-per-workgroup kernels that write A-fragment
// operands.  Workgroups are dealt round-robin over the 8 XCDs; this numbering puts the
// 8 rows that share each 128-byte line of the output (rows 8a .. 8a + 7) on one XCD, so
// its L2 merges their 16-byte pieces into whole lines.  Launch ceil(M / 64) * 64
// workgroups; rows past M exit.
__device__ __forceinline__ int xcd_row(int bid) {
  return (bid >> 6) * 64 + (bid & 7) * 8 + ((bid >> 3) & 7);
}
__host__ inline int xcd_row_grid(int M) { return (M + 63) / 64 * 64; }

// Residual update and the next LayerNorm of one row: x += sum_s P[s] + bias, then
// LN(x) * g + b goes out in A-fragment order (and to `out` when given).  One thread per
// 4 columns (blockDim = d / 4 rounded up to whole waves).
__global__ void __launch_bounds__(1024) reduce_res_ln_kernel(int M, int d, int nsplit,
                                                             const float* P, const uint16_t* bias,
                                                             float* x, const uint16_t* g,
                                                             const uint16_t* b, uint16_t* frag,
                                                             int RT, float* out) {
  __shared__ float red_mean[16], red_var[16];
  const int m = xcd_row(blockIdx.x), j = threadIdx.x * 4;
  if (m >= M) return;
  const bool on = j < d;
  const int jc = on ? j : 0;
  const size_t e = (size_t)m * d + jc;
  // every load of the row up front (one round trip): partials, bias, residual, and the
  // LayerNorm gain and shift
  const float4 bb = ld_bf16x4(bias, jc);
  const float4 x0 = *(const float4*)(x + e);
  const float4 gv = ld_bf16x4(g, jc), bv = ld_bf16x4(b, jc);
  const float4 v = split_sum4_flat(P, (size_t)M * d, e, nsplit);
  float4 xv{0.f, 0.f, 0.f, 0.f};
  if (on) {
    xv = x0;
    xv.x += v.x + bb.x; xv.y += v.y + bb.y; xv.z += v.z + bb.z; xv.w += v.w + bb.w;
    *(float4*)(x + e) = xv;
  }
  const float mean = row_block_sum_once(on ? (xv.x + xv.y) + (xv.z + xv.w) : 0.f, red_mean) / (float)d;
  const float4 c{xv.x - mean, xv.y - mean, xv.z - mean, xv.w - mean};
  const float var = row_block_sum_once(on ? (c.x * c.x + c.y * c.y) + (c.z * c.z + c.w * c.w) : 0.f, red_var);
  const float rstd = 1.0f / sqrtf(var / (float)d + 1e-5f);
  if (on) {
    const float4 y{c.x * rstd * gv.x + bv.x, c.y * rstd * gv.y + bv.y, c.z * rstd * gv.z + bv.z,
                   c.w * rstd * gv.w + bv.w};
    afrag_store4(frag, RT, m, j, y);
    if (out) *(float4*)(out + e) = y;
  }
}

// Embedding of the block rows fused with the first LayerNorm: x = E_tok[token] (or the
// caller's input row) + E_pos[pos], then LN(x) * g + b in A-fragment order.  One thread
// per 4 columns (blockDim = d / 4 rounded up to whole waves), every load up front.
__global__ void __launch_bounds__(1024) embed_ln_kernel(int M, int d, const RowDesc* rows,
                                                       const uint16_t* tok_emb,
                                                       const uint16_t* pos_emb, float* x,
                                                       const float* in_rows, const uint16_t* g,
                                                       const uint16_t* b, uint16_t* frag, int RT) {
  __shared__ float red_mean[16], red_var[16];
  const int m = xcd_row(blockIdx.x), j = threadIdx.x * 4;
  if (m >= M) return;
  const bool on = j < d;
  const int jc = on ? j : 0;
  const float4 gv = ld_bf16x4(g, jc), bv = ld_bf16x4(b, jc);
  const RowDesc r = rows[m];
  const float4 te = in_rows ? *(const float4*)(in_rows + (size_t)m * d + jc)
                            : ld_bf16x4(tok_emb + (size_t)r.token * d, jc);
  const float4 pe = ld_bf16x4(pos_emb + (size_t)r.pos * d, jc);
  const float4 v{te.x + pe.x, te.y + pe.y, te.z + pe.z, te.w + pe.w};
  if (on) *(float4*)(x + (size_t)m * d + j) = v;
  const float mean = row_block_sum_once(on ? (v.x + v.y) + (v.z + v.w) : 0.f, red_mean) / (float)d;
  const float4 c{v.x - mean, v.y - mean, v.z - mean, v.w - mean};
  const float var = row_block_sum_once(on ? (c.x * c.x + c.y * c.y) + (c.z * c.z + c.w * c.w) : 0.f, red_var);
  const float rstd = 1.0f / sqrtf(var / (float)d + 1e-5f);
  if (on)
    afrag_store4(frag, RT, m, j,
                 float4{c.x * rstd * gv.x + bv.x, c.y * rstd * gv.y + bv.y, c.z * rstd * gv.z + bv.z,
                        c.w * rstd * gv.w + bv.w});
}

__global__ void zero_i32_kernel(int* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += blockDim.x * gridDim.x) p[i] = 0;
}

// ---------------------------------------------------------------- argmax + margin
// Per row: largest logit (lowest index on ties) and the runner-up value.

struct Top2 {
  float v1;
  int i1;
  float v2;
};
__device__ __forceinline__ Top2 top2_merge(Top2 a, Top2 b) {
  const bool a_wins = (a.v1 > b.v1) || (a.v1 == b.v1 && a.i1 < b.i1);
  Top2 r;
  if (a_wins) { r.v1 = a.v1; r.i1 = a.i1; r.v2 = fmaxf(a.v2, b.v1); }
  else        { r.v1 = b.v1; r.i1 = b.i1; r.v2 = fmaxf(b.v2, a.v1); }
  return r;
}

__global__ void __launch_bounds__(256) argmax_kernel(int V, const float* logits, size_t ld,
                                                     const RowDesc* rows, int* greedy,
                                                     float* margin, int* err) {
  __shared__ Top2 red[4];
  __shared__ int bad_s;
  const int m = blockIdx.x;
  const float* lr = logits + (size_t)m * ld;
  if (threadIdx.x == 0) bad_s = 0;
  __syncthreads();
  Top2 t{-INFINITY, 0x7fffffff, -INFINITY};
  int bad = 0;
  // this thread's indices j = tid, tid + 256, ... in increasing order; sixteen loads are
  // requested before they are used (a row's scan is otherwise one round trip per value)
  auto take = [&](float v, int j) {
    if (!isfinite(v)) { bad = 1; return; }
    if (v > t.v1) { t.v2 = t.v1; t.v1 = v; t.i1 = j; }
    else if (v > t.v2) { t.v2 = v; }
  };
  int j0 = threadIdx.x;
  for (; j0 + 15 * 256 < V; j0 += 16 * 256) {
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = lr[j0 + u * 256];
#pragma unroll
    for (int u = 0; u < 16; ++u) take(v[u], j0 + u * 256);
  }
  for (int j = j0; j < V; j += 256) take(lr[j], j);
  if (bad) atomicOr(&bad_s, 1);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    Top2 u;
    u.v1 = __shfl_xor(t.v1, o, kWave);
    u.i1 = __shfl_xor(t.i1, o, kWave);
    u.v2 = __shfl_xor(t.v2, o, kWave);
    t = top2_merge(t, u);
  }
  const int w = threadIdx.x / kWave;
  if (threadIdx.x % kWave == 0) red[w] = t;
  __syncthreads();
  if (threadIdx.x == 0) {
    Top2 r = red[0];
    for (int i = 1; i < 4; ++i) r = top2_merge(r, red[i]);
    const bool valid_row = rows ? rows[m].seq >= 0 : true;
    if (bad_s && valid_row && err) atomicOr(err, 16);
    greedy[m] = (bad_s && valid_row) ? -1 : r.i1;
    if (margin) margin[m] = r.v1 - r.v2;
  }
}

// ---------------------------------------------------------------- accept / commit

__global__ void accept_kernel(int B, int k_max, const SeqDesc* seqs, const int* tokens,
                              const int* greedy, int* accept_len, int* out_tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const SeqDesc s = seqs[b];
  int a = -1;
  if (s.valid) {
    bool ok = true;
    for (int i = 0; i <= s.k; ++i) ok = ok && greedy[s.row0 + i] >= 0;
    if (ok) {
      a = 0;
      while (a < s.k && tokens[s.row0 + 1 + a] == greedy[s.row0 + a]) ++a;
    }
  }
  accept_len[b] = a;
  for (int i = 0; i <= k_max; ++i)
    out_tokens[(size_t)b * (k_max + 1) + i] = (a >= 0 && i <= a) ? greedy[s.row0 + i] : -1;
}

// Draft-tree accept: from the root, move to the lowest-index child whose token equals the
// current node's greedy token; the emitted tokens are the greedy tokens along the path.
__global__ void accept_tree_kernel(int B, int k_max, const SeqDesc* seqs, const int* tokens,
                                   const int* parents, const int* greedy, int* accept_len,
                                   int* out_tokens, int* out_path) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const SeqDesc s = seqs[b];
  int* path = out_path + (size_t)b * (k_max + 1);
  int a = -1;
  if (s.valid) {
    bool ok = true;
    for (int i = 0; i <= s.k; ++i) ok = ok && greedy[s.row0 + i] >= 0;
    if (ok) {
      a = 0;
      path[0] = 0;
      int u = 0;
      while (true) {
        const int g = greedy[s.row0 + u];
        int nxt = -1;
        for (int c = u + 1; c <= s.k && nxt < 0; ++c)
          if (parents[s.row0 + c] == u && tokens[s.row0 + c] == g) nxt = c;
        if (nxt < 0) break;
        u = nxt;
        path[++a] = u;
      }
    }
  }
  accept_len[b] = a;
  for (int i = 0; i <= k_max; ++i) {
    const bool on = a >= 0 && i <= a;
    out_tokens[(size_t)b * (k_max + 1) + i] = on ? greedy[s.row0 + path[i]] : -1;
    if (!on) path[i] = -1;
  }
}

// Accepted tree path node j (block row path[j], slot n + path[j]) -> slot n + j, for one
// (layer, K|V) per block, eight nodes at a time: each thread moves the same (head, lane)
// element of every slot, reading all eight sources before writing any destination.  A
// source is never an earlier node's destination (path[j] >= j), so reading a batch before
// writing it, and batches in path order, move every slot's original contents.
template <class S>
__global__ void __launch_bounds__(256) kv_compact_kernel(int H, const int* kv_len, const int* accept_len,
                                                         const int* path, int path_stride,
                                                         typename S::T* pool, int num_pages,
                                                         const int* block_table, int pages_per_seq) {
  using T = typename S::T;
  const int b = blockIdx.x, layer = blockIdx.y >> 1, kv = blockIdx.y & 1;
  const int a = min(accept_len[b], path_stride - 1);
  if (a <= 0) return;
  const int n = kv_len[b];
  const int* p = path + (size_t)b * path_stride;
  for (int j0 = 1; j0 <= a; j0 += 8) {
    size_t sb[8], db[8];
    bool mv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u;
      const int node = j <= a ? p[j] : 0;
      // (a path row never precedes its index; slots past the block table are left alone)
      mv[u] = j <= a && node > j && (n + node) / kTile < pages_per_seq;
      const int src = mv[u] ? n + node : 0, dst = mv[u] ? n + j : 0;
      const int ps = min(max(block_table[(size_t)b * pages_per_seq + src / kTile], 0), num_pages - 1);
      const int pd = min(max(block_table[(size_t)b * pages_per_seq + dst / kTile], 0), num_pages - 1);
      sb[u] = kv_tile_base(layer, kv, ps, 0, num_pages, H) + tile_off(kv, src % kTile, 0);
      db[u] = kv_tile_base(layer, kv, pd, 0, num_pages, H) + tile_off(kv, dst % kTile, 0);
    }
    for (int e = threadIdx.x; e < H * kHead; e += blockDim.x) {
      const int h = e / kHead, c = e % kHead;
      const size_t off = (size_t)h * kTileElems + (tile_off(kv, 0, c));
      T v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = mv[u] ? pool[sb[u] + off] : T();
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (mv[u]) pool[db[u] + off] = v[u];
    }
  }
}

__global__ void commit_kernel(int B, int* kv_len, const int* accept_len) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int a = accept_len[b];
  if (a >= 0) kv_len[b] += a + 1;
}

// ---------------------------------------------------------------- prefix import

// EXPORT = false: src [L][2][n][H][64] -> pool; EXPORT = true: pool -> dst.
template <class S, bool EXPORT>
__global__ void kv_copy_kernel(int L, int H, int n, int b, typename S::T* lin,
                               typename S::T* pool, int num_pages, const int* block_table,
                               int pages_per_seq, int* err) {
  // one thread per element of the logical array [L][2][n][H][64]
  const size_t total = (size_t)L * 2 * n * H * kHead;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  size_t r = idx;
  const int j = r % kHead; r /= kHead;
  const int h = r % H; r /= H;
  const int p = r % n; r /= n;
  const int kv = r % 2; r /= 2;
  const int layer = (int)r;
  const int pg = block_table[(size_t)b * pages_per_seq + p / kTile];
  if (pg < 0 || pg >= num_pages) {
    atomicOr(err, 2);
    return;
  }
  const size_t at = kv_tile_base(layer, kv, pg, h, num_pages, H) + tile_off(kv, p % kTile, j);
  if (EXPORT) lin[idx] = pool[at];
  else pool[at] = lin[idx];
}

// ---------------------------------------------------------------- draft heads

__global__ void gather_hidden_kernel(int B, int d, int layout, int k_max, const int* cu_rows,
                                     const int* accept_len, const float* hidden, float* hsel) {
  const int b = blockIdx.x;
  const int a = accept_len[b];
  const int row0 = layout == 0 ? b * (k_max + 1) : cu_rows[b];
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    hsel[(size_t)b * d + j] = a >= 0 ? hidden[(size_t)(row0 + a) * d + j] : 0.f;
}

__global__ void assemble_next_kernel(int B, int n_heads, int k_max, const int* accept_len,
                                     const int* out_tokens, const int* head_greedy,
                                     int* next_tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int a = accept_len[b];
  int* nt = next_tokens + (size_t)b * (n_heads + 1);
  nt[0] = a >= 0 ? out_tokens[(size_t)b * (k_max + 1) + a] : -1;
  for (int i = 0; i < n_heads; ++i) nt[1 + i] = a >= 0 ? head_greedy[(size_t)i * B + b] : -1;
}

// ---------------------------------------------------------------- launchers

void launch_prep(const StepArgs& a, SeqDesc* seqs, RowDesc* rows, int* err, hipStream_t st) {
  hipLaunchKernelGGL(prep_seq_kernel, dim3((a.B + 255) / 256), dim3(256), 0, st, a, seqs, err);
  hipLaunchKernelGGL(prep_row_kernel, dim3((a.rows + 255) / 256), dim3(256), 0, st, a, seqs, rows);
}

template <class S>
void launch_embed(int M, int d, const RowDesc* rows, const void* tok, const void* pos, float* x,
                  const float* in_rows, hipStream_t st) {
  hipLaunchKernelGGL(embed_kernel<S>, dim3(M), dim3(256), 0, st, d, rows,
                     (const typename S::T*)tok, (const typename S::T*)pos, x, in_rows);
}
template void launch_embed<F32>(int, int, const RowDesc*, const void*, const void*, float*, const float*, hipStream_t);
template void launch_embed<BF16>(int, int, const RowDesc*, const void*, const void*, float*, const float*, hipStream_t);

template <class S>
void launch_layernorm(int M, int d, const float* x, const void* g, const void* b, float* out,
                      hipStream_t st) {
  hipLaunchKernelGGL(layernorm_kernel<S>, dim3(M), dim3(256), 0, st, d, x,
                     (const typename S::T*)g, (const typename S::T*)b, out);
}
template void launch_layernorm<F32>(int, int, const float*, const void*, const void*, float*, hipStream_t);
template void launch_layernorm<BF16>(int, int, const float*, const void*, const void*, float*, hipStream_t);

template <class S>
void launch_layernorm_frag(int M, int d, const float* x, const void* g, const void* b,
                           uint16_t* frag, int RT, float* out, hipStream_t st) {
  hipLaunchKernelGGL(layernorm_frag_kernel<S>, dim3(M), dim3(256), 0, st, d, x,
                     (const typename S::T*)g, (const typename S::T*)b, frag, RT, out);
}
template void launch_layernorm_frag<BF16>(int, int, const float*, const void*, const void*, uint16_t*, int, float*, hipStream_t);

void launch_reduce_res_ln(int M, int d, int nsplit, const float* P, const void* bias, float* x,
                          const void* g, const void* b, uint16_t* frag, int RT, float* out,
                          hipStream_t st) {
  const int threads = (d / 4 + kWave - 1) / kWave * kWave;
  hipLaunchKernelGGL(reduce_res_ln_kernel, dim3(xcd_row_grid(M)), dim3(threads), 0, st, M, d, nsplit, P,
                     (const uint16_t*)bias, x, (const uint16_t*)g, (const uint16_t*)b, frag, RT, out);
}

void launch_embed_ln(int M, int d, const RowDesc* rows, const void* tok, const void* pos, float* x,
                     const float* in_rows, const void* g, const void* b, uint16_t* frag, int RT,
                     hipStream_t st) {
  const int threads = (d / 4 + kWave - 1) / kWave * kWave;
  hipLaunchKernelGGL(embed_ln_kernel, dim3(xcd_row_grid(M)), dim3(threads), 0, st, M, d, rows,
                     (const uint16_t*)tok, (const uint16_t*)pos, x, in_rows, (const uint16_t*)g,
                     (const uint16_t*)b, frag, RT);
}

// ---------------------------------------------------------------- draft-block inputs

// taps4[b] = [taps_0 ; taps_1 ; taps_2 ; hidden] at sequence b's last verified row (zeros
// for a skipped sequence).
__global__ void draft_gather_taps_kernel(int d, int layout, int k_max, const int* cu_rows,
                                         const int* accept_len, int rows, const float* taps,
                                         const float* hidden, float* taps4) {
  const int b = blockIdx.x;
  const int a = accept_len[b];
  const int row = (layout == 0 ? b * (k_max + 1) : cu_rows[b]) + (a < 0 ? 0 : a);
  for (int j = threadIdx.x; j < 4 * d; j += blockDim.x) {
    const int which = j / d, c = j % d;
    const float* src = which < 3 ? taps + ((size_t)which * rows + row) * d : hidden + (size_t)row * d;
    taps4[(size_t)b * 4 * d + j] = a < 0 ? 0.f : src[c];
  }
}

// z[b] = [feat[b] ; E_tok[token_b]], token_b = tokens[b * token_stride + (token_index ?
// token_index[b] : 0)] (a negative index, i.e. a skipped sequence, reads slot 0).
template <class S>
__global__ void draft_concat_kernel(int d, const float* feat, const typename S::T* tok_emb,
                                    const int* tokens, int token_stride, const int* token_index,
                                    float* z) {
  const int b = blockIdx.x;
  const int ti = token_index ? max(token_index[b], 0) : 0;
  const int t = max(tokens[(size_t)b * token_stride + ti], 0);
  for (int j = threadIdx.x; j < 2 * d; j += blockDim.x)
    z[(size_t)b * 2 * d + j] = j < d ? feat[(size_t)b * d + j] : S::ld(tok_emb, (size_t)t * d + (j - d));
}

// window[b] = [max(0, c - half), min(T_b, c + half + 1)) around anchor c (a negative
// anchor, i.e. a skipped sequence, gives the first frame).
__global__ void draft_window_kernel(int B, const int* anchor, const int* enc_len, int half, int* window) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int c = max(anchor[b], 0), T = max(enc_len[b], 1);
  const int lo = max(0, min(c - half, T - 1));
  window[2 * b] = lo;
  window[2 * b + 1] = max(lo + 1, min(T, c + half + 1));
}

__global__ void draft_gather_taps_frag_kernel(int d, int layout, int k_max, const int* cu_rows,
                                              const int* accept_len, int rows, const float* taps,
                                              const float* hidden, uint16_t* frag, int RT) {
  const int b = blockIdx.x;
  const int a = accept_len[b];
  const int row = (layout == 0 ? b * (k_max + 1) : cu_rows[b]) + (a < 0 ? 0 : a);
  for (int j = threadIdx.x; j < 4 * d; j += blockDim.x) {
    const int which = j / d, c = j % d;
    const float* src = which < 3 ? taps + ((size_t)which * rows + row) * d : hidden + (size_t)row * d;
    afrag_store(frag, RT, b, j, a < 0 ? 0.f : src[c]);
  }
}

__global__ void draft_concat_frag_kernel(int d, const float* feat, const uint16_t* tok_emb,
                                         const int* tokens, int token_stride, const int* token_index,
                                         uint16_t* frag, int RT) {
  const int b = blockIdx.x;
  const int ti = token_index ? max(token_index[b], 0) : 0;
  const int t = max(tokens[(size_t)b * token_stride + ti], 0);
  for (int j = threadIdx.x; j < 2 * d; j += blockDim.x)
    afrag_store(frag, RT, b, j, j < d ? feat[(size_t)b * d + j] : bf16_to_f32(tok_emb[(size_t)t * d + (j - d)]));
}

__global__ void sum_partials_bias_kernel(int M, int N, int nsplit, const float* P,
                                         const uint16_t* bias, float* out) {
  const int m = blockIdx.x;
  for (int j = threadIdx.x * 4; j < N; j += blockDim.x * 4) {
    const size_t e = (size_t)m * N + j;
    float4 v = split_sum4_flat(P, (size_t)M * N, e, nsplit);
    const float4 bb = ld_bf16x4(bias, j);
    v.x += bb.x; v.y += bb.y; v.z += bb.z; v.w += bb.w;
    *(float4*)(out + e) = v;
  }
}

void launch_draft_gather_taps_frag(int B, int d, int layout, int k_max, const int* cu_rows,
                                   const int* accept_len, int rows, const float* taps,
                                   const float* hidden, uint16_t* frag, int RT, hipStream_t st) {
  hipLaunchKernelGGL(draft_gather_taps_frag_kernel, dim3(B), dim3(256), 0, st, d, layout, k_max,
                     cu_rows, accept_len, rows, taps, hidden, frag, RT);
}

void launch_draft_concat_frag(int B, int d, const float* feat, const void* tok_emb,
                              const int* tokens, int token_stride, const int* token_index,
                              uint16_t* frag, int RT, hipStream_t st) {
  hipLaunchKernelGGL(draft_concat_frag_kernel, dim3(B), dim3(256), 0, st, d, feat,
                     (const uint16_t*)tok_emb, tokens, token_stride, token_index, frag, RT);
}

void launch_sum_partials_bias(int M, int N, int nsplit, const float* P, const void* bias, float* out,
                              hipStream_t st) {
  hipLaunchKernelGGL(sum_partials_bias_kernel, dim3(M), dim3(256), 0, st, M, N, nsplit, P,
                     (const uint16_t*)bias, out);
}

void launch_draft_gather_taps(int B, int d, int layout, int k_max, const int* cu_rows,
                              const int* accept_len, int rows, const float* taps,
                              const float* hidden, float* taps4, hipStream_t st) {
  hipLaunchKernelGGL(draft_gather_taps_kernel, dim3(B), dim3(256), 0, st, d, layout, k_max, cu_rows,
                     accept_len, rows, taps, hidden, taps4);
}

void launch_draft_concat(int B, int d, const float* feat, const void* tok_emb, int bf16,
                         const int* tokens, int token_stride, const int* token_index, float* z,
                         hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(draft_concat_kernel<BF16>, dim3(B), dim3(256), 0, st, d, feat,
                       (const uint16_t*)tok_emb, tokens, token_stride, token_index, z);
  else
    hipLaunchKernelGGL(draft_concat_kernel<F32>, dim3(B), dim3(256), 0, st, d, feat,
                       (const float*)tok_emb, tokens, token_stride, token_index, z);
}

void launch_draft_window(int B, const int* anchor, const int* enc_len, int half, int* window,
                         hipStream_t st) {
  hipLaunchKernelGGL(draft_window_kernel, dim3((B + 127) / 128), dim3(128), 0, st, B, anchor,
                     enc_len, half, window);
}

void launch_zero_i32(int* p, int n, hipStream_t st) {
  if (n <= 0) return;
  hipLaunchKernelGGL(zero_i32_kernel, dim3(min((n + 255) / 256, 1024)), dim3(256), 0, st, p, n);
}

void launch_argmax(int M, int V, const float* logits, size_t ld, const RowDesc* rows, int* greedy,
                   float* margin, int* err, hipStream_t st) {
  hipLaunchKernelGGL(argmax_kernel, dim3(M), dim3(256), 0, st, V, logits, ld, rows, greedy, margin, err);
}

void launch_accept(int B, int k_max, const SeqDesc* seqs, const int* tokens, const int* greedy,
                   int* accept_len, int* out_tokens, hipStream_t st) {
  hipLaunchKernelGGL(accept_kernel, dim3((B + 127) / 128), dim3(128), 0, st, B, k_max, seqs, tokens,
                     greedy, accept_len, out_tokens);
}

void launch_accept_tree(int B, int k_max, const SeqDesc* seqs, const int* tokens, const int* parents,
                        const int* greedy, int* accept_len, int* out_tokens, int* out_path,
                        hipStream_t st) {
  hipLaunchKernelGGL(accept_tree_kernel, dim3((B + 127) / 128), dim3(128), 0, st, B, k_max, seqs,
                     tokens, parents, greedy, accept_len, out_tokens, out_path);
}

template <class S>
void launch_kv_compact(int B, int L, int H, const int* kv_len, const int* accept_len, const int* path,
                       int path_stride, void* pool, int num_pages, const int* block_table,
                       int pages_per_seq, hipStream_t st) {
  hipLaunchKernelGGL(kv_compact_kernel<S>, dim3(B, 2 * L), dim3(256), 0, st, H, kv_len, accept_len,
                     path, path_stride, (typename S::T*)pool, num_pages, block_table, pages_per_seq);
}
template void launch_kv_compact<F32>(int, int, int, const int*, const int*, const int*, int, void*, int,
                                     const int*, int, hipStream_t);
template void launch_kv_compact<BF16>(int, int, int, const int*, const int*, const int*, int, void*, int,
                                      const int*, int, hipStream_t);

void launch_commit(int B, int* kv_len, const int* accept_len, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3((B + 127) / 128), dim3(128), 0, st, B, kv_len, accept_len);
}

template <class S>
void launch_kv_copy(bool to_linear, int L, int H, int n, int b, void* lin, void* pool, int num_pages,
                    const int* block_table, int pages_per_seq, int* err, hipStream_t st) {
  const size_t total = (size_t)L * 2 * n * H * kHead;
  if (total == 0) return;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (to_linear)
    hipLaunchKernelGGL((kv_copy_kernel<S, true>), grid, dim3(256), 0, st, L, H, n, b,
                       (typename S::T*)lin, (typename S::T*)pool, num_pages, block_table,
                       pages_per_seq, err);
  else
    hipLaunchKernelGGL((kv_copy_kernel<S, false>), grid, dim3(256), 0, st, L, H, n, b,
                       (typename S::T*)lin, (typename S::T*)pool, num_pages, block_table,
                       pages_per_seq, err);
}
template void launch_kv_copy<F32>(bool, int, int, int, int, void*, void*, int, const int*, int, int*, hipStream_t);
template void launch_kv_copy<BF16>(bool, int, int, int, int, void*, void*, int, const int*, int, int*, hipStream_t);

void launch_gather_hidden(int B, int d, int layout, int k_max, const int* cu_rows,
                          const int* accept_len, const float* hidden, float* hsel, hipStream_t st) {
  hipLaunchKernelGGL(gather_hidden_kernel, dim3(B), dim3(256), 0, st, B, d, layout, k_max, cu_rows,
                     accept_len, hidden, hsel);
}

void launch_assemble_next(int B, int n_heads, int k_max, const int* accept_len, const int* out_tokens,
                          const int* head_greedy, int* next_tokens, hipStream_t st) {
  hipLaunchKernelGGL(assemble_next_kernel, dim3((B + 127) / 128), dim3(128), 0, st, B, n_heads, k_max,
                     accept_len, out_tokens, head_greedy, next_tokens);
}

}  // namespace ad
