// Attention of the block rows on the gfx950 matrix cores (bf16 caches).
//
// One workgroup handles one (sequence, head, group of up to 16 block rows); its waves
// take one chunk of keys each.  The projection before the attention leaves split-K
// partial products; the workgroup finishes them for its head (sum in split order plus
// bias): the queries go to LDS and, for self-attention, the block's keys and values are
// rounded to bf16 and written into the paged cache (write-through; commit only moves
// the cache length) before any wave reads the cache.
// Scores are computed transposed, S^T = K Q^T (keys on the 16 MFMA rows, queries on the
// 16 columns), so every lane holds scores of a single query: the online softmax needs
// only two cross-lane steps and the probabilities are already in the operand order of
// O^T = V^T P^T.  Queries and probabilities enter the products as hi/lo bf16 pairs.
//
// Keys are cut into fixed chunks at absolute positions 0, chunk, 2 chunk, ...; each chunk
// keeps (max, sum, unnormalised output) per query in LDS and the workgroup merges them in
// chunk order.  A key a query must not see (past its causal limit or past the
// sequence) gets probability 0, and value slots past the sequence are zeroed before
// the product, so stale or poisoned cache slots never reach the output.
#include "common.h"
#include "launch.h"

namespace ad {

__device__ __forceinline__ uint32_t pack2(uint16_t a, uint16_t b) {
  return (uint32_t)a | ((uint32_t)b << 16);
}

// eight float32 values -> (hi, lo) bf16x8 operands
__device__ __forceinline__ void split8(const float* v, bf16x8& hi, bf16x8& lo) {
  uint16_t h[8], l[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) split_hilo(v[j], h[j], l[j]);
  hi = as_bf16x8(make_uint4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7])));
  lo = as_bf16x8(make_uint4(pack2(l[0], l[1]), pack2(l[2], l[3]), pack2(l[4], l[5]), pack2(l[6], l[7])));
}

// keep the first n_keep (clamped to 0..4) bf16 elements of an 8-byte value, zero the rest
// (selects, no branches: loads stay in flight)
__device__ __forceinline__ uint2 mask4(uint2 v, int n_keep) {
  const uint32_t m0 = (n_keep >= 1 ? 0x0000ffffu : 0u) | (n_keep >= 2 ? 0xffff0000u : 0u);
  const uint32_t m1 = (n_keep >= 3 ? 0x0000ffffu : 0u) | (n_keep >= 4 ? 0xffff0000u : 0u);
  return make_uint2(v.x & m0, v.y & m1);
}

// One 32-key block in registers: for each 16-key tile its two key halves (this lane's 16
// lanes of key row c16), and for each 16-lane value tile dt the operand
// (tile-0 tokens 4 grp .. +3 | tile-1 tokens 4 grp .. +3) of value lane 16 dt + c16.
struct KVTiles {
  uint4 k00, k01, k10, k11;
  uint4 v0, v1, v2, v3;
};

// Load the two 16-key tiles of the 32-key block starting at blk.  Tiles past k_end are
// replaced by the chunk's first tile (always valid) and their values zeroed, so every
// lane issues the same unconditional loads.
template <bool CROSS>
__device__ __forceinline__ void load_tile(const AttnArgs& a, const SeqDesc& s, int h, int t0,
                                          int k_beg, int k_end, int pg_lane, int c16, int grp,
                                          uint4& k0, uint4& k1, uint2 (&v)[4]) {
  const int keep = k_end - (t0 + grp * 4);
  t0 = t0 < k_end ? t0 : k_beg;
  const uint16_t* kb;
  const uint16_t* vb;
  if (CROSS) {
    const size_t tile = (size_t)((s.enc_off + t0) / kTile) * kTileElems;
    kb = a.kv + cross_base(a.layer, 0, h, a.H, a.frames_cap) + tile;
    vb = a.kv + cross_base(a.layer, 1, h, a.H, a.frames_cap) + tile;
  } else {
    const int pg = __shfl(pg_lane, (t0 - k_beg) / kTile, kWave);
    kb = a.kv + kv_tile_base(a.layer, 0, pg, h, a.num_pages, a.H);
    vb = a.kv + kv_tile_base(a.layer, 1, pg, h, a.num_pages, a.H);
  }
  const uint16_t* kp = kb + c16 * kHead + grp * 16;
  k0 = *(const uint4*)kp;
  k1 = *(const uint4*)(kp + 8);
  const uint16_t* vp = vb + grp * 4;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) v[dt] = mask4(*(const uint2*)(vp + (dt * 16 + c16) * kTile), keep);
}

// Load the two 16-key tiles of the 32-key block starting at blk.  Tiles past k_end are
// replaced by the chunk's first tile (always valid) and their values zeroed, so every
// lane issues the same unconditional loads.
template <bool CROSS>
__device__ __forceinline__ void load_block(const AttnArgs& a, const SeqDesc& s, int h, int blk,
                                           int k_beg, int k_end, int pg_lane, int c16, int grp,
                                           KVTiles& t) {
  uint2 va[4], vb[4];
  load_tile<CROSS>(a, s, h, blk, k_beg, k_end, pg_lane, c16, grp, t.k00, t.k01, va);
  load_tile<CROSS>(a, s, h, blk + 16, k_beg, k_end, pg_lane, c16, grp, t.k10, t.k11, vb);
  t.v0 = make_uint4(va[0].x, va[0].y, vb[0].x, vb[0].y);
  t.v1 = make_uint4(va[1].x, va[1].y, vb[1].x, vb[1].y);
  t.v2 = make_uint4(va[2].x, va[2].y, vb[2].x, vb[2].y);
  t.v3 = make_uint4(va[3].x, va[3].y, vb[3].x, vb[3].y);
}

// One 32-key block of the online softmax and the two products.
__device__ __forceinline__ void attend_block(const KVTiles& cur, int blk, int k_end, int vis,
                                             bool qvalid, int grp, const bf16x8 (&qh)[2],
                                             const bf16x8 (&ql)[2], f32x4 (&o)[4], float& m_run,
                                             float& l_run) {
  float sv[8];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 k0 = as_bf16x8(tt ? cur.k10 : cur.k00), k1 = as_bf16x8(tt ? cur.k11 : cur.k01);
    st = mfma_bf16(k0, qh[0], st);
    st = mfma_bf16(k1, qh[1], st);
    st = mfma_bf16(k0, ql[0], st);
    st = mfma_bf16(k1, ql[1], st);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = blk + tt * 16 + grp * 4 + i;
      sv[tt * 4 + i] = (qvalid && key < k_end && key < vis) ? st[i] : -INFINITY;
    }
  }
  float bm = sv[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) bm = fmaxf(bm, sv[j]);
  bm = fmaxf(bm, __shfl_xor(bm, 16, kWave));
  bm = fmaxf(bm, __shfl_xor(bm, 32, kWave));
  const float m_new = fmaxf(m_run, bm);
  const float scale = (m_new == -INFINITY) ? 1.f : __expf(m_run - m_new);
  float p[8], ps = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    p[j] = (sv[j] == -INFINITY) ? 0.f : __expf(sv[j] - m_new);
    ps += p[j];
  }
  ps += __shfl_xor(ps, 16, kWave);
  ps += __shfl_xor(ps, 32, kWave);
  l_run = l_run * scale + ps;
  m_run = m_new;
  bf16x8 ph, pl;
  split8(p, ph, pl);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    o[dt] *= scale;
    const bf16x8 vt = as_bf16x8(dt == 0 ? cur.v0 : (dt == 1 ? cur.v1 : (dt == 2 ? cur.v2 : cur.v3)));
    o[dt] = mfma_bf16(vt, ph, o[dt]);
    o[dt] = mfma_bf16(vt, pl, o[dt]);
  }
}

__device__ __forceinline__ float finish_proj(const AttnArgs& a, int m, int col) {
  const size_t plane = (size_t)a.rows * a.qkv_n, e = (size_t)m * a.qkv_n + col;
  float v = a.qkv_part[e];
  for (int t = 1; t < a.qkv_splits; ++t) v += a.qkv_part[t * plane + e];
  return v + bf16_to_f32(a.qkv_bias[col]);
}

template <bool CROSS>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(1, 2)))
attn_mfma_kernel(AttnArgs a) {
  extern __shared__ float part[];  // [waves][kAttnPart], then the queries [16][64]
  const int h = blockIdx.x;
  const int b = blockIdx.y / a.qgroups, qg = blockIdx.y % a.qgroups;
  const SeqDesc s = a.seqs[b];
  if (!s.valid) return;
  const int q0 = qg * 16;
  const int nq = min(16, s.k + 1 - q0);
  if (nq <= 0) return;
  const int n_keys = CROSS ? s.T : s.n + q0 + nq;
  const int n_chunks = (n_keys + a.chunk - 1) / a.chunk;
  const int ch = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63, c16 = lane & 15, grp = lane >> 4;
  const bool qvalid = c16 < nq;
  float* Pc = part + ch * kAttnPart;
  float* qs = part + a.max_chunks * kAttnPart;

  // finish the projection: this head's queries of the group, and (self-attention) the
  // keys / values of every block row of the sequence into the cache
  for (int idx = threadIdx.x; idx < 16 * kHead; idx += blockDim.x) {
    const int r = idx >> 6, j = idx & 63;
    qs[idx] = r < nq ? finish_proj(a, s.row0 + q0 + r, h * kHead + j) : 0.f;
  }
  if (!CROSS) {
    for (int idx = threadIdx.x; idx < (s.k + 1) * 2 * kHead; idx += blockDim.x) {
      const int r = idx >> 7, kv = (idx >> 6) & 1, j = idx & 63;
      const float v = finish_proj(a, s.row0 + r, a.d + kv * a.d + h * kHead + j);
      const int pos = s.n + r;
      int pg = a.block_table[(size_t)b * a.pages_per_seq + pos / kTile];
      pg = min(max(pg, 0), a.num_pages - 1);
      ((uint16_t*)a.kv)[kv_tile_base(a.layer, kv, pg, h, a.num_pages, a.H) + tile_off(kv, pos % kTile, j)] =
          f32_to_bf16(v);
    }
  }
  __syncthreads();

  if (ch < n_chunks) {
    const int k_beg = ch * a.chunk, k_end = min(k_beg + a.chunk, n_keys);
    const int vis = CROSS ? s.T : s.n + q0 + c16 + 1;
    // self-attention: the chunk's page indices, one per lane (lanes past the chunk
    // repeat its first page)
    int pg_lane = 0;
    if (!CROSS) {
      const int npg = (k_end - k_beg + kTile - 1) / kTile;
      const int p = k_beg / kTile + (lane < npg ? lane : 0);
      pg_lane = min(max(a.block_table[(size_t)b * a.pages_per_seq + p], 0), a.num_pages - 1);
    }

    // Q^T operand: query c16, dims 16 grp + 8 hh + j, scaled by 1/8 (exact)
    bf16x8 qh[2], ql[2];
    {
      float v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] = qs[c16 * kHead + grp * 16 + j] * 0.125f;
      split8(v, qh[0], ql[0]);
      split8(v + 8, qh[1], ql[1]);
    }

    f32x4 o[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    // ping-pong over 32-key blocks; a block past the chunk end is fully masked and
    // leaves the state bit-for-bit unchanged
    KVTiles ta, tb;
    load_block<CROSS>(a, s, h, k_beg, k_beg, k_end, pg_lane, c16, grp, ta);
    for (int blk = k_beg; blk < k_end; blk += 64) {
      load_block<CROSS>(a, s, h, blk + 32, k_beg, k_end, pg_lane, c16, grp, tb);
      attend_block(ta, blk, k_end, vis, qvalid, grp, qh, ql, o, m_run, l_run);
      load_block<CROSS>(a, s, h, blk + 64, k_beg, k_end, pg_lane, c16, grp, ta);
      attend_block(tb, blk + 32, k_end, vis, qvalid, grp, qh, ql, o, m_run, l_run);
    }
    if (grp == 0) {
      Pc[c16] = m_run;
      Pc[16 + c16] = l_run;
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) Pc[32 + (dt * 16 + grp * 4 + i) * 16 + c16] = o[dt][i];
  }
  __syncthreads();

  // merge the chunks in chunk order: output (query qq, dim dd) per thread
  for (int idx = threadIdx.x; idx < 16 * 64; idx += blockDim.x) {
    const int qq = idx & 15, dd = idx >> 4;
    if (qq >= nq) continue;
    float M = -INFINITY;
    for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, part[c * kAttnPart + qq]);
    float L = 0.f, acc = 0.f;
    for (int c = 0; c < n_chunks; ++c) {
      const float* Q = part + c * kAttnPart;
      const float mc = Q[qq];
      const float wgt = (mc == -INFINITY) ? 0.f : __expf(mc - M);
      L += wgt * Q[16 + qq];
      acc += wgt * Q[32 + dd * 16 + qq];
    }
    afrag_store(a.out, a.out_RT, s.row0 + q0 + qq, h * kHead + dd, acc / L);
  }
}

void launch_attn_mfma(const AttnArgs& a, int B, hipStream_t st) {
  const dim3 grid(a.H, B * a.qgroups), block(64 * a.max_chunks);
  const size_t lds = ((size_t)a.max_chunks * kAttnPart + 16 * kHead) * sizeof(float);
  if (a.cross) hipLaunchKernelGGL(attn_mfma_kernel<true>, grid, block, lds, st, a);
  else hipLaunchKernelGGL(attn_mfma_kernel<false>, grid, block, lds, st, a);
}

}  // namespace ad
