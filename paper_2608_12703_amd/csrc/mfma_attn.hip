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

// eight float32 values -> (hi, lo) bf16x8 operands (paired hardware conversions)
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

// keep the first n_keep (clamped to 0..8) bf16 elements of a 16-byte value, zero the
// rest (selects, no branches: loads stay in flight)
__device__ __forceinline__ uint4 mask8(uint4 v, int n_keep) {
  auto m = [&](int lo) -> uint32_t {
    return (n_keep > lo ? 0x0000ffffu : 0u) | (n_keep > lo + 1 ? 0xffff0000u : 0u);
  };
  return make_uint4(v.x & m(0), v.y & m(2), v.z & m(4), v.w & m(6));
}

// One 32-key block in registers.  Key rows of the score products are interleaved: in
// product tt, MFMA row r holds key 8 (r / 4) + 4 tt + r % 4, so after both products
// the lanes of group g hold the scores of keys 8 g .. 8 g + 7, which is exactly the key
// range the same lanes supply to the value product.  kt0 / kt1: this lane's key row of
// product tt (two 16-byte halves each); v[dt]: keys 8 g .. 8 g + 7 of value lane
// 16 dt + c16 (one 16-byte load from a lane-major tile).
struct KVTiles {
  uint4 k00, k01, k10, k11;
  uint4 v0, v1, v2, v3;
};

// Load the 32-key block starting at blk (a multiple of 32 from the chunk start).  A
// 16-key tile past k_end is replaced by the chunk's last tile (valid, and just read, so
// the reload hits the cache), so every lane issues the same unconditional loads.
template <bool CROSS>
__device__ __forceinline__ void load_block(const AttnArgs& a, const SeqDesc& s, int h, int blk,
                                           int k_beg, int k_end, int pg_lane, int c16, int grp,
                                           KVTiles& t) {
  const uint16_t* kb[2];
  const uint16_t* vb[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    int t0 = blk + 16 * u;
    t0 = t0 < k_end ? t0 : k_beg + (k_end - 1 - k_beg) / kTile * kTile;
    if (CROSS) {
      const size_t tile = (size_t)((s.enc_off + t0) / kTile) * kTileElems;
      kb[u] = a.kv + cross_base(a.layer, 0, h, a.H, a.frames_cap) + tile;
      vb[u] = a.kv + cross_base(a.layer, 1, h, a.H, a.frames_cap) + tile;
    } else {
      const int pg = __shfl(pg_lane, (t0 - k_beg) / kTile, kWave);
      kb[u] = a.kv + kv_tile_base(a.layer, 0, pg, h, a.num_pages, a.H);
      vb[u] = a.kv + kv_tile_base(a.layer, 1, pg, h, a.num_pages, a.H);
    }
  }
  // key rows: lane c16 of product tt reads key 8 (c16 / 4) + 4 tt + c16 % 4, i.e. tile
  // c16 / 8, token 8 ((c16 / 4) % 2) + 4 tt + c16 % 4; lane group grp reads dims
  // 16 grp .. 16 grp + 15 of it (the queries use the same dim order)
  const uint16_t* kt = (c16 < 8 ? kb[0] : kb[1]) + (((c16 >> 2) & 1) * 8 + (c16 & 3)) * kHead + grp * 16;
  t.k00 = *(const uint4*)kt;
  t.k01 = *(const uint4*)(kt + 8);
  t.k10 = *(const uint4*)(kt + 4 * kHead);
  t.k11 = *(const uint4*)(kt + 4 * kHead + 8);
  // values: keys 8 grp .. 8 grp + 7 = tile grp / 2, tokens 8 (grp % 2) .. + 7 (slots past
  // the sequence are zeroed where the block is used)
  const uint16_t* vt = (grp < 2 ? vb[0] : vb[1]) + (grp & 1) * 8 + c16 * kTile;
  t.v0 = *(const uint4*)(vt + 0 * 16 * kTile);
  t.v1 = *(const uint4*)(vt + 1 * 16 * kTile);
  t.v2 = *(const uint4*)(vt + 2 * 16 * kTile);
  t.v3 = *(const uint4*)(vt + 3 * 16 * kTile);
}

// One 32-key block of the online softmax and the two products.  MASKED: the block
// reaches past k_end or past some query's causal limit; keys a query must not see get
// probability 0 and value slots past k_end are zeroed (stale or poisoned cache slots
// never reach the output).  Unmasked blocks skip all of that.  Queries past the group
// (zero rows) are computed but never stored.
template <bool MASKED>
__device__ __forceinline__ void attend_block(const KVTiles& cur, int blk, int k_end, int vis,
                                             int grp, const bf16x8 (&qh)[2],
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
      const int key = blk + grp * 8 + tt * 4 + i;
      sv[tt * 4 + i] = (!MASKED || (key < k_end && key < vis)) ? st[i] : -INFINITY;
    }
  }
  const float bm = rows4_max(fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                                   fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7]))));
  const float m_new = fmaxf(m_run, bm);
  // m_run = -inf (first block) gives scale 0; only a fully masked history can leave
  // m_new = -inf, and then nothing changes
  const float scale = (MASKED && m_new == -INFINITY) ? 1.f : __expf(m_run - m_new);
  float p[8], ps = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    p[j] = (MASKED && sv[j] == -INFINITY) ? 0.f : __expf(sv[j] - m_new);
    ps += p[j];
  }
  ps = rows4_sum(ps);
  l_run = l_run * scale + ps;
  m_run = m_new;
  bf16x8 ph, pl;
  split8(p, ph, pl);
  const int keep = k_end - (blk + 8 * grp);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    o[dt] *= scale;
    uint4 vr = dt == 0 ? cur.v0 : (dt == 1 ? cur.v1 : (dt == 2 ? cur.v2 : cur.v3));
    if (MASKED) vr = mask8(vr, keep);
    const bf16x8 vt = as_bf16x8(vr);
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
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(3)))
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
    {
      KVTiles ta, tb;
      load_block<CROSS>(a, s, h, k_beg, k_beg, k_end, pg_lane, c16, grp, ta);
      // blocks below `clean` need no masking for any query of the group
      const int clean = CROSS ? k_end : min(k_end, s.n + q0 + 1);
      auto attend = [&](const KVTiles& t, int blk) {
        if (blk + 32 <= clean) attend_block<false>(t, blk, k_end, vis, grp, qh, ql, o, m_run, l_run);
        else attend_block<true>(t, blk, k_end, vis, grp, qh, ql, o, m_run, l_run);
      };
      for (int blk = k_beg; blk < k_end; blk += 64) {
        load_block<CROSS>(a, s, h, blk + 32, k_beg, k_end, pg_lane, c16, grp, tb);
        attend(ta, blk);
        load_block<CROSS>(a, s, h, blk + 64, k_beg, k_end, pg_lane, c16, grp, ta);
        attend(tb, blk + 32);
      }
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
