// Attention of the block rows on the gfx950 matrix cores (bf16 caches).
//
// One workgroup handles one (sequence, head, group of up to 16 block rows); its waves
// take one chunk of keys each.  The projection before the attention leaves split-K
// partial products; the workgroup finishes them for its head (sum in split order plus
// bias): the queries go to LDS and, for self-attention, the block's keys and values are
// rounded to bf16 and written into the paged cache (write-through; commit only moves
// the cache length).  The waves request their first key blocks before that prologue and
// do not wait for the cache writes: a self-attention block that reaches the block's own
// rows takes their keys and values from an LDS copy instead.
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

// Cross-attention: this lane's first key element of the 32-frame block starting at blk
// (keys and values already in operand order, 1 KB per load; the block's values follow
// its keys).  A block past the chunk is replaced by the chunk's last block, and a chunk
// wholly before a cross-attention window (k_end <= k_beg) reloads its first block, which
// lies inside the sequence's slots.
__device__ __forceinline__ const uint16_t* cross_block(const AttnArgs& a, const SeqDesc& s, int h,
                                                      int blk, int k_beg, int k_end, int c16, int grp) {
  const int b0 = blk < k_end ? blk
                             : (k_end > k_beg ? k_beg + (k_end - 1 - k_beg) / kCrossBlock * kCrossBlock : k_beg);
  const size_t bo = (size_t)((s.enc_off + b0) / kCrossBlock) * 2 * kCrossBlockElems + (grp * 16 + c16) * 8;
  return a.kv + cross_base(a.layer, h, a.H, a.frames_cap) + bo;
}
__device__ __forceinline__ void load_keys(const uint16_t* kp, KVTiles& t) {
  t.k00 = *(const uint4*)(kp + 0 * 512);
  t.k01 = *(const uint4*)(kp + 1 * 512);
  t.k10 = *(const uint4*)(kp + 2 * 512);
  t.k11 = *(const uint4*)(kp + 3 * 512);
}
__device__ __forceinline__ void load_values(const uint16_t* kp, KVTiles& t) {
  const uint16_t* vp = kp + kCrossBlockElems;
  t.v0 = *(const uint4*)(vp + 0 * 512);
  t.v1 = *(const uint4*)(vp + 1 * 512);
  t.v2 = *(const uint4*)(vp + 2 * 512);
  t.v3 = *(const uint4*)(vp + 3 * 512);
}

// Load the 32-key block starting at blk (a multiple of 32 from the chunk start).  A
// 16-key tile past k_end is replaced by the chunk's last tile (valid, and just read, so
// the reload hits the cache), so every lane issues the same unconditional loads.
template <bool CROSS>
__device__ __forceinline__ void load_block(const AttnArgs& a, const SeqDesc& s, int h, int blk,
                                           int k_beg, int k_end, int pg_lane, int c16, int grp,
                                           KVTiles& t) {
  if (CROSS) {
    const uint16_t* kp = cross_block(a, s, h, blk, k_beg, k_end, c16, grp);
    load_keys(kp, t);
    load_values(kp, t);
    return;
  }
  const uint16_t* kb[2];
  const uint16_t* vb[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    int t0 = blk + 16 * u;
    t0 = t0 < k_end ? t0 : k_beg + (k_end - 1 - k_beg) / kTile * kTile;
    const int pg = __shfl(pg_lane, (t0 - k_beg) / kTile, kWave);
    kb[u] = a.kv + kv_tile_base(a.layer, 0, pg, h, a.num_pages, a.H);
    vb[u] = a.kv + kv_tile_base(a.layer, 1, pg, h, a.num_pages, a.H);
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
// reaches past k_end or into the block's own rows; a query sees key `key` when
// k_lo <= key < k_end and either key < n0 (the committed cache) or bit key - n0 of its
// row mask tm is set (its ancestors in the block and itself: the rows before it for a
// chain).  Keys a query must not see get probability 0 and value slots past k_end are
// zeroed (stale or poisoned cache slots never reach the output).  Unmasked blocks skip
// all of that.  Queries past the group (zero rows) are computed but never stored.
// The block's scores (this lane's query, keys 8 grp .. 8 grp + 7), masked keys -inf.
template <bool MASKED, bool SCORES = false>
__device__ __forceinline__ void block_scores(const KVTiles& cur, int blk, int k_lo, int k_end, int n0,
                                             unsigned long long tm, int grp, const bf16x8 (&qh)[2],
                                             const bf16x8 (&ql)[2], float (&sv)[8],
                                             float* srow = nullptr) {
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
      const bool see = key >= k_lo && key < k_end && (key < n0 || ((tm >> ((key - n0) & 63)) & 1));
      sv[tt * 4 + i] = (!MASKED || see) ? st[i] : -INFINITY;
    }
  }
  // the anchor layer keeps every score of its query rows (keys past the sequence hold
  // -inf; the row stride covers whole 32-key blocks; a block past the chunk stores none)
  if (SCORES && srow && blk < k_end) {
    *(float4*)(srow + blk + grp * 8) = float4{sv[0], sv[1], sv[2], sv[3]};
    *(float4*)(srow + blk + grp * 8 + 4) = float4{sv[4], sv[5], sv[6], sv[7]};
  }
}

// The online-softmax update with the block's scores and the value product.
template <bool MASKED>
__device__ __forceinline__ void block_softmax_pv(const KVTiles& cur, const float (&sv)[8], int blk,
                                                 int k_end, int grp, f32x4 (&o)[4], float& m_run,
                                                 float& l_run) {
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

template <bool MASKED, bool SCORES = false>
__device__ __forceinline__ void attend_block(const KVTiles& cur, int blk, int k_lo, int k_end, int n0,
                                             unsigned long long tm, int grp, const bf16x8 (&qh)[2],
                                             const bf16x8 (&ql)[2], f32x4 (&o)[4], float& m_run,
                                             float& l_run, float* srow = nullptr) {
  float sv[8];
  block_scores<MASKED, SCORES>(cur, blk, k_lo, k_end, n0, tm, grp, qh, ql, sv, srow);
  block_softmax_pv<MASKED>(cur, sv, blk, k_end, grp, o, m_run, l_run);
}

// Self-attention: replace the keys / values of the block's own rows (positions n ..
// n + nrows - 1, possibly stale in the loaded tiles) by their LDS copies: nk[r][64]
// (keys, row-major) and nvt[64][kMaxBlockRows] (values, transposed).
__device__ __forceinline__ uint4 patch_values(uint4 v, const uint16_t* row, int r0, int nrows) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = r0 + j;
    const bool in = r >= 0 && r < nrows;
    const uint32_t e = row[in ? r : 0];
    const int sh = (j & 1) * 16;
    const uint32_t upd = (w[j >> 1] & ~(0xffffu << sh)) | (e << sh);
    w[j >> 1] = in ? upd : w[j >> 1];
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ uint4 sel4(bool c, uint4 a, uint4 b) {
  return make_uint4(c ? a.x : b.x, c ? a.y : b.y, c ? a.z : b.z, c ? a.w : b.w);
}
__device__ __forceinline__ KVTiles patch_new_rows(const KVTiles& t, int blk, int n, int nrows,
                                                  const uint16_t* nk, const uint16_t* nvt,
                                                  int c16, int grp) {
  KVTiles u;
  const int r = blk + 8 * (c16 >> 2) + (c16 & 3) - n;    // key row of product 0 (+4: product 1)
  const bool in0 = r >= 0 && r < nrows, in1 = r + 4 >= 0 && r + 4 < nrows;
  const uint4* s0 = (const uint4*)(nk + (in0 ? r : 0) * kHead + grp * 16);
  const uint4* s1 = (const uint4*)(nk + (in1 ? r + 4 : 0) * kHead + grp * 16);
  u.k00 = sel4(in0, s0[0], t.k00);
  u.k01 = sel4(in0, s0[1], t.k01);
  u.k10 = sel4(in1, s1[0], t.k10);
  u.k11 = sel4(in1, s1[1], t.k11);
  const int r0 = blk + 8 * grp - n;
  u.v0 = patch_values(t.v0, nvt + (0 * 16 + c16) * kMaxBlockRows, r0, nrows);
  u.v1 = patch_values(t.v1, nvt + (1 * 16 + c16) * kMaxBlockRows, r0, nrows);
  u.v2 = patch_values(t.v2, nvt + (2 * 16 + c16) * kMaxBlockRows, r0, nrows);
  u.v3 = patch_values(t.v3, nvt + (3 * 16 + c16) * kMaxBlockRows, r0, nrows);
  return u;
}

// Finish four consecutive columns (col % 4 == 0) of the projection of row m: the split
// partials summed in split order, plus the bias.
__device__ __forceinline__ float4 finish_proj4(const AttnArgs& a, int m, int col) {
  float4 v = split_sum4(a.qkv_part, (size_t)a.rows * a.qkv_n, (size_t)m * a.qkv_n + col, a.qkv_splits);
  const uint2 bu = *(const uint2*)(a.qkv_bias + col);
  v.x += bf16_to_f32(bu.x & 0xffff);
  v.y += bf16_to_f32(bu.x >> 16);
  v.z += bf16_to_f32(bu.y & 0xffff);
  v.w += bf16_to_f32(bu.y >> 16);
  return v;
}

template <bool CROSS, bool SCORES, bool PAD = false>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(3)))
attn_mfma_kernel(AttnArgs a) {
  extern __shared__ float part[];  // [waves][kAttnPart], then the queries [16][64]
  const int h = blockIdx.x;
  const int b = blockIdx.y / a.qgroups, qg = blockIdx.y % a.qgroups;
  const int ch = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63, c16 = lane & 15, grp = lane >> 4;
  // self-attention: the page indices of this wave's own chunk (one per lane, lanes past
  // the chunk's tiles repeat its first tile) do not depend on the sequence descriptor,
  // so they are requested beside it
  int pg_spec = 0;
  if (!CROSS) {
    const int tiles = a.chunk / kTile;
    const int p = min(ch * tiles + (lane < tiles ? lane : 0), a.pages_per_seq - 1);
    pg_spec = a.block_table[(size_t)b * a.pages_per_seq + p];
  }
  // Prologue loads: this thread's first query item and (self) its first block-row item,
  // SP split planes each, as straight-line code.  Loads complete in issue order, so
  // waiting for these later leaves the key loads issued after them in flight.
  constexpr int SP = CROSS ? 8 : 4;
  const int S = a.qkv_splits;
  const size_t plane = (size_t)a.rows * a.qkv_n;
  const int qr = threadIdx.x >> 4, qj = (threadIdx.x & 15) * 4;        // query item
  const int kr = threadIdx.x >> 5, kkv = (threadIdx.x >> 4) & 1;       // block-row item
  const int kcol = a.d + kkv * a.d + h * kHead + qj;
  const int q0 = qg * 16;
  float4 qp[SP], kp[SP];
  uint2 qb, kbias;
  size_t qe = 0, ke = 0;
  auto request = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < SP; ++u) qp[u] = *(const float4*)(a.qkv_part + (size_t)min(u, S - 1) * plane + qe);
    qb = *(const uint2*)(a.qkv_bias + h * kHead + qj);
    if (!CROSS) {
#pragma unroll
      for (int u = 0; u < SP; ++u) kp[u] = *(const float4*)(a.qkv_part + (size_t)min(u, S - 1) * plane + ke);
      kbias = *(const uint2*)(a.qkv_bias + kcol);
    }
  };
  if constexpr (PAD) {
    // padded rows: sequence b's rows start at b * row_stride, so the partials are
    // requested before the descriptor arrives (rows clamped to the sequence's own; an
    // item past the block's rows is loaded but never used)
    const int r0 = b * a.row_stride;
    qe = (size_t)(r0 + min(q0 + qr, a.row_stride - 1)) * a.qkv_n + h * kHead + qj;
    ke = (size_t)(r0 + min(kr, a.row_stride - 1)) * a.qkv_n + kcol;
    request();
  }
  const SeqDesc s = a.seqs[b];
  if constexpr (PAD) {
    // keep those requests ahead of the descriptor's use (the early returns below would
    // otherwise let the compiler sink them past it); the fields used here are read
    // before this point, so they stay scalar loads
    asm volatile("" ::"s"(s.row0), "s"(s.k), "s"(s.n), "s"(s.valid) : "memory");
  }
  if (!s.valid) return;
  const int nq = min(16, s.k + 1 - q0);
  if (nq <= 0) return;
  if (SCORES && a.best_clear && h == 0 && qg == 0 && threadIdx.x == 0) a.best_clear[b] = 0;
  // cross-attention sees frames [wlo, whi) (all frames unless a window was given)
  const int n_keys = CROSS ? s.whi : s.n + q0 + nq;
  const int k_lo = CROSS ? s.wlo : 0;
  const int n_chunks = (n_keys + a.chunk - 1) / a.chunk;
  float* Pc = part + ch * kAttnPart;
  float* qs = part + a.max_chunks * kAttnPart;

  const bool active = ch < n_chunks;
  // a cross-attention wave past the last chunk issues the loads of chunk 0 (valid
  // addresses, results unused); a self-attention wave past it issues no key loads
  // the chunk's keys [k_beg, k_end); blocks before the window's first 32-key block are
  // skipped (a chunk wholly before the window streams nothing and merges with weight 0)
  const int k_end = min((active ? ch * a.chunk : 0) + a.chunk, n_keys);
  const int k_beg = max(active ? ch * a.chunk : 0, k_lo / kCrossBlock * kCrossBlock);
  // self-attention: the chunk's page indices, one per lane (lanes past the chunk's last
  // page repeat its first page; only an active wave uses them)
  int pg_lane = 0;
  if (!CROSS) {
    const int npg = (k_end - k_beg + kTile - 1) / kTile;
    pg_lane = min(max(__shfl(pg_spec, lane < npg ? lane : 0, kWave), 0), a.num_pages - 1);
  }
  uint16_t* nk = (uint16_t*)(qs + 16 * kHead);   // self: the block rows' keys and values
  uint16_t* nvt = nk + kMaxBlockRows * kHead;
  const int nrows = s.k + 1;

  const bool q_on = threadIdx.x < 16 * 16 && qr < nq;
  const bool k_on = !CROSS && (int)threadIdx.x < nrows * 32;
  if constexpr (!PAD) {
    qe = (size_t)(s.row0 + q0 + (q_on ? qr : 0)) * a.qkv_n + h * kHead + qj;
    ke = (size_t)(s.row0 + (k_on ? kr : 0)) * a.qkv_n + kcol;
    request();
  }
  int kpg = 0;   // page of this thread's block-row item
  unsigned long long tmask = 0;   // self: the row mask of this lane's query
  if (!CROSS) {
    const int slot = s.n + (k_on ? kr : 0);
    kpg = a.block_table[(size_t)b * a.pages_per_seq + slot / kTile];
    tmask = a.tree[s.row0 + q0 + min(c16, nq - 1)].mask;
  }
  // keep the key loads below after the prologue loads (issue order is completion order)
  asm volatile("" ::: "memory");
  // the first two key blocks
  KVTiles ta, tb;
  if (CROSS || active) {
    load_block<CROSS>(a, s, h, k_beg, k_beg, k_end, pg_lane, c16, grp, ta);
    load_block<CROSS>(a, s, h, k_beg + 32, k_beg, k_end, pg_lane, c16, grp, tb);
  }
  // split sum in split order (planes past SP, if any, in a loop), plus the bias
  auto finish = [&](const float4 (&pp)[SP], uint2 bu, size_t e) -> float4 {
    // planes past S add -0, which leaves every value (signed zeros included) unchanged;
    // no branch, so the loads above stay unconditional
    float4 v = pp[0];
#pragma unroll
    for (int u = 1; u < SP; ++u) {
      const bool in = u < S;
      v.x += in ? pp[u].x : -0.f;
      v.y += in ? pp[u].y : -0.f;
      v.z += in ? pp[u].z : -0.f;
      v.w += in ? pp[u].w : -0.f;
    }
    for (int t = SP; t < S; ++t) {
      const float4 w = *(const float4*)(a.qkv_part + (size_t)t * plane + e);
      v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    v.x += bf16_to_f32(bu.x & 0xffff);
    v.y += bf16_to_f32(bu.x >> 16);
    v.z += bf16_to_f32(bu.y & 0xffff);
    v.w += bf16_to_f32(bu.y >> 16);
    return v;
  };
  // the block rows' keys and values: into the cache (bf16) and the LDS copy
  auto put_kv = [&](int r, int kv, int j, int pg, float4 v) {
    const int slot = s.n + r;   // block row r's cache slot (its position for a chain)
    uint16_t* dst = (uint16_t*)a.kv + kv_tile_base(a.layer, kv, pg, h, a.num_pages, a.H);
    const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint16_t e = f32_to_bf16(vv[u]);
      dst[tile_off(kv, slot % kTile, j + u)] = e;
      if (kv == 0) nk[r * kHead + j + u] = e;
      else nvt[(j + u) * kMaxBlockRows + r] = e;
    }
  };

  // finish the projection: this head's queries of the group, and (self-attention) the
  // keys / values of every block row of the sequence
  // (the anchor readout keeps this layer's finished queries: q_save)
  {
    const float4 qv = finish(qp, qb, qe);
    if (threadIdx.x < 16 * 16) *(float4*)(qs + qr * kHead + qj) = q_on ? qv : float4{0.f, 0.f, 0.f, 0.f};
    if (CROSS && a.q_save && q_on) *(float4*)(a.q_save + (size_t)(s.row0 + q0 + qr) * a.d + h * kHead + qj) = qv;
  }
  for (int idx = threadIdx.x + blockDim.x; idx < 16 * 16; idx += blockDim.x) {   // small blocks
    const int r = idx >> 4, j = (idx & 15) * 4;
    const float4 v = r < nq ? finish_proj4(a, s.row0 + q0 + r, h * kHead + j) : float4{0.f, 0.f, 0.f, 0.f};
    *(float4*)(qs + r * kHead + j) = v;
    if (CROSS && a.q_save && r < nq) *(float4*)(a.q_save + (size_t)(s.row0 + q0 + r) * a.d + h * kHead + j) = v;
  }
  if (!CROSS) {
    const float4 kv4 = finish(kp, kbias, ke);
    if (k_on) put_kv(kr, kkv, qj, min(max(kpg, 0), a.num_pages - 1), kv4);
    for (int idx = threadIdx.x + blockDim.x; idx < nrows * 32; idx += blockDim.x) {
      const int r = idx >> 5, kv = (idx >> 4) & 1, j = (idx & 15) * 4;
      const int slot = s.n + r;
      const int pg = min(max(a.block_table[(size_t)b * a.pages_per_seq + slot / kTile], 0), a.num_pages - 1);
      put_kv(r, kv, j, pg, finish_proj4(a, s.row0 + r, a.d + kv * a.d + h * kHead + j));
    }
  }
  // LDS-only barrier: the key loads above and the cache writes stay in flight
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  if (active) {
    // committed keys all visible; the block's rows through the lane's row mask
    const int n0 = CROSS ? s.T : s.n;
    // the anchor layer: this lane's query row's scores (rows past the group store none)
    float* srow = (SCORES && c16 < nq) ? a.score_out + ((size_t)(s.row0 + q0 + c16) * a.H + h) * a.score_ld
                                       : nullptr;
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

    // ping-pong over 32-key blocks with the other block's loads in flight; only blocks
    // that start inside the chunk are processed (one past its end would be fully masked
    // and leave the state bit-for-bit unchanged)
    {
      // blocks below `clean` need no masking for any query of the group and (self)
      // hold committed keys only
      const int clean = CROSS ? k_end : min(k_end, s.n);
      if constexpr (CROSS) {
        // a block's key registers are free once its scores are in: the keys of the block
        // two ahead are requested then, and its values after the value product, so more
        // bytes stay in flight while the softmax runs
        // (pf: request the block two ahead; the last two blocks of the chunk request none)
        auto step = [&](KVTiles& t, int blk, bool pf) __attribute__((always_inline)) {
          const uint16_t* np = cross_block(a, s, h, blk + 64, k_beg, k_end, c16, grp);
          float sv[8];
          if (blk + 32 <= clean && blk >= k_lo) {
            block_scores<false, SCORES>(t, blk, k_lo, k_end, n0, tmask, grp, qh, ql, sv, srow);
            if (pf) load_keys(np, t);
            block_softmax_pv<false>(t, sv, blk, k_end, grp, o, m_run, l_run);
          } else {
            block_scores<true, SCORES>(t, blk, k_lo, k_end, n0, tmask, grp, qh, ql, sv, srow);
            if (pf) load_keys(np, t);
            block_softmax_pv<true>(t, sv, blk, k_end, grp, o, m_run, l_run);
          }
          if (pf) load_values(np, t);
        };
        int blk = k_beg;
        for (; blk + 96 < k_end; blk += 64) {
          step(ta, blk, true);
          step(tb, blk + 32, true);
        }
        // one to three blocks left (none for a chunk wholly before the window), the first
        // two already in ta, tb
        if (blk + 64 < k_end) {
          step(ta, blk, true);
          step(tb, blk + 32, false);
          step(ta, blk + 64, false);
        } else if (blk < k_end) {
          step(ta, blk, false);
          if (blk + 32 < k_end) step(tb, blk + 32, false);
        }
      } else {
        auto attend = [&](const KVTiles& t, int blk) __attribute__((always_inline)) {
          if (blk + 32 <= clean && blk >= k_lo)
            attend_block<false>(t, blk, k_lo, k_end, n0, tmask, grp, qh, ql, o, m_run, l_run);
          else
            attend_block<true>(patch_new_rows(t, blk, s.n, nrows, nk, nvt, c16, grp), blk, k_lo, k_end,
                               n0, tmask, grp, qh, ql, o, m_run, l_run);
        };
        // no block past the chunk is requested (cross-attention likewise): a load whose
        // result is never used still has to land before its registers are reused, a full
        // round trip at the end
        int blk = k_beg;
        for (; blk + 96 < k_end; blk += 64) {
          attend(ta, blk);
          load_block<CROSS>(a, s, h, blk + 64, k_beg, k_end, pg_lane, c16, grp, ta);
          attend(tb, blk + 32);
          load_block<CROSS>(a, s, h, blk + 96, k_beg, k_end, pg_lane, c16, grp, tb);
        }
        // one to three blocks left, the first two already in ta, tb
        attend(ta, blk);
        if (blk + 64 < k_end) {
          load_block<CROSS>(a, s, h, blk + 64, k_beg, k_end, pg_lane, c16, grp, ta);
          attend(tb, blk + 32);
          attend(ta, blk + 64);
        } else if (blk + 32 < k_end) {
          attend(tb, blk + 32);
        }
      }
    }
    if (grp == 0) {
      Pc[c16] = m_run;
      Pc[16 + c16] = l_run;
    }
    // O row c16 (query), dims 16 dt + 4 grp .. + 3: one 16-byte LDS write each
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      *(float4*)(Pc + 32 + c16 * kAttnORow + dt * 16 + grp * 4) = float4{o[dt][0], o[dt][1], o[dt][2], o[dt][3]};
  }
  // LDS-only barrier (the cache writes need not have landed)
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // merge the chunks in chunk order: four consecutive dims d4 .. d4 + 3 of query qq per
  // thread (every output's sums run in the same order as one output per thread)
  for (int idx = threadIdx.x; idx < 16 * 16; idx += blockDim.x) {
    const int qq = idx & 15, d4 = (idx >> 4) * 4;
    if (qq >= nq) continue;
    float M = -INFINITY;
    for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, part[c * kAttnPart + qq]);
    float L = 0.f;
    float4 acc{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < n_chunks; ++c) {
      const float* Q = part + c * kAttnPart;
      const float mc = Q[qq];
      const float wgt = (mc == -INFINITY) ? 0.f : __expf(mc - M);
      L += wgt * Q[16 + qq];
      const float4 ov = *(const float4*)(Q + 32 + qq * kAttnORow + d4);
      acc.x += wgt * ov.x;
      acc.y += wgt * ov.y;
      acc.z += wgt * ov.z;
      acc.w += wgt * ov.w;
    }
    afrag_store4(a.out, a.out_RT, s.row0 + q0 + qq, h * kHead + d4,
                 float4{acc.x / L, acc.y / L, acc.z / L, acc.w / L});
    if (SCORES && d4 == 0) a.stat_out[(size_t)(s.row0 + q0 + qq) * a.H + h] = float2{M, L};
  }
}

void launch_attn_mfma(const AttnArgs& a, int B, hipStream_t st) {
  const dim3 grid(a.H, B * a.qgroups), block(64 * a.max_chunks);
  const size_t lds = ((size_t)a.max_chunks * kAttnPart + 16 * kHead) * sizeof(float) +
                     (a.cross ? 0 : 2 * kMaxBlockRows * kHead * sizeof(uint16_t));
  if (a.cross && a.score_out) hipLaunchKernelGGL((attn_mfma_kernel<true, true>), grid, block, lds, st, a);
  else if (a.cross) hipLaunchKernelGGL((attn_mfma_kernel<true, false>), grid, block, lds, st, a);
  else if (a.row_stride > 0) hipLaunchKernelGGL((attn_mfma_kernel<false, false, true>), grid, block, lds, st, a);
  else hipLaunchKernelGGL((attn_mfma_kernel<false, false>), grid, block, lds, st, a);
}

}  // namespace ad
