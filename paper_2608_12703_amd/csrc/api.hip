// C-ABI entry points of libad.so: argument validation, workspace layout and the order
// of kernel launches that makes one verify step.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ad.h"
#include "common.h"
#include "launch.h"

struct ad_model {
  ad_model_desc desc;
  std::vector<const void*> p;
  const uint16_t* packed = nullptr;   // tiled weights (ad_model_pack), or NULL
  std::vector<size_t> pack_off;       // their element offsets (packed_offsets)
  // launch timing (ad_profile_enable / ad_profile_read)
  int prof_kernel = 0;
  std::vector<hipEvent_t> prof_start, prof_stop;
  int prof_used = 0;
};

namespace {

thread_local std::string g_err = "";

ad_status fail(ad_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

enum GlobalParam { P_TOK = 0, P_POS = 1, P_LNF_G = 2, P_LNF_B = 3 };
enum LayerParam {
  LN1_G, LN1_B, W_QKV, B_QKV, W_O, B_O, LN2_G, LN2_B, W_XQ, B_XQ, W_XKV, B_XKV, W_XO, B_XO,
  LN3_G, LN3_B, W_1, B_1, W_2, B_2, N_LAYER_PARAMS
};

const void* lp(const ad_model* m, int layer, int which) {
  return m->p[4 + layer * N_LAYER_PARAMS + which];
}

// Tiled-weight buffer: per layer W_QKV, W_O, W_XQ, W_XO, W_1, W_2 and the encoder K/V
// projection W_XKV (read by the prefill), then the LM head.
constexpr int kPackedPerLayer = 7;
const int kPackedWhich[kPackedPerLayer] = {W_QKV, W_O, W_XQ, W_XO, W_1, W_2, W_XKV};
constexpr int kPackedXkv = 6;   // slot of W_XKV

void packed_shape(const ad_model_desc& D, int which, int& N, int& K) {
  const int d = D.d_model, F = D.d_ffn;
  N = d; K = d;
  if (which == W_QKV) N = 3 * d;
  if (which == W_XKV) N = 2 * d;
  if (which == W_1) N = F;
  if (which == W_2) K = F;
}

// element offsets of every tiled matrix (index layer * 6 + slot; the LM head last)
std::vector<size_t> packed_offsets(const ad_model_desc& D) {
  std::vector<size_t> off;
  size_t o = 0;
  for (int l = 0; l < D.n_layers; ++l)
    for (int j = 0; j < kPackedPerLayer; ++j) {
      int N, K;
      packed_shape(D, kPackedWhich[j], N, K);
      off.push_back(o);
      o += (ad::packed_weight_elems(N, K) + 127) / 128 * 128;   // 256-byte aligned
    }
  off.push_back(o);
  o += (ad::packed_weight_elems(D.vocab, D.d_model) + 127) / 128 * 128;
  off.push_back(o);   // total
  return off;
}

// Workspace carve-up for a step with M rows and B sequences.
struct Workspace {
  ad::SeqDesc* seqs;
  ad::RowDesc* rows;
  ad::RowTree* tree;   // [M] depth and ancestor mask of every block row
  float* x;        // residual stream [M][d]
  float* ln;       // float32 path: LayerNorm output [M][d]
  float* q;        // queries [M][d]
  float* att;      // float32 path: attention output [M][d]
  float* hid;      // float32 path: GELU output [M][F]
  float* apart;    // float32 path: attention partials per key group
  int gself, gcross;   // float32 path: key groups of self- and cross-attention
  float* hidden;   // final LayerNorm output [M][d]
  float* logits;   // float32 path: [M][V]
  int* greedy;     // [M]
  uint16_t* afrag; // bf16 path: d-wide product operand, A-fragment order
  uint16_t* hfrag; // bf16 path: F-wide product operand (GELU output)
  float* gpart;    // bf16 path: split-K partial products
  void* ampart;    // bf16 path: LM-head top-2 records
  float* q_anchor; // the anchor layer's cross-attention queries [M][d]
  float* xscore;   // anchor readout scratch (scores, then per-chunk statistics)
  unsigned long long* abest;   // fused readout: per-sequence merged best
  int RT, qgroups;
  size_t bytes;
};

int div_up(int a, int b) { return (a + b - 1) / b; }

Workspace carve(const ad_model_desc& d, int M, int B, int k_max, char* base) {
  Workspace w{};
  size_t off = 0;
  auto take = [&](size_t n) {
    char* p = base ? base + off : nullptr;
    off += align256(n);
    return p;
  };
  const size_t D = d.d_model, F = d.d_ffn, V = d.vocab;
  w.RT = div_up(div_up(M, 16), 16) * 16;  // row tiles of the product operands
  w.qgroups = div_up(k_max + 1, 16);
  w.seqs = (ad::SeqDesc*)take(sizeof(ad::SeqDesc) * (size_t)B);
  w.rows = (ad::RowDesc*)take(sizeof(ad::RowDesc) * (size_t)M);
  w.tree = (ad::RowTree*)take(sizeof(ad::RowTree) * (size_t)M);
  w.x = (float*)take(4 * M * D);
  w.q = (float*)take(4 * M * D);
  w.hidden = (float*)take(4 * M * D);
  w.greedy = (int*)take(4ull * M);
  w.q_anchor = (float*)take(4 * M * D);
  w.xscore = (float*)take(4 * ad::anchor_scratch_floats(M, B, d.n_heads, d.max_frames));
  w.abest = (unsigned long long*)take(8ull * B);
  if (d.dtype == AD_F32) {
    w.ln = (float*)take(4 * M * D);
    w.att = (float*)take(4 * M * D);
    w.hid = (float*)take(4 * M * F);
    w.gself = ad::attn_valu_groups(d.max_pos);
    w.gcross = ad::attn_valu_groups(d.max_frames);
    w.apart = (float*)take(4 * ad::attn_valu_part_floats(M, d.n_heads, std::max(w.gself, w.gcross)));
    w.logits = (float*)take(4 * M * V);
  } else {
    const int Mp = w.RT * 16;
    w.afrag = (uint16_t*)take(4ull * Mp * D);
    w.hfrag = (uint16_t*)take(4ull * Mp * F);
    size_t gp = 0;
    // projections that leave split-K partials (the FFN up-projection does not)
    const int shapes[5][2] = {{3 * (int)D, (int)D}, {(int)D, (int)D}, {(int)D, (int)D},
                              {(int)D, (int)D}, {(int)D, (int)F}};
    for (auto& sh : shapes) gp = std::max(gp, ad::gemm_part_floats(M, sh[0], sh[1]));
    w.gpart = (float*)take(4 * gp);
    w.ampart = take(16ull * M * ad::lm_records((int)V));
  }
  w.bytes = off;
  return w;
}

ad_status check_hip(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(AD_EHIP, std::string(where) + ": " + hipGetErrorString(e));
  return AD_OK;
}

// Brackets one kernel launch with a profiling event pair when that class is enabled.
// Timing of the selected kernel class: a start / stop event pair on the stream around
// its launch (or, for the pair classes, around a short sequence of launches).
struct ProfScope {
  ad_model* m;
  hipStream_t st;
  int idx = -1;
  ProfScope(const ad_model* model, int kernel, hipStream_t stream)
      : m(const_cast<ad_model*>(model)), st(stream) {
    if (m->prof_kernel == kernel && m->prof_used < (int)m->prof_start.size()) {
      idx = m->prof_used++;
      (void)hipEventRecord(m->prof_start[idx], st);
    }
  }
  void stop() {
    if (idx >= 0) (void)hipEventRecord(m->prof_stop[idx], st);
    idx = -1;
  }
  ~ProfScope() { stop(); }
};

// The residual stream after layer l into the step's tap slots that name it.
void copy_taps(const ad_step* s, int l, const float* x, int M, int d, hipStream_t st) {
  if (!s->out_taps) return;
  for (int i = 0; i < 3; ++i)
    if (s->tap_layers[i] == l)
      (void)hipMemcpyAsync(s->out_taps + (size_t)i * M * d, x, sizeof(float) * M * d,
                           hipMemcpyDeviceToDevice, st);
}

// The bf16 path keeps the anchor layer's scores in its cross-attention (no window: the
// readout covers every frame); otherwise the readout recomputes them.
bool anchor_fused(const ad_model* m, const ad_step* s) {
  return m->desc.dtype == AD_BF16 && s->anchor_layer >= 0 && !s->cross_window;
}

ad::AnchorArgs anchor_args(const ad_model* m, const ad_step* s, const Workspace& w) {
  const ad_model_desc& D = m->desc;
  ad::AnchorArgs a{};
  a.seqs = w.seqs;
  a.accept_len = s->accept_len;
  a.q = w.q_anchor;
  a.kv = s->cross.data;
  a.layer = s->anchor_layer;
  a.H = D.n_heads;
  a.d = D.d_model;
  a.frames_cap = s->cross.frames_cap;
  a.max_frames = D.max_frames;
  a.nchunks = div_up(D.max_frames, ad::kAnchorChunk);
  a.score = w.xscore;
  a.stats = (float2*)(w.xscore + ad::anchor_score_floats(s->rows, s->batch, D.n_heads, D.max_frames));
  a.fused = anchor_fused(m, s);
  a.best = w.abest;
  a.score_ld = ad::anchor_score_ld(D.max_frames);
  a.out_anchor = s->out_anchor;
  a.out_peak = s->out_anchor_peak;
  a.path = s->parents ? s->out_path : nullptr;   // a tree's last verified row: the path's end
  a.path_stride = s->k_max + 1;
  return a;
}

// The accept scan: prefix scan of a chain, or the walk down a draft tree.
void accept(const ad_step* s, const Workspace& w, const int* greedy, hipStream_t st) {
  if (s->parents)
    ad::launch_accept_tree(s->batch, s->k_max, w.seqs, s->tokens, s->parents, greedy, s->accept_len,
                           s->out_tokens, s->out_path, st);
  else
    ad::launch_accept(s->batch, s->k_max, w.seqs, s->tokens, greedy, s->accept_len, s->out_tokens, st);
}

template <class S>
void run_step_valu(const ad_model* m, const ad_step* s, const Workspace& w, hipStream_t st) {
  const ad_model_desc& D = m->desc;
  const int M = s->rows, d = D.d_model, F = D.d_ffn, H = D.n_heads, V = D.vocab;
  ad::StepArgs a{s->batch, s->layout, s->k_max, s->rows, V, D.max_pos, D.max_frames,
                 s->tokens, s->k, s->cu_rows, s->kv.kv_len, s->kv.block_table,
                 s->kv.pages_per_seq, s->kv.num_pages, s->cross.enc_len, s->cross.enc_off,
                 s->cross.frames_cap, s->cross_window, s->parents, w.tree};
  ad::launch_prep(a, w.seqs, w.rows, s->err_flag, st);
  ad::launch_embed<S>(M, d, w.rows, m->p[P_TOK], m->p[P_POS], w.x, s->in_rows, st);

  ad::EpiArgs e{};
  e.rows = w.rows;
  e.block_table = s->kv.block_table;
  e.pages_per_seq = s->kv.pages_per_seq;
  e.num_pages = s->kv.num_pages;
  e.H = H;
  e.d = d;
  e.frames_cap = s->cross.frames_cap;
  for (int l = 0; l < D.n_layers; ++l) {
    e.layer = l;
    // self-attention sublayer
    ad::launch_layernorm<S>(M, d, w.x, lp(m, l, LN1_G), lp(m, l, LN1_B), w.ln, st);
    e.out = w.q; e.ldo = d; e.cache = s->kv.pool;
    ad::launch_gemm_valu<S>(ad::EPI_QKV, M, 3 * d, d, w.ln, lp(m, l, W_QKV), lp(m, l, B_QKV), e, st);
    {
      ProfScope ps(m, AD_PROF_SELF_ATTN, st);
      ad::launch_self_attn_valu<S>(s->batch, M, H, d, l, w.seqs, w.rows, w.q, w.apart, w.gself, w.att,
                                   s->kv.pool, s->kv.num_pages, s->kv.block_table, s->kv.pages_per_seq,
                                   w.tree, st);
    }
    e.out = w.x; e.ldo = d;
    ad::launch_gemm_valu<S>(ad::EPI_RESID, M, d, d, w.att, lp(m, l, W_O), lp(m, l, B_O), e, st);
    // cross-attention sublayer
    ad::launch_layernorm<S>(M, d, w.x, lp(m, l, LN2_G), lp(m, l, LN2_B), w.ln, st);
    e.out = w.q; e.ldo = d;
    ad::launch_gemm_valu<S>(ad::EPI_STORE, M, d, d, w.ln, lp(m, l, W_XQ), lp(m, l, B_XQ), e, st);
    if (l == s->anchor_layer) {
      (void)hipMemcpyAsync(w.q_anchor, w.q, sizeof(float) * M * d, hipMemcpyDeviceToDevice, st);
      if (s->out_xq)
        (void)hipMemcpyAsync(s->out_xq, w.q, sizeof(float) * M * d, hipMemcpyDeviceToDevice, st);
    }
    {
      ProfScope ps(m, AD_PROF_CROSS_ATTN, st);
      ad::launch_cross_attn_valu<S>(s->batch, M, H, d, l, w.seqs, w.rows, w.q, w.apart, w.gcross, w.att,
                                    s->cross.data, s->cross.frames_cap, st);
    }
    e.out = w.x; e.ldo = d;
    ad::launch_gemm_valu<S>(ad::EPI_RESID, M, d, d, w.att, lp(m, l, W_XO), lp(m, l, B_XO), e, st);
    // feed-forward sublayer
    ad::launch_layernorm<S>(M, d, w.x, lp(m, l, LN3_G), lp(m, l, LN3_B), w.ln, st);
    e.out = w.hid; e.ldo = F;
    ad::launch_gemm_valu<S>(ad::EPI_GELU, M, F, d, w.ln, lp(m, l, W_1), lp(m, l, B_1), e, st);
    e.out = w.x; e.ldo = d;
    ad::launch_gemm_valu<S>(ad::EPI_RESID, M, d, F, w.hid, lp(m, l, W_2), lp(m, l, B_2), e, st);
    copy_taps(s, l, w.x, M, d, st);
  }
  float* hidden = s->out_hidden ? s->out_hidden : w.hidden;
  ad::launch_layernorm<S>(M, d, w.x, m->p[P_LNF_G], m->p[P_LNF_B], hidden, st);
  float* logits = s->out_logits ? s->out_logits : w.logits;
  e.out = logits; e.ldo = V;
  {
    ProfScope ps(m, AD_PROF_LM_HEAD, st);
    ad::launch_gemm_valu<S>(ad::EPI_STORE, M, V, d, hidden, m->p[P_TOK], nullptr, e, st);
  }
  int* greedy = s->out_greedy ? s->out_greedy : w.greedy;
  ad::launch_argmax(M, V, logits, V, w.rows, greedy, s->out_margin, s->err_flag, st);
  accept(s, w, greedy, st);
  if (s->anchor_layer >= 0) ad::launch_anchor<S>(anchor_args(m, s, w), s->batch, st);
}

// bf16 model.  The projections write split-K partial products that the next kernel
// finishes: the attention kernels (queries, and the block's keys / values into the
// cache) or the residual + LayerNorm row kernel.  The FFN up-projection runs unsplit with
// bias + GELU in its epilogue.
void run_step_mfma(const ad_model* m, const ad_step* s, const Workspace& w, hipStream_t st) {
  const ad_model_desc& D = m->desc;
  const int M = s->rows, d = D.d_model, F = D.d_ffn, H = D.n_heads, V = D.vocab, RT = w.RT;
  ad::StepArgs a{s->batch, s->layout, s->k_max, s->rows, V, D.max_pos, D.max_frames,
                 s->tokens, s->k, s->cu_rows, s->kv.kv_len, s->kv.block_table,
                 s->kv.pages_per_seq, s->kv.num_pages, s->cross.enc_len, s->cross.enc_off,
                 s->cross.frames_cap, s->cross_window, s->parents, w.tree};
  ad::launch_prep(a, w.seqs, w.rows, s->err_flag, st);
  ad::launch_embed_ln(M, d, w.rows, m->p[P_TOK], m->p[P_POS], w.x, s->in_rows, lp(m, 0, LN1_G),
                      lp(m, 0, LN1_B), w.afrag, RT, st);

  const std::vector<size_t>& poff = m->pack_off;
  // weight `which` of layer l (layer -1: the LM head), tiled when the model is packed
  auto wt = [&](int l, int which, const void* rowmajor, int& packed) -> const uint16_t* {
    packed = m->packed != nullptr;
    if (!packed) return (const uint16_t*)rowmajor;
    if (l < 0) return m->packed + poff[D.n_layers * kPackedPerLayer];
    const int slot = (int)(std::find(kPackedWhich, kPackedWhich + kPackedPerLayer, which) - kPackedWhich);
    return m->packed + poff[l * kPackedPerLayer + slot];
  };
  auto gemm = [&](int epi, int N, int K, const uint16_t* A, int l, int which, ad::EpiArgs e,
                  int prof, const void* bias = nullptr) {
    ad::GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.RT = RT; g.A = A;
    g.W = wt(l, which, l < 0 ? m->p[P_TOK] : lp(m, l, which), g.packed);
    g.bias = (const uint16_t*)bias;
    g.part = w.gpart;
    g.e = e;
    ProfScope ps(m, prof, st);
    ad::launch_gemm_mfma(epi, g, st);
  };
  const ad::EpiArgs none{};
  ad::AttnArgs at{};
  at.H = H; at.d = d; at.seqs = w.seqs; at.out = w.afrag; at.out_RT = RT;
  at.num_pages = s->kv.num_pages; at.block_table = s->kv.block_table;
  at.pages_per_seq = s->kv.pages_per_seq; at.frames_cap = s->cross.frames_cap;
  at.qgroups = w.qgroups; at.qkv_part = w.gpart; at.rows = M; at.tree = w.tree;
  at.row_stride = s->layout == AD_PADDED ? s->k_max + 1 : 0;

  for (int l = 0; l < D.n_layers; ++l) {
    at.layer = l;
    // self-attention sublayer (LN1 was applied by the previous row kernel)
    gemm(ad::EPI_PARTIAL, 3 * d, d, w.afrag, l, W_QKV, none, AD_PROF_GEMM);
    at.cross = 0; at.kv = (const uint16_t*)s->kv.pool; at.chunk = ad::kSelfChunk;
    at.max_chunks = div_up(D.max_pos, ad::kSelfChunk);
    at.qkv_splits = ad::gemm_splits(3 * d, d); at.qkv_n = 3 * d;
    at.qkv_bias = (const uint16_t*)lp(m, l, B_QKV);
    {
      ProfScope ps(m, AD_PROF_SELF_ATTN, st);
      ad::launch_attn_mfma(at, s->batch, st);
    }
    gemm(ad::EPI_PARTIAL, d, d, w.afrag, l, W_O, none, AD_PROF_GEMM);
    ad::launch_reduce_res_ln(M, d, ad::gemm_splits(d, d), w.gpart, lp(m, l, B_O), w.x,
                             lp(m, l, LN2_G), lp(m, l, LN2_B), w.afrag, RT, nullptr, st);
    // cross-attention sublayer (the pair classes time the query projection with and
    // without the attention after it: their difference is the attention kernel alone)
    ProfScope xq_cross(m, AD_PROF_XQ_CROSS, st);
    {
      ProfScope xq(m, AD_PROF_XQ, st);
      gemm(ad::EPI_PARTIAL, d, d, w.afrag, l, W_XQ, none, AD_PROF_GEMM);
    }
    at.cross = 1; at.kv = (const uint16_t*)s->cross.data; at.chunk = ad::kCrossChunk;
    at.max_chunks = div_up(D.max_frames, ad::kCrossChunk);
    at.qkv_splits = ad::gemm_splits(d, d); at.qkv_n = d;
    at.qkv_bias = (const uint16_t*)lp(m, l, B_XQ);
    const bool fuse = l == s->anchor_layer && anchor_fused(m, s);
    at.q_save = l == s->anchor_layer && (!fuse || s->out_xq) ? w.q_anchor : nullptr;
    at.score_out = fuse ? w.xscore : nullptr;
    at.stat_out = fuse ? (float2*)(w.xscore + ad::anchor_score_floats(M, s->batch, H, D.max_frames)) : nullptr;
    at.score_ld = ad::anchor_score_ld(D.max_frames);
    at.best_clear = fuse ? w.abest : nullptr;
    {
      ProfScope ps(m, AD_PROF_CROSS_ATTN, st);
      ad::launch_attn_mfma(at, s->batch, st);
    }
    xq_cross.stop();
    if (l == s->anchor_layer && s->out_xq)
      (void)hipMemcpyAsync(s->out_xq, w.q_anchor, sizeof(float) * M * d, hipMemcpyDeviceToDevice, st);
    gemm(ad::EPI_PARTIAL, d, d, w.afrag, l, W_XO, none, AD_PROF_GEMM);
    ad::launch_reduce_res_ln(M, d, ad::gemm_splits(d, d), w.gpart, lp(m, l, B_XO), w.x,
                             lp(m, l, LN3_G), lp(m, l, LN3_B), w.afrag, RT, nullptr, st);
    // feed-forward sublayer
    {
      ad::EpiArgs e{};
      e.frag = w.hfrag; e.frag_RT = RT;
      gemm(ad::EPI_GELU, F, d, w.afrag, l, W_1, e, AD_PROF_GEMM, lp(m, l, B_1));
    }
    gemm(ad::EPI_PARTIAL, d, F, w.hfrag, l, W_2, none, AD_PROF_GEMM);
    const bool last = l + 1 == D.n_layers;
    float* hidden = s->out_hidden ? s->out_hidden : w.hidden;
    ad::launch_reduce_res_ln(M, d, ad::gemm_splits(d, F), w.gpart, lp(m, l, B_2), w.x,
                             last ? m->p[P_LNF_G] : lp(m, l + 1, LN1_G),
                             last ? m->p[P_LNF_B] : lp(m, l + 1, LN1_B), w.afrag, RT,
                             last ? hidden : nullptr, st);
    copy_taps(s, l, w.x, M, d, st);
  }
  ad::EpiArgs e{};
  e.out = s->out_logits; e.ldo = V; e.am_part = w.ampart;
  gemm(ad::EPI_ARGMAX, V, d, w.afrag, -1, 0, e, AD_PROF_LM_HEAD);
  int* greedy = s->out_greedy ? s->out_greedy : w.greedy;
  ad::launch_argmax_final(M, ad::lm_records(V), w.ampart, w.rows, greedy, s->out_margin, s->err_flag, st);
  accept(s, w, greedy, st);
  if (s->anchor_layer >= 0) {
    ProfScope ps(m, AD_PROF_ANCHOR, st);
    ad::launch_anchor<ad::BF16>(anchor_args(m, s, w), s->batch, st);
  }
}

ad_status validate_desc(const ad_model_desc* d) {
  if (!d) return fail(AD_EINVAL, "model descriptor is NULL");
  if (d->dtype != AD_F32 && d->dtype != AD_BF16) return fail(AD_EINVAL, "unknown dtype");
  if (d->n_layers <= 0 || d->d_model <= 0 || d->n_heads <= 0 || d->d_ffn <= 0 || d->vocab <= 1 ||
      d->max_pos <= 0 || d->max_frames <= 0)
    return fail(AD_ERANGE, "model sizes must be positive (vocab >= 2)");
  if (d->d_model != AD_HEAD_DIM * d->n_heads)
    return fail(AD_EUNSUPPORTED, "d_model must equal 64 * n_heads");
  if (d->n_heads > 64) return fail(AD_EUNSUPPORTED, "n_heads must be <= 64 (d_model <= 4096)");
  if (d->d_ffn % 64 != 0) return fail(AD_EUNSUPPORTED, "d_ffn must be a multiple of 64");
  // one attention wave per key chunk, at most 8 waves per workgroup
  static_assert(8 * ad::kCrossChunk >= 2048 && 8 * ad::kSelfChunk >= 1024, "chunk limits");
  if (d->max_frames > 2048 || d->max_pos > 1024)
    return fail(AD_EUNSUPPORTED, "max_frames must be <= 2048 and max_pos <= 1024");
  return AD_OK;
}

// Library-owned step scratch for callers that cannot allocate device memory
// (ad_verify_step_static).  In host code `scratch` names a host-side stand-in, not a
// device address: the device address of each GPU's copy comes from hipGetSymbolAddress,
// taken once per device (with that device current) and kept in g_scratch_dev.
constexpr size_t kStaticScratchBytes = AD_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

ad_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(AD_EHIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return fail(AD_EUNSUPPORTED, "device index past the static scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(AD_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return AD_OK;
}

}  // namespace

extern "C" {

const char* ad_last_error(void) { return g_err.c_str(); }

int32_t ad_model_param_count(const ad_model_desc* desc) {
  return desc ? 4 + N_LAYER_PARAMS * desc->n_layers : -1;
}

ad_status ad_model_create(const ad_model_desc* desc, const void* const* params, int32_t n_params,
                          ad_model** out) {
  if (!out) return fail(AD_EINVAL, "out is NULL");
  *out = nullptr;
  ad_status st = validate_desc(desc);
  if (st != AD_OK) return st;
  if (!params) return fail(AD_EINVAL, "params is NULL");
  if (n_params != ad_model_param_count(desc))
    return fail(AD_EINVAL, "expected " + std::to_string(ad_model_param_count(desc)) + " parameters");
  for (int i = 0; i < n_params; ++i)
    if (!params[i]) return fail(AD_EINVAL, "parameter " + std::to_string(i) + " is NULL");
  for (int i = 0; i < n_params; ++i)
    if ((uintptr_t)params[i] % 16)
      return fail(AD_EINVAL, "parameter " + std::to_string(i) + " is not 16-byte aligned");
  ad_model* m = new ad_model;
  m->desc = *desc;
  m->p.assign(params, params + n_params);
  *out = m;
  return AD_OK;
}

static void prof_free(ad_model* m) {
  for (auto e : m->prof_start) (void)hipEventDestroy(e);
  for (auto e : m->prof_stop) (void)hipEventDestroy(e);
  m->prof_start.clear();
  m->prof_stop.clear();
  m->prof_used = 0;
  m->prof_kernel = 0;
}

ad_status ad_model_pack_size(const ad_model* model, size_t* bytes) {
  if (!model || !bytes) return fail(AD_EINVAL, "NULL argument");
  if (model->desc.dtype != AD_BF16) return fail(AD_EUNSUPPORTED, "weight tiling is for bf16 models");
  *bytes = packed_offsets(model->desc).back() * sizeof(uint16_t);
  return AD_OK;
}

ad_status ad_model_pack(ad_model* model, void* buffer, size_t bytes, void* stream) {
  if (!model) return fail(AD_EINVAL, "model is NULL");
  if (model->desc.dtype != AD_BF16) return fail(AD_EUNSUPPORTED, "weight tiling is for bf16 models");
  if (!buffer) {
    model->packed = nullptr;
    model->pack_off.clear();
    return AD_OK;
  }
  if ((uintptr_t)buffer % 256) return fail(AD_EINVAL, "pack buffer must be 256-byte aligned");
  const ad_model_desc& D = model->desc;
  const std::vector<size_t> off = packed_offsets(D);
  if (bytes < off.back() * sizeof(uint16_t))
    return fail(AD_ENOSPACE, "pack buffer needs " + std::to_string(off.back() * sizeof(uint16_t)) + " bytes");
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  uint16_t* P = (uint16_t*)buffer;
  for (int l = 0; l < D.n_layers; ++l)
    for (int j = 0; j < kPackedPerLayer; ++j) {
      int N, K;
      packed_shape(D, kPackedWhich[j], N, K);
      ad::launch_pack_weight((const uint16_t*)lp(model, l, kPackedWhich[j]), N, K,
                             P + off[l * kPackedPerLayer + j], st);
    }
  ad::launch_pack_weight((const uint16_t*)model->p[P_TOK], D.vocab, D.d_model,
                         P + off[D.n_layers * kPackedPerLayer], st);
  const ad_status rc = check_hip("ad_model_pack");
  if (rc != AD_OK) return rc;
  model->packed = P;
  model->pack_off = off;
  return AD_OK;
}

ad_status ad_model_destroy(ad_model* model) {
  if (model) prof_free(model);
  delete model;
  return AD_OK;
}

ad_status ad_profile_enable(ad_model* model, int32_t kernel, int32_t max_launches) {
  if (!model) return fail(AD_EINVAL, "model is NULL");
  if (max_launches < 0 || max_launches > (1 << 20)) return fail(AD_ERANGE, "max_launches out of range");
  if (max_launches > 0 && (kernel < AD_PROF_CROSS_ATTN || kernel > AD_PROF_ANCHOR))
    return fail(AD_EINVAL, "unknown kernel class");
  prof_free(model);
  if (max_launches == 0) return AD_OK;
  model->prof_start.resize(max_launches);
  model->prof_stop.resize(max_launches);
  for (int i = 0; i < max_launches; ++i) {
    // no system-scope fence: a default event record releases (writes back) the caches,
    // which would stall the timed kernel and inflate its measured duration
    if (hipEventCreateWithFlags(&model->prof_start[i], hipEventDisableSystemFence) != hipSuccess ||
        hipEventCreateWithFlags(&model->prof_stop[i], hipEventDisableSystemFence) != hipSuccess) {
      model->prof_start.resize(i);
      model->prof_stop.resize(i);
      prof_free(model);
      return fail(AD_EHIP, "hipEventCreate failed");
    }
  }
  model->prof_kernel = kernel;
  return AD_OK;
}

ad_status ad_profile_read(ad_model* model, double* total_ms, int32_t* launches) {
  if (!model || !total_ms || !launches) return fail(AD_EINVAL, "NULL argument");
  double t = 0.0;
  for (int i = 0; i < model->prof_used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(model->prof_stop[i]) != hipSuccess ||
        hipEventElapsedTime(&ms, model->prof_start[i], model->prof_stop[i]) != hipSuccess)
      return fail(AD_EHIP, "reading profiling events failed");
    t += ms;
  }
  *total_ms = t;
  *launches = model->prof_used;
  model->prof_used = 0;
  return AD_OK;
}

ad_status ad_workspace_size(const ad_model* model, int32_t max_rows, int32_t max_batch,
                            int32_t k_max, size_t* bytes) {
  if (!model || !bytes) return fail(AD_EINVAL, "NULL argument");
  if (max_rows <= 0 || max_batch <= 0 || k_max < 0)
    return fail(AD_ERANGE, "max_rows and max_batch must be positive, k_max non-negative");
  *bytes = carve(model->desc, max_rows, max_batch, k_max, nullptr).bytes;
  return AD_OK;
}

ad_status ad_verify_step(const ad_model* model, const ad_step* s, void* stream) {
  if (!model || !s) return fail(AD_EINVAL, "model or step is NULL");
  const ad_model_desc& D = model->desc;
  if (!s->tokens || !s->k || !s->kv.pool || !s->kv.kv_len || !s->kv.block_table || !s->cross.data ||
      !s->cross.enc_len || !s->cross.enc_off || !s->accept_len || !s->out_tokens || !s->err_flag ||
      !s->workspace)
    return fail(AD_EINVAL, "a required step pointer is NULL");
  if (s->layout != AD_PADDED && s->layout != AD_PACKED) return fail(AD_EINVAL, "unknown layout");
  if (s->layout == AD_PACKED && !s->cu_rows) return fail(AD_EINVAL, "packed layout needs cu_rows");
  if (s->batch < 1) return fail(AD_ERANGE, "batch must be >= 1");
  if (s->k_max < 0 || s->k_max + 1 > D.max_pos) return fail(AD_ERANGE, "k_max out of range");
  if (s->k_max + 1 > ad::kMaxBlockRows)
    return fail(AD_EUNSUPPORTED, "at most 64 rows per sequence are verified (k_max <= 63)");
  if (s->parents && !s->out_path) return fail(AD_EINVAL, "parents need out_path");
  if (s->out_xq && s->anchor_layer < 0) return fail(AD_EINVAL, "out_xq needs anchor_layer >= 0");
  const long long full = (long long)s->batch * (s->k_max + 1);
  if (s->layout == AD_PADDED && s->rows != full)
    return fail(AD_ERANGE, "padded layout needs rows == batch * (k_max + 1)");
  if (s->layout == AD_PACKED && (s->rows < s->batch || s->rows > full))
    return fail(AD_ERANGE, "packed rows must lie in [batch, batch * (k_max + 1)]");
  if (s->kv.num_pages < 1 || s->kv.pages_per_seq < 1) return fail(AD_ERANGE, "empty page pool");
  if (s->cross.frames_cap < ad::kCrossBlock || s->cross.frames_cap % ad::kCrossBlock)
    return fail(AD_ERANGE, "frames_cap must be a positive multiple of 32");
  if (s->anchor_layer < -1 || s->anchor_layer >= D.n_layers)
    return fail(AD_ERANGE, "anchor_layer must be -1 or a layer index");
  if (s->anchor_layer >= 0 && !s->out_anchor)
    return fail(AD_EINVAL, "the anchor readout needs out_anchor");
  for (int i = 0; i < 3; ++i) {
    if (s->tap_layers[i] < -1 || s->tap_layers[i] >= D.n_layers)
      return fail(AD_ERANGE, "tap_layers must be -1 or layer indices");
    if (s->tap_layers[i] >= 0 && !s->out_taps) return fail(AD_EINVAL, "tap_layers need out_taps");
  }
  if ((uintptr_t)s->workspace % 256) return fail(AD_EINVAL, "workspace must be 256-byte aligned");
  if ((uintptr_t)s->in_rows % 16) return fail(AD_EINVAL, "in_rows must be 16-byte aligned");
  const Workspace need = carve(D, s->rows, s->batch, s->k_max, nullptr);
  if (s->workspace_bytes < need.bytes)
    return fail(AD_ENOSPACE, "workspace needs " + std::to_string(need.bytes) + " bytes");
  (void)hipGetLastError();
  const Workspace w = carve(D, s->rows, s->batch, s->k_max, (char*)s->workspace);
  hipStream_t st = (hipStream_t)stream;
  if (D.dtype == AD_BF16) run_step_mfma(model, s, w, st);
  else run_step_valu<ad::F32>(model, s, w, st);
  return check_hip("ad_verify_step");
}

ad_status ad_verify_step_static(const ad_model* model, const ad_step* s, void* stream) {
  if (!model || !s) return fail(AD_EINVAL, "model or step is NULL");
  if (s->rows <= 0 || s->batch < 1 || s->k_max < 0) return fail(AD_ERANGE, "rows, batch and k_max out of range");
  const size_t need = carve(model->desc, s->rows, s->batch, s->k_max, nullptr).bytes;
  if (need > kStaticScratchBytes)
    return fail(AD_ENOSPACE, "this step needs " + std::to_string(need) + " bytes of scratch; the static scratch "
                             "holds " + std::to_string(kStaticScratchBytes) + " (use ad_verify_step with a workspace)");
  void* p = nullptr;
  const ad_status rc = static_scratch(&p);
  if (rc != AD_OK) return rc;
  ad_step t = *s;
  t.workspace = p;
  t.workspace_bytes = kStaticScratchBytes;
  return ad_verify_step(model, &t, stream);
}

// ad_draft_input's scratch.  float32 models: the gathered rows [B][4d], the feature
// [B][d] and the concatenated rows [B][2d] for the VALU products.  bf16 models: the
// matrix-core products' A operand (A-fragment order, up to 4d wide), their split-K
// partials and the feature.
struct DraftInputWs {
  size_t frag, part, feat, bytes;
  int RT;
};
DraftInputWs draft_input_ws(const ad_model_desc& D, int B) {
  DraftInputWs w{};
  const size_t d = D.d_model;
  if (D.dtype != AD_BF16) {
    w.bytes = sizeof(float) * 7 * d * B;
    return w;
  }
  w.RT = div_up(div_up(B, 16), 16) * 16;
  w.frag = 0;
  w.part = align256((size_t)w.RT * 16 * 4 * d * 4);
  const size_t parts = std::max(ad::gemm_part_floats(B, (int)d, 4 * (int)d),
                                ad::gemm_part_floats(B, (int)d, 2 * (int)d));
  w.feat = w.part + align256(4 * parts);
  w.bytes = w.feat + align256(4 * d * B);
  return w;
}

ad_status ad_draft_input_workspace_size(const ad_model* model, int32_t batch, size_t* bytes) {
  if (!model || !bytes) return fail(AD_EINVAL, "NULL argument");
  if (batch < 1) return fail(AD_ERANGE, "batch must be >= 1");
  *bytes = draft_input_ws(model->desc, batch).bytes;
  return AD_OK;
}

ad_status ad_draft_input(const ad_model* model, const void* w_fuse, const void* b_fuse,
                         const void* w_in, const void* b_in, int32_t batch, const float* taps,
                         const float* hidden, int32_t layout, int32_t k_max,
                         const int32_t* cu_rows, const int32_t* accept_len, int32_t rows,
                         const float* feature, const int32_t* tokens, int32_t token_stride,
                         const int32_t* token_index, const int32_t* anchor,
                         const int32_t* enc_len, int32_t half_window, int32_t* window,
                         float* out, void* workspace, size_t workspace_bytes, void* stream) {
  if (!model || !w_fuse || !b_fuse || !w_in || !b_in || !tokens || !out || !workspace)
    return fail(AD_EINVAL, "NULL argument");
  if (batch < 1 || token_stride < 1) return fail(AD_ERANGE, "batch and token_stride must be >= 1");
  if (taps) {
    if (!hidden || !accept_len) return fail(AD_EINVAL, "taps need hidden and accept_len");
    if (layout != AD_PADDED && layout != AD_PACKED) return fail(AD_EINVAL, "unknown layout");
    if (layout == AD_PACKED && !cu_rows) return fail(AD_EINVAL, "packed layout needs cu_rows");
    if (rows < batch || k_max < 0) return fail(AD_ERANGE, "rows must be >= batch, k_max >= 0");
  } else if (!feature) {
    return fail(AD_EINVAL, "either taps or feature is needed");
  }
  if (anchor && (!enc_len || !window)) return fail(AD_EINVAL, "anchor needs enc_len and window");
  if (anchor && half_window < 0) return fail(AD_ERANGE, "half_window must be >= 0");
  const ad_model_desc& D = model->desc;
  const int d = D.d_model;
  size_t need = 0;
  ad_draft_input_workspace_size(model, batch, &need);
  if ((uintptr_t)workspace % 256) return fail(AD_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < need) return fail(AD_ENOSPACE, "workspace needs " + std::to_string(need) + " bytes");
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  if (D.dtype == AD_BF16) {
    // matrix-core products: A operand in fragment order, split-K partials, then the sum
    // of the partials plus the bias
    const DraftInputWs w = draft_input_ws(D, batch);
    char* base = (char*)workspace;
    uint16_t* frag = (uint16_t*)(base + w.frag);
    float* part = (float*)(base + w.part);
    float* feat = (float*)(base + w.feat);
    auto product = [&](int K, const void* W, const void* bias, float* dst) {
      ad::GemmArgs g{};
      g.M = batch; g.N = d; g.K = K; g.RT = w.RT; g.A = frag; g.W = (const uint16_t*)W;
      g.packed = 0; g.part = part;
      ad::launch_gemm_mfma(ad::EPI_PARTIAL, g, st);
      ad::launch_sum_partials_bias(batch, d, ad::gemm_splits(d, K), part, bias, dst, st);
    };
    const float* f = feature;
    if (taps) {
      ad::launch_draft_gather_taps_frag(batch, d, layout, k_max, cu_rows, accept_len, rows, taps,
                                        hidden, frag, w.RT, st);
      product(4 * d, w_fuse, b_fuse, feat);
      f = feat;
    }
    ad::launch_draft_concat_frag(batch, d, f, model->p[P_TOK], tokens, token_stride, token_index,
                                 frag, w.RT, st);
    product(2 * d, w_in, b_in, out);
    if (anchor) ad::launch_draft_window(batch, anchor, enc_len, half_window, window, st);
    return check_hip("ad_draft_input");
  }
  float* taps4 = (float*)workspace;
  float* feat = taps4 + (size_t)4 * d * batch;
  float* z = feat + (size_t)d * batch;
  const float* f = feature;
  ad::EpiArgs e{};
  e.ldo = d;
  const bool bf16 = false;
  if (taps) {
    ad::launch_draft_gather_taps(batch, d, layout, k_max, cu_rows, accept_len, rows, taps, hidden,
                                 taps4, st);
    e.out = feat;
    if (bf16) ad::launch_gemm_valu<ad::BF16>(ad::EPI_STORE, batch, d, 4 * d, taps4, w_fuse, b_fuse, e, st);
    else ad::launch_gemm_valu<ad::F32>(ad::EPI_STORE, batch, d, 4 * d, taps4, w_fuse, b_fuse, e, st);
    f = feat;
  }
  ad::launch_draft_concat(batch, d, f, model->p[P_TOK], bf16, tokens, token_stride, token_index, z, st);
  e.out = out;
  if (bf16) ad::launch_gemm_valu<ad::BF16>(ad::EPI_STORE, batch, d, 2 * d, z, w_in, b_in, e, st);
  else ad::launch_gemm_valu<ad::F32>(ad::EPI_STORE, batch, d, 2 * d, z, w_in, b_in, e, st);
  if (anchor) ad::launch_draft_window(batch, anchor, enc_len, half_window, window, st);
  return check_hip("ad_draft_input");
}

ad_status ad_kv_commit(int32_t* kv_len, const int32_t* accept_len, int32_t batch, void* stream) {
  if (!kv_len || !accept_len) return fail(AD_EINVAL, "NULL argument");
  if (batch < 1) return fail(AD_ERANGE, "batch must be >= 1");
  (void)hipGetLastError();
  ad::launch_commit(batch, kv_len, accept_len, (hipStream_t)stream);
  return check_hip("ad_kv_commit");
}

struct LossWs {
  size_t stats, Z, gq, lpart, lrow, tok, feat, flag, counts, bytes;
  int nchunk, g_ld;
};
LossWs loss_ws(const ad_model_desc& D, int batch, int R) {
  LossWs w{};
  const size_t M = (size_t)batch * R;
  w.nchunk = ad::loss_chunks(D.max_frames);
  w.g_ld = (D.max_frames + 31) / 32 * 32;   // whole 32-frame blocks per row
  size_t off = 0;
  auto take = [&](size_t n) { const size_t o = off; off += align256(n); return o; };
  w.stats = take(8 * M * D.n_heads);
  w.Z = take(4 * M);
  w.gq = take(4 * M * w.g_ld);
  w.lpart = take(4 * M * w.nchunk);
  w.lrow = take(4 * M);
  w.tok = take(4 * M);
  w.feat = take(4 * M);
  w.flag = take(4 * M);
  w.counts = take(8);
  w.bytes = off;
  return w;
}

ad_status ad_anchordraft_loss_workspace_size(const ad_model* draft, int32_t batch, int32_t rows_per_seq,
                                             size_t* bytes) {
  if (!draft || !bytes) return fail(AD_EINVAL, "NULL argument");
  if (batch < 1 || rows_per_seq < 1) return fail(AD_ERANGE, "batch and rows_per_seq must be >= 1");
  *bytes = loss_ws(draft->desc, batch, rows_per_seq).bytes;
  return AD_OK;
}

ad_status ad_anchordraft_loss(const ad_model* draft, const ad_cross* cross, int32_t layer, int32_t batch,
                              int32_t rows_per_seq, const float* xq, const int32_t* center, float sigma,
                              float lambda, const float* logits, const int32_t* targets,
                              const float* feat, const float* feat_target, float* out_terms,
                              float* out_row, float* out_dxq, float* out_dlogits, float* out_dfeat,
                              int32_t* err_flag, void* workspace, size_t workspace_bytes, void* stream) {
  if (!draft || !out_terms || !err_flag || !workspace) return fail(AD_EINVAL, "NULL argument");
  const ad_model_desc& D = draft->desc;
  if (D.dtype != AD_BF16) return fail(AD_EUNSUPPORTED, "the loss kernels take bf16 draft models");
  if (batch < 1 || rows_per_seq < 1) return fail(AD_ERANGE, "batch and rows_per_seq must be >= 1");
  if (xq) {
    if (!cross || !cross->data || !cross->enc_len || !cross->enc_off || !center)
      return fail(AD_EINVAL, "xq needs cross (data, enc_len, enc_off) and center");
    if (cross->frames_cap < ad::kCrossBlock || cross->frames_cap % ad::kCrossBlock)
      return fail(AD_ERANGE, "frames_cap must be a positive multiple of 32");
    if (layer < 0 || layer >= D.n_layers) return fail(AD_ERANGE, "layer must be a layer index");
    if (!(sigma > 0.f) || !std::isfinite(sigma)) return fail(AD_ERANGE, "sigma must be positive");
    if (!(lambda >= 0.f) || !std::isfinite(lambda)) return fail(AD_ERANGE, "lambda must be >= 0");
  } else if (out_dxq || out_row) {
    return fail(AD_EINVAL, "out_dxq and out_row need xq");
  }
  if ((logits || feat) && !targets) return fail(AD_EINVAL, "logits and feat need targets");
  if (feat && !feat_target) return fail(AD_EINVAL, "feat needs feat_target");
  if (out_dlogits && !logits) return fail(AD_EINVAL, "out_dlogits needs logits");
  if (out_dfeat && !feat) return fail(AD_EINVAL, "out_dfeat needs feat");
  const LossWs w = loss_ws(D, batch, rows_per_seq);
  if ((uintptr_t)workspace % 256) return fail(AD_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < w.bytes) return fail(AD_ENOSPACE, "workspace needs " + std::to_string(w.bytes) + " bytes");
  char* base = (char*)workspace;
  ad::LossArgs a{};
  a.B = batch; a.R = rows_per_seq; a.M = batch * rows_per_seq; a.H = D.n_heads; a.d = D.d_model;
  a.V = D.vocab; a.layer = layer; a.max_frames = D.max_frames; a.nchunk = w.nchunk;
  a.g_ld = w.g_ld;
  if (xq) {
    a.kv = (const uint16_t*)cross->data; a.frames_cap = cross->frames_cap;
    a.enc_len = cross->enc_len; a.enc_off = cross->enc_off;
  }
  a.xq = xq; a.center = center; a.sigma = sigma; a.lam = xq ? lambda : 0.f;
  a.logits = logits; a.targets = targets; a.feat = feat; a.feat_target = feat_target;
  a.stats = (float2*)(base + w.stats); a.Z = (float*)(base + w.Z); a.gq = (float*)(base + w.gq);
  a.lpart = (float*)(base + w.lpart); a.lrow = (float*)(base + w.lrow); a.tok_row = (float*)(base + w.tok);
  a.feat_row = (float*)(base + w.feat); a.rowflag = (int*)(base + w.flag);
  a.counts = (int*)(base + w.counts);
  a.out_terms = out_terms; a.out_row = out_row; a.out_dxq = out_dxq; a.out_dlogits = out_dlogits;
  a.out_dfeat = out_dfeat; a.err = err_flag;
  (void)hipGetLastError();
  ad::launch_anchordraft_loss(a, (hipStream_t)stream);
  return check_hip("ad_anchordraft_loss");
}

ad_status ad_kv_commit_tree(const ad_model* model, const ad_kv* kv, const int32_t* accept_len,
                            const int32_t* path, int32_t path_stride, int32_t batch, void* stream) {
  if (!model || !kv || !kv->pool || !kv->kv_len || !kv->block_table || !accept_len || !path)
    return fail(AD_EINVAL, "NULL argument");
  if (batch < 1 || path_stride < 1 || kv->num_pages < 1 || kv->pages_per_seq < 1)
    return fail(AD_ERANGE, "batch, path_stride, num_pages and pages_per_seq must be positive");
  const ad_model_desc& D = model->desc;
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  if (D.dtype == AD_BF16)
    ad::launch_kv_compact<ad::BF16>(batch, D.n_layers, D.n_heads, kv->kv_len, accept_len, path,
                                    path_stride, kv->pool, kv->num_pages, kv->block_table,
                                    kv->pages_per_seq, st);
  else
    ad::launch_kv_compact<ad::F32>(batch, D.n_layers, D.n_heads, kv->kv_len, accept_len, path,
                                   path_stride, kv->pool, kv->num_pages, kv->block_table,
                                   kv->pages_per_seq, st);
  ad::launch_commit(batch, kv->kv_len, accept_len, st);
  return check_hip("ad_kv_commit_tree");
}

ad_status ad_cross_kv_prefill(const ad_model* model, const void* enc, const ad_cross* cross, void* stream) {
  if (!model || !enc || !cross || !cross->data) return fail(AD_EINVAL, "NULL argument");
  if (cross->frames_cap < ad::kCrossBlock || cross->frames_cap % ad::kCrossBlock)
    return fail(AD_ERANGE, "frames_cap must be a positive multiple of 32");
  const ad_model_desc& D = model->desc;
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  ad::EpiArgs e{};
  e.cache = cross->data;
  e.H = D.n_heads;
  e.d = D.d_model;
  e.frames_cap = cross->frames_cap;
  // bf16 models: the matrix cores (a large dense product); float32 models: the VALU.
  // With two or more layers the bf16 path first copies the encoder states into fragment
  // order, staged in the last layer's part of the cache (frames_cap x 2d elements, at
  // least the frames_cap x d of the copy), which is only written by the last launch;
  // that launch reads the row-major states.  A tiled model supplies tiled weights.
  const bool stage = D.dtype == AD_BF16 && D.n_layers >= 2;
  const size_t layer_elems = (size_t)2 * D.n_heads * cross->frames_cap * 64;
  uint16_t* staged = (uint16_t*)cross->data + (size_t)(D.n_layers - 1) * layer_elems;
  if (stage) {
    const uintptr_t e0 = (uintptr_t)enc, e1 = e0 + (size_t)cross->frames_cap * D.d_model * 2;
    const uintptr_t s0 = (uintptr_t)staged, s1 = s0 + layer_elems * 2;
    if (e0 < s1 && s0 < e1) return fail(AD_EINVAL, "enc overlaps the last layer's cross-K/V slots");
  }
  if (stage) ad::launch_pack_rows((const uint16_t*)enc, cross->frames_cap, D.d_model, staged, st);
  for (int l = 0; l < D.n_layers; ++l) {
    e.layer = l;
    if (D.dtype == AD_BF16) {
      const bool a_packed = stage && l < D.n_layers - 1;
      const bool w_packed = model->packed != nullptr;
      const uint16_t* W = w_packed ? model->packed + model->pack_off[l * kPackedPerLayer + kPackedXkv]
                                   : (const uint16_t*)lp(model, l, W_XKV);
      ad::launch_xkv_mfma(cross->frames_cap, 2 * D.d_model, D.d_model,
                          a_packed ? staged : (const uint16_t*)enc, a_packed, W, w_packed,
                          (const uint16_t*)lp(model, l, B_XKV), (uint16_t*)cross->data, l, D.n_heads,
                          D.d_model, cross->frames_cap, st);
    } else
      ad::launch_gemm_valu<ad::F32>(ad::EPI_XKV, cross->frames_cap, 2 * D.d_model, D.d_model,
                                    (const float*)enc, lp(model, l, W_XKV), lp(model, l, B_XKV), e, st);
  }
  return check_hip("ad_cross_kv_prefill");
}

ad_status ad_draft_heads_workspace_size(const ad_model* model, int32_t n_heads, int32_t batch,
                                        size_t* bytes) {
  if (!model || !bytes) return fail(AD_EINVAL, "NULL argument");
  if (n_heads < 1 || batch < 1) return fail(AD_ERANGE, "n_heads and batch must be positive");
  const ad_model_desc& D = model->desc;
  *bytes = align256(4ull * batch * D.d_model) + align256(4ull * n_heads * batch * D.vocab) +
           align256(4ull * n_heads * batch);
  return AD_OK;
}

ad_status ad_draft_heads(const ad_model* model, const void* heads_w, int32_t n_heads, const float* hidden,
                         int32_t layout, int32_t k_max, const int32_t* cu_rows, const int32_t* accept_len,
                         const int32_t* out_tokens, int32_t batch, int32_t* next_tokens, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (!model || !heads_w || !hidden || !accept_len || !out_tokens || !next_tokens || !workspace)
    return fail(AD_EINVAL, "NULL argument");
  if (layout != AD_PADDED && layout != AD_PACKED) return fail(AD_EINVAL, "unknown layout");
  if (layout == AD_PACKED && !cu_rows) return fail(AD_EINVAL, "packed layout needs cu_rows");
  if (n_heads < 1 || batch < 1 || k_max < 0) return fail(AD_ERANGE, "sizes out of range");
  size_t need = 0;
  ad_draft_heads_workspace_size(model, n_heads, batch, &need);
  if ((uintptr_t)workspace % 256) return fail(AD_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < need) return fail(AD_ENOSPACE, "workspace needs " + std::to_string(need) + " bytes");
  const ad_model_desc& D = model->desc;
  char* base = (char*)workspace;
  float* hsel = (float*)base;
  base += align256(4ull * batch * D.d_model);
  float* logits = (float*)base;
  base += align256(4ull * n_heads * batch * D.vocab);
  int* greedy = (int*)base;
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  ad::launch_gather_hidden(batch, D.d_model, layout, k_max, cu_rows, accept_len, hidden, hsel, st);
  const size_t esz = D.dtype == AD_BF16 ? 2 : 4;
  ad::EpiArgs e{};
  for (int i = 0; i < n_heads; ++i) {
    e.out = logits + (size_t)i * batch * D.vocab;
    e.ldo = D.vocab;
    const void* w = (const char*)heads_w + (size_t)i * D.vocab * D.d_model * esz;
    if (D.dtype == AD_BF16)
      ad::launch_gemm_valu<ad::BF16>(ad::EPI_STORE, batch, D.vocab, D.d_model, hsel, w, nullptr, e, st);
    else
      ad::launch_gemm_valu<ad::F32>(ad::EPI_STORE, batch, D.vocab, D.d_model, hsel, w, nullptr, e, st);
  }
  // the err flag of the step is not touched here: non-finite head logits give -1 drafts
  ad::launch_argmax(n_heads * batch, D.vocab, logits, D.vocab, nullptr, greedy, nullptr, nullptr, st);
  ad::launch_assemble_next(batch, n_heads, k_max, accept_len, out_tokens, greedy, next_tokens, st);
  return check_hip("ad_draft_heads");
}

static ad_status kv_copy(const char* what, bool to_linear, const ad_model* model, const ad_kv* kv,
                         int32_t b, void* lin, int32_t n, int32_t* err_flag, void* stream) {
  if (!model || !kv || !kv->pool || !kv->block_table || !err_flag || (n > 0 && !lin))
    return fail(AD_EINVAL, std::string(what) + ": NULL argument");
  const ad_model_desc& D = model->desc;
  if (b < 0 || n < 0 || n > D.max_pos || n > kv->pages_per_seq * ad::kTile)
    return fail(AD_ERANGE, std::string(what) + ": sequence index or prefix length out of range");
  (void)hipGetLastError();
  hipStream_t st = (hipStream_t)stream;
  if (D.dtype == AD_BF16)
    ad::launch_kv_copy<ad::BF16>(to_linear, D.n_layers, D.n_heads, n, b, lin, kv->pool, kv->num_pages,
                                 kv->block_table, kv->pages_per_seq, err_flag, st);
  else
    ad::launch_kv_copy<ad::F32>(to_linear, D.n_layers, D.n_heads, n, b, lin, kv->pool, kv->num_pages,
                                kv->block_table, kv->pages_per_seq, err_flag, st);
  return check_hip(what);
}

ad_status ad_kv_import(const ad_model* model, const ad_kv* kv, int32_t b, const void* src, int32_t n,
                       int32_t* err_flag, void* stream) {
  return kv_copy("ad_kv_import", false, model, kv, b, const_cast<void*>(src), n, err_flag, stream);
}

ad_status ad_kv_export(const ad_model* model, const ad_kv* kv, int32_t b, void* dst, int32_t n,
                       int32_t* err_flag, void* stream) {
  return kv_copy("ad_kv_export", true, model, kv, b, dst, n, err_flag, stream);
}

}  // extern "C"
