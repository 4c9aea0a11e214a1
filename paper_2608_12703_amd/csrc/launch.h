// Internal launcher declarations shared by the libad translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace ad {

// Plain-old-data copy of the step's scalars and device pointers handed to kernels.
struct StepArgs {
  int B, layout, k_max, rows;
  int V, max_pos, max_frames;
  const int* tokens;
  const int* k;
  const int* cu_rows;
  const int* kv_len;
  const int* block_table;
  int pages_per_seq, num_pages;
  const int* enc_len;
  const int* enc_off;
  int frames_cap;
  const int* cross_window;   // [B][2] frames [lo, hi), or NULL: all frames
  const int* parents;        // [rows] draft-tree parents within the block, or NULL: linear
  RowTree* tree;             // [rows] built from parents by the prep kernel
};

// Where a GEMM's epilogue sends its output.
enum Epi : int {
  EPI_STORE = 0,   // out[m][n] = acc + bias                  (float32)
  EPI_RESID = 1,   // out[m][n] += acc + bias                 (residual stream)
  EPI_GELU = 2,    // out[m][n] = GELU(acc + bias)            (float32)
  EPI_QKV = 3,     // n < d: q; d <= n < 3d: key / value into the paged cache
  EPI_XKV = 4,     // cross-K/V prefill: n < d key, else value, into the cross cache
  EPI_ARGMAX = 5,  // LM head: per-tile top-2 records (and optionally the logits)
  EPI_PARTIAL = 6, // raw product (split-K partial when S > 1) into part[s][m][n]
};

struct EpiArgs {
  float* out;
  size_t ldo;
  uint16_t* frag;   // EPI_GELU: output in A-fragment order (hi/lo) with frag_RT row tiles
  int frag_RT;
  void* am_part;    // EPI_ARGMAX: float4 [M][tiles] top-2 records
  // cache writes
  const RowDesc* rows;
  void* cache;
  const int* block_table;
  int pages_per_seq, num_pages, H, d, layer, frames_cap;
};

void launch_prep(const StepArgs& a, SeqDesc* seqs, RowDesc* rows, int* err, hipStream_t st);
// x = E_tok[token] + E_pos[pos] per row, or in_rows[row] + E_pos[pos] when in_rows is set.
template <class S>
void launch_embed(int M, int d, const RowDesc* rows, const void* tok, const void* pos, float* x,
                  const float* in_rows, hipStream_t st);
template <class S>
void launch_layernorm(int M, int d, const float* x, const void* g, const void* b, float* out,
                      hipStream_t st);
void launch_argmax(int M, int V, const float* logits, size_t ld, const RowDesc* rows, int* greedy,
                   float* margin, int* err, hipStream_t st);
void launch_accept(int B, int k_max, const SeqDesc* seqs, const int* tokens, const int* greedy,
                   int* accept_len, int* out_tokens, hipStream_t st);
void launch_commit(int B, int* kv_len, const int* accept_len, hipStream_t st);
// Draft trees: the accept scan walks the tree (parents non-NULL) and records the path.
void launch_accept_tree(int B, int k_max, const SeqDesc* seqs, const int* tokens, const int* parents,
                        const int* greedy, int* accept_len, int* out_tokens, int* out_path,
                        hipStream_t st);
// Moves the keys / values of each accepted tree path node j (block row path[j]) to cache
// slot n + j, for every layer (before the commit moves the length).
template <class S>
void launch_kv_compact(int B, int L, int H, const int* kv_len, const int* accept_len, const int* path,
                       int path_stride, void* pool, int num_pages, const int* block_table,
                       int pages_per_seq, hipStream_t st);
// Logical [L][2][n][H][64] <-> paged pool copy of sequence b's positions 0..n-1.
template <class S>
void launch_kv_copy(bool to_linear, int L, int H, int n, int b, void* lin, void* pool, int num_pages,
                    const int* block_table, int pages_per_seq, int* err, hipStream_t st);
void launch_gather_hidden(int B, int d, int layout, int k_max, const int* cu_rows,
                          const int* accept_len, const float* hidden, float* hsel, hipStream_t st);
void launch_assemble_next(int B, int n_heads, int k_max, const int* accept_len, const int* out_tokens,
                          const int* head_greedy, int* next_tokens, hipStream_t st);

// C = A W^T (+ bias) with the epilogue `epi`; A is float32 [M][K], W is [N][K] of S.
template <class S>
void launch_gemm_valu(int epi, int M, int N, int K, const float* A, const void* W, const void* bias,
                      const EpiArgs& e, hipStream_t st);

// Cross-attention keys / values of a bf16 model's encoder states on the matrix cores:
// cache <- enc [M][K] W [N][K]^T + bias in the cross-K/V layout of `layer` (N = 2d, M a
// multiple of 32).  a_packed: enc as written by launch_pack_rows; w_packed: W tiled by
// launch_pack_weight; otherwise row-major.
void launch_xkv_mfma(int M, int N, int K, const uint16_t* A, bool a_packed, const uint16_t* W,
                     bool w_packed, const uint16_t* bias, uint16_t* cache, int layer, int H, int d,
                     int frames_cap, hipStream_t st);
// Row-major bf16 [M][K] (M a multiple of 16, K of 32) into the fragment order the
// prefill reads (M * K elements).
void launch_pack_rows(const uint16_t* A, int M, int K, uint16_t* P, hipStream_t st);

// bf16 matrix-core product: X (A-fragment order, RT row tiles, RT a multiple of 16)
// times W^T.
struct GemmArgs {
  int M, N, K, RT;
  const uint16_t* A;
  const uint16_t* W;     // [N][K] row-major, or tiled by pack_weight (packed = 1)
  int packed;
  const uint16_t* bias;
  int S, KB, ntiles, mchunks;  // set by the launcher
  float* part;           // split-K partial products [S][M][N]
  EpiArgs e;
};
// epi = EPI_PARTIAL (split-K partial products into `part`), EPI_GELU (unsplit; bias +
// GELU into e.frag in A-fragment order) or EPI_ARGMAX (LM head: per-tile top-2 records
// into e.am_part, optional logits into e.out).
void launch_gemm_mfma(int epi, GemmArgs g, hipStream_t st);
// Weight tiling read by the matrix-core GEMM: for each 128-column tile and 32-wide K step
// one contiguous 8 KB stage, in the order the kernel stages it (column tile, lane, 8 k).
// Columns past N are zero.  Elements of the tiled copy of an N x K matrix:
size_t packed_weight_elems(int N, int K);
void launch_pack_weight(const uint16_t* W, int N, int K, uint16_t* P, hipStream_t st);
void launch_argmax_final(int M, int nrec, const void* part, const RowDesc* rows, int* greedy,
                         float* margin, int* err, hipStream_t st);
int gemm_splits(int N, int K);
int gemm_launch_splits(int epi, int N, int K);
size_t gemm_part_floats(int M, int N, int K);
int lm_records(int V);

// Matrix-core attention over bf16 caches; output in A-fragment order.
constexpr int kAttnORow = 68;                  // floats per query row of a chunk's output
constexpr int kAttnPart = 16 + 16 + 16 * kAttnORow;   // per chunk: max, sum, O [16][68]
constexpr int kSelfChunk = 128;                // keys per wave, self-attention
constexpr int kCrossChunk = 384;               // frames per wave, cross-attention
constexpr int kMaxBlockRows = 64;              // bf16 path: rows (k + 1) per sequence
struct AttnArgs {
  int H, d, layer, cross;
  const SeqDesc* seqs;
  // the block's queries (and for self-attention its keys and values) arrive as the
  // split-K partial products of the projection: qkv_part[s][m][n], n in [0, qkv_n)
  const float* qkv_part;
  int qkv_splits, qkv_n, rows;
  const uint16_t* qkv_bias;
  uint16_t* out;
  int out_RT;
  const uint16_t* kv;
  int num_pages;
  const int* block_table;
  int pages_per_seq, frames_cap;
  int chunk, max_chunks, qgroups;   // max_chunks waves per workgroup (at most 8)
  // self-attention, padded row layout: rows per sequence (sequence b's rows start at
  // b * row_stride); 0 when the rows are packed (their start comes from the descriptor)
  int row_stride;
  float* q_save;   // cross-attention only, may be NULL: the finished queries, [rows][d]
  const RowTree* tree;   // self-attention of a draft-tree block (NULL: causal block)
  // cross-attention at the anchor layer, may be NULL: every query row's scores
  // [rows][H][score_ld] (keys past the sequence: -inf) and softmax (max, sum) [rows][H]
  float* score_out;
  float2* stat_out;
  int score_ld;
  unsigned long long* best_clear;   // [B] zeroed here for the readout's merge (or NULL)
};
void launch_attn_mfma(const AttnArgs& a, int B, hipStream_t st);

// Verification-attention anchor readout: for every valid sequence, block row a_b's
// cross-attention weights at one layer (recomputed from the saved queries and the
// layer's keys), averaged over heads; the frame with the largest average.
constexpr int kAnchorChunk = 384;   // frames per workgroup of the score kernel
struct AnchorArgs {
  const SeqDesc* seqs;
  const int* accept_len;
  const float* q;          // [rows][d] finished queries of the layer
  const void* kv;          // cross K/V cache
  int layer, H, d, frames_cap, max_frames, nchunks;
  float* score;            // scratch [B][H][max_frames]
  float2* stats;           // scratch [B][H][nchunks]: (max, sum of exp(score - max))
  int* out_anchor;         // [B]
  float* out_peak;         // [B] or NULL
  const int* path;         // draft trees: [B][path_stride] accepted nodes (NULL: linear)
  int path_stride;
  // 1: the scores were kept by the anchor layer's cross-attention, per block row:
  // score [rows][H][score_ld], stats [rows][H] (max, sum); only the pick kernel runs
  int fused, score_ld;
  unsigned long long* best;   // fused: [B] merged (weight bits, ~frame), 0 between steps
};
// scratch of the readout for B sequences and `rows` block rows: the scores' part, then
// scores + statistics (either layout)
size_t anchor_score_floats(int rows, int B, int H, int max_frames);
int anchor_score_ld(int max_frames);
// The AnchorDraft training objective over B sequences of R padded rows (row t of
// sequence b is b * R + t; M = B * R).
struct LossArgs {
  int B, R, M, H, d, V, layer, frames_cap, max_frames, nchunk, g_ld;
  const uint16_t* kv;          // cross K/V cache (bf16)
  const int* enc_len;
  const int* enc_off;
  const float* xq;             // [M][d] the layer's cross-attention queries, or NULL
  const int* center;           // [M] aligned frame, -1 for none
  float sigma, lam;
  const float* logits;         // [M][V] or NULL
  const int* targets;          // [M] next token, -1 for none (or NULL)
  const float* feat;           // [M][d] predicted features, or NULL
  const float* feat_target;    // [M][d]
  // workspace
  float2* stats;               // [M][H] softmax (max, sum)
  float* Z;                    // [M] Gaussian normalisers
  float* gq;                   // [M][g_ld] g = -q / (H Abar) per row and frame
  float* lpart;                // [M][nchunk] cross-entropy partials per 32-frame block
  float* lrow;                 // [M] each row's cross-entropy
  float* tok_row;              // [M]
  float* feat_row;             // [M]
  int* rowflag;                // [M] bit 0 aligned, bit 1 has a next token
  int* counts;                 // [2] |V|, |T|
  // outputs
  float* out_terms;            // [4] L, L_tok, L_feat, L_anchor
  float* out_row;              // [M] or NULL
  float* out_dxq;              // [M][d] or NULL
  float* out_dlogits;          // [M][V] or NULL
  float* out_dfeat;            // [M][d] or NULL
  int* err;
};
int loss_chunks(int max_frames);
void launch_anchordraft_loss(const LossArgs& a, hipStream_t st);
size_t anchor_scratch_floats(int rows, int B, int H, int max_frames);
template <class S>
void launch_anchor(const AnchorArgs& a, int B, hipStream_t st);

// LayerNorm of float32 rows into A-fragment order (hi/lo bf16) for the next product,
// and optionally also as float32 rows (out may be NULL).
template <class S>
void launch_layernorm_frag(int M, int d, const float* x, const void* g, const void* b,
                           uint16_t* frag, int RT, float* out, hipStream_t st);
void launch_zero_i32(int* p, int n, hipStream_t st);
// bf16 model: x += sum of split-K partials + bias, then LayerNorm -> A fragments (and out).
void launch_reduce_res_ln(int M, int d, int nsplit, const float* P, const void* bias, float* x,
                          const void* g, const void* b, uint16_t* frag, int RT, float* out,
                          hipStream_t st);
// bf16 model: embedding (or in_rows, as in launch_embed) fused with the first LayerNorm.
void launch_embed_ln(int M, int d, const RowDesc* rows, const void* tok, const void* pos, float* x,
                     const float* in_rows, const void* g, const void* b, uint16_t* frag, int RT,
                     hipStream_t st);
// Draft-block input rows: Z[b] = [f_b ; E_tok[token_b]] with f_b either the fused target
// features (computed by the caller into feat) or the previous step's output; and the
// four target representations of sequence b's last verified row gathered into
// taps4[b] = [taps_0 ; taps_1 ; taps_2 ; hidden] (see ad_draft_input).
void launch_draft_gather_taps(int B, int d, int layout, int k_max, const int* cu_rows,
                              const int* accept_len, int rows, const float* taps,
                              const float* hidden, float* taps4, hipStream_t st);
void launch_draft_concat(int B, int d, const float* feat, const void* tok_emb, int bf16,
                         const int* tokens, int token_stride, const int* token_index, float* z,
                         hipStream_t st);
void launch_draft_window(int B, const int* anchor, const int* enc_len, int half, int* window,
                         hipStream_t st);
// The same inputs for the matrix-core product: written in A-fragment order (RT row tiles)
// instead of float32 rows.
void launch_draft_gather_taps_frag(int B, int d, int layout, int k_max, const int* cu_rows,
                                   const int* accept_len, int rows, const float* taps,
                                   const float* hidden, uint16_t* frag, int RT, hipStream_t st);
void launch_draft_concat_frag(int B, int d, const float* feat, const void* tok_emb,
                              const int* tokens, int token_stride, const int* token_index,
                              uint16_t* frag, int RT, hipStream_t st);
// out[m][n] = sum_s P[s][m][n] (split order) + bias[n], float32 rows.
void launch_sum_partials_bias(int M, int N, int nsplit, const float* P, const void* bias, float* out,
                              hipStream_t st);

// Attention of every block row over the paged self cache (causal inside the block) or
// over the sequence's encoder frames.  q and out are float32 [rows][d]; part is scratch
// of attn_valu_part_floats(M, H, G) floats, G = attn_valu_groups(the longest key range:
// max_pos for self-attention, max_frames for cross-attention).
int attn_valu_groups(int max_keys);
inline size_t attn_valu_part_floats(int M, int H, int G) { return (size_t)M * H * G * (2 + 64); }
template <class S>
void launch_self_attn_valu(int B, int M, int H, int d, int layer, const SeqDesc* seqs, const RowDesc* rows,
                           const float* q, float* part, int G, float* out, const void* pool, int num_pages,
                           const int* block_table, int pages_per_seq, const RowTree* tree, hipStream_t st);
template <class S>
void launch_cross_attn_valu(int B, int M, int H, int d, int layer, const SeqDesc* seqs, const RowDesc* rows,
                            const float* q, float* part, int G, float* out, const void* cross, int frames_cap,
                            hipStream_t st);

}  // namespace ad
