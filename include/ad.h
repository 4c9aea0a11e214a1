/*
 * ad.h -- C-ABI of libad.so: the batched speculative-verify step for single-model
 * speculative decoding of a Whisper-shape ASR decoder on MI355X (gfx950).
 *
 * Method (paper, section 3 "Speculative Loop"): in each round the target scores a
 * drafted block [t0, d_1..d_k] in one decoder pass, takes its greedy token g_i at every
 * block row and keeps the longest draft prefix with d_i = g_{i-1}; the round emits the
 * a accepted drafts plus the target's own token g_a, so it advances 1 + a tokens
 * (appendix "Cost derivation").  The accepted tokens and their cached keys/values feed
 * the next round (appendix "Real cached loop").
 *
 * Conventions for every entry point:
 *  - All pointers named "device" are HIP device pointers owned by the caller; the
 *    library never allocates or frees device memory on the step path and never keeps a
 *    pointer past the call (except the parameter views held by an ad_model).
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and is
 *    asynchronous: nothing is synchronised and nothing is read back to the host.
 *  - Validate-then-enqueue: host-detectable errors (NULL pointers, bad enums, sizes out
 *    of range, workspace too small) return a negative ad_status and enqueue nothing.
 *  - Device-detectable errors (a token id outside the vocabulary, a page index outside
 *    the pool, a per-sequence length out of range, non-finite logits) OR a bit into
 *    *err_flag; the affected sequence is skipped: its cache is not written and its
 *    accept length is -1.  err_flag must be zeroed by the caller before a round.
 *  - ad_last_error() returns a thread-local description of the last failure.
 *  - Calls that overlap on one stream are ordered; calls on different streams that
 *    share buffers race and are the caller's responsibility.
 *
 * Storage: dtype AD_F32 stores parameters, encoder states and caches in float32;
 * AD_BF16 stores them in bfloat16.  Activations (the residual stream, LayerNorm,
 * attention and GELU outputs, scores, logits) are float32 in both cases; bf16 matrix
 * products accumulate in float32.
 */
#ifndef AD_H_
#define AD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AD_OK = 0,
  AD_EINVAL = -1,        /* NULL pointer, unknown enum, inconsistent descriptor      */
  AD_ERANGE = -2,        /* a size outside its allowed range                        */
  AD_ENOSPACE = -3,      /* workspace smaller than ad_workspace_size() requires      */
  AD_EHIP = -4,          /* a HIP launch or runtime call failed                      */
  AD_EUNSUPPORTED = -5   /* shape the kernels do not support (e.g. head width != 64) */
} ad_status;

typedef enum { AD_F32 = 0, AD_BF16 = 1 } ad_dtype;

/* Row layout of a verify step.  PADDED: sequence b owns rows b*(k_max+1) ..
 * b*(k_max+1)+k_max and rows past its own k_b are padding.  PACKED: sequence b owns
 * rows cu_rows[b] .. cu_rows[b+1]-1 and cu_rows[b+1]-cu_rows[b] = k_b + 1. */
typedef enum { AD_PADDED = 0, AD_PACKED = 1 } ad_layout;

/* device-side error bits OR-ed into *err_flag */
#define AD_ERR_LENGTH 1   /* k_b, n_b + k_b + 1 or packed row counts out of range */
#define AD_ERR_PAGE 2     /* block-table entry outside [0, num_pages)              */
#define AD_ERR_TOKEN 4    /* token id outside [0, vocab)                           */
#define AD_ERR_FRAMES 8   /* T_b outside [1, max_frames] or past frames_cap        */
#define AD_ERR_NONFINITE 16 /* NaN/Inf logits at a valid row                       */
#define AD_ERR_TREE 32    /* draft-tree parent not an earlier row of the block     */

#define AD_HEAD_DIM 64    /* every attention head is 64 wide (score scale 1/8)     */
#define AD_PAGE_TOKENS 16 /* tokens per self-KV page                               */

typedef struct {
  int32_t n_layers;   /* L                                                        */
  int32_t d_model;    /* d = 64 * n_heads                                         */
  int32_t n_heads;    /* H                                                        */
  int32_t d_ffn;      /* F                                                        */
  int32_t vocab;      /* V                                                        */
  int32_t max_pos;    /* learned positions (448 for the Whisper shape)            */
  int32_t max_frames; /* encoder frames per sequence (1500 for the Whisper shape) */
  int32_t dtype;      /* ad_dtype                                                 */
} ad_model_desc;

typedef struct ad_model ad_model;

/* Number of parameter pointers ad_model_create expects: 4 + 20 * n_layers. */
int32_t ad_model_param_count(const ad_model_desc* desc);

/*
 * Create a model handle holding non-owning views of caller-allocated device parameters
 * (all of the model dtype, row-major, matrices stored [out_features][in_features]).
 * params[] order:
 *   0 tok_emb [V][d] (also the tied LM head)   1 pos_emb [max_pos][d]
 *   2 lnf_g [d]   3 lnf_b [d]
 *   then per layer l, at 4 + 20 l:
 *   +0 ln1_g [d]  +1 ln1_b [d]  +2 w_qkv [3d][d] (rows q | k | v)  +3 b_qkv [3d]
 *   +4 w_o [d][d] +5 b_o [d]
 *   +6 ln2_g [d]  +7 ln2_b [d]  +8 w_xq [d][d]  +9 b_xq [d]
 *   +10 w_xkv [2d][d] (rows k | v) +11 b_xkv [2d]  +12 w_xo [d][d]  +13 b_xo [d]
 *   +14 ln3_g [d] +15 ln3_b [d] +16 w_1 [F][d]  +17 b_1 [F]  +18 w_2 [d][F]  +19 b_2 [d]
 * The decoder is pre-LN: x += SelfAttn(LN1 x); x += CrossAttn(LN2 x);
 * x += W2 GELU(W1 LN3 x + b1) + b2; logits = LN_f(x) tok_emb^T (the paper's
 * Whisper-large-v3 target, appendix "Whisper Cross-Architecture Check").
 * Every parameter pointer must be 16-byte aligned (kernels load 16-byte vectors).
 * Errors: AD_EINVAL (NULL, wrong n_params, bad dtype, misaligned pointer),
 * AD_EUNSUPPORTED (d != 64 H, H > 64, F not a multiple of 64, max_frames > 2048,
 * max_pos > 1024), AD_ERANGE (non-positive sizes).
 */
ad_status ad_model_create(const ad_model_desc* desc, const void* const* params,
                          int32_t n_params, ad_model** out);
ad_status ad_model_destroy(ad_model* model);

/*
 * Optional weight tiling for the bf16 matrix-core path.  ad_model_pack_size gives the
 * bytes of a caller-allocated device buffer; ad_model_pack fills it with a tiled copy of
 * every projection matrix (the encoder K/V projection included) and of the tied LM
 * head (for each 128-column tile and 32-wide
 * K step, one contiguous 8 KB block in the order the kernels stage it) and makes the
 * model read its weights from there.  The buffer must stay allocated and unchanged while
 * the model is used; pack again after changing the parameters.  buffer = NULL returns
 * the model to its row-major parameters.  Results are bit-identical either way; the
 * tiled copy streams from HBM in whole contiguous blocks.
 * Errors: AD_EINVAL (NULL model, buffer not 256-byte aligned), AD_ENOSPACE (bytes too
 * small), AD_EUNSUPPORTED (float32 model).
 */
ad_status ad_model_pack_size(const ad_model* model, size_t* bytes);
ad_status ad_model_pack(ad_model* model, void* buffer, size_t bytes, void* stream);

/*
 * Paged self-attention KV cache.  pool holds
 *   n_layers * 2 * num_pages * n_heads * 16 * 64 elements of the model dtype
 * arranged as [layer][K|V][page][head][16-token tile]; the element order inside a tile
 * is private to the library (write it only through ad_verify_step / ad_kv_import).
 * Sequence b's position p lives in page block_table[b * pages_per_seq + p / 16].
 */
typedef struct {
  void* pool;                 /* device                                              */
  int32_t num_pages;
  int32_t pages_per_seq;      /* row stride of block_table; >= ceil(max_pos / 16)   */
  int32_t* kv_len;            /* device [B]: committed length n_b                    */
  const int32_t* block_table; /* device [B][pages_per_seq]                           */
} ad_kv;

/*
 * Encoder keys/values (the decoder's view of the frozen audio encoding, computed once
 * per utterance by ad_cross_kv_prefill).  data holds
 *   n_layers * 2 * n_heads * frames_cap * 64 elements of the model dtype
 * arranged as [layer][head][32-frame block][K|V] (private order within a block: the
 * operand order of the attention products).
 * Sequence b uses slots enc_off[b] .. enc_off[b] + enc_len[b] - 1; enc_off[b] must be
 * a multiple of 32 (AD_ERR_FRAMES otherwise).  PADDED encoders use enc_off[b] =
 * b * T_max, PACKED ones a running sum of T_b rounded up to 32; both give identical
 * results.
 */
typedef struct {
  void* data;                 /* device                                              */
  int32_t frames_cap;         /* multiple of 32                                      */
  const int32_t* enc_len;     /* device [B]: T_b                                     */
  const int32_t* enc_off;     /* device [B]                                          */
} ad_cross;

typedef struct {
  int32_t batch;              /* B >= 1                                              */
  int32_t layout;             /* ad_layout                                           */
  int32_t k_max;              /* max draft length, 0 <= k_max < max_pos and
                                 k_max <= 63 (AD_EUNSUPPORTED otherwise)               */
  int32_t rows;               /* PADDED: B*(k_max+1); PACKED: sum_b (k_b + 1)        */
  const int32_t* tokens;      /* device [rows]: per sequence t0, d_1 .. d_{k_b}      */
  const int32_t* k;           /* device [B]: k_b in [0, k_max]                       */
  const int32_t* cu_rows;     /* device [B+1] (PACKED only; NULL for PADDED)         */
  ad_kv kv;
  ad_cross cross;
  int32_t* accept_len;        /* device [B] out: a_b, or -1 for a skipped sequence   */
  int32_t* out_tokens;        /* device [B][k_max+1] out: g_0..g_{a_b}, then -1      */
  int32_t* out_greedy;        /* device [rows] out (optional): g at every row        */
  float* out_logits;          /* device [rows][vocab] out (optional)                 */
  float* out_hidden;          /* device [rows][d] out (optional): LN_f output        */
  float* out_margin;          /* device [rows] out (optional): top-1 minus top-2     */
  int32_t* err_flag;          /* device [1]: AD_ERR_* bits are OR-ed in              */
  void* workspace;            /* device scratch, >= ad_workspace_size() bytes, 256-byte aligned */
  size_t workspace_bytes;
  /* Verification-attention anchor readout (optional; paper, section "Correction and
   * Cost", paragraph "Verification-Attention Correction", and appendix "Runtime
   * Correction"): with 0 <= anchor_layer < n_layers, after the accept scan the
   * cross-attention weights of block row a_b (the last verified position) at that layer
   * are recomputed from the layer's queries and key cache, averaged over the heads, and
   * out_anchor[b] receives the frame 0 .. T_b - 1 with the largest average (lowest index
   * on ties; -1 for a skipped sequence), out_anchor_peak[b] (optional) that average.
   * anchor_layer = -1 turns the readout off (out_anchor may then be NULL).           */
  int32_t anchor_layer;
  int32_t* out_anchor;        /* device [B] out                                      */
  float* out_anchor_peak;     /* device [B] out (optional)                           */
  /* Running the audio-conditioned draft block (see ad_draft_input), all optional:
   * in_rows replaces every row's token embedding (the position embedding of the row's
   * position is still added; tokens are still validated and scanned); cross_window[b] =
   * {lo, hi} restricts sequence b's cross-attention to frames lo .. hi - 1 (0 <= lo < hi
   * <= T_b, else AD_ERR_FRAMES; the anchor readout always covers every frame); out_taps
   * receives, for each tap_layers[i] >= 0, the residual stream after that layer at every
   * row (the four target representations the draft reads are these three and
   * out_hidden).                                                                     */
  const float* in_rows;       /* device [rows][d_model] (optional), 16-byte aligned  */
  const int32_t* cross_window; /* device [B][2] (optional)                           */
  int32_t tap_layers[3];      /* layer indices, -1 for none                          */
  float* out_taps;            /* device [3][rows][d_model] out (optional)            */
  /* Draft trees (optional; paper, appendix "Tree-decoder implementation check": all
   * nodes of a candidate tree verified in one pass under a tree attention mask).  With
   * parents given, block row i >= 1 of sequence b is a tree node whose parent is row
   * p = parents[row0_b + i] of the same block, 0 <= p < i (AD_ERR_TREE otherwise; the
   * entry of row 0, the root holding the pending token, is ignored).  Node i sits at
   * position n_b + depth(i) and attends to the committed cache, its ancestors and
   * itself; its keys / values go to cache slot n_b + i.  The accept scan walks from the
   * root, each time to the lowest-index child whose token equals the current node's
   * greedy token: a_b = the number of moves, out_tokens[b] = the greedy tokens along the
   * path, out_path[b][j] = the path's j-th row (0 = root) for j <= a_b, then -1.  The
   * anchor readout uses row out_path[b][a_b].  Commit with ad_kv_commit_tree, which also
   * moves the path's keys / values to slots n_b .. n_b + a_b.  A chain (parents[i] =
   * i - 1) gives exactly the results of parents = NULL.                               */
  const int32_t* parents;     /* device [rows] (optional)                            */
  int32_t* out_path;          /* device [B][k_max+1] out (required with parents)     */
  /* The cross-attention query rows of layer anchor_layer at every row (optional, needs
   * anchor_layer >= 0): the input of ad_anchordraft_loss when the step runs the draft
   * block over training positions.                                                  */
  float* out_xq;              /* device [rows][d_model] out (optional)               */
} ad_step;

/* Bytes of workspace a step with up to max_rows rows, max_batch sequences and draft
 * length up to k_max needs. */
ad_status ad_workspace_size(const ad_model* model, int32_t max_rows, int32_t max_batch,
                            int32_t k_max, size_t* bytes);

/*
 * Setup, once per utterance (not part of the per-round step): project encoder states
 * into every layer's cross-attention keys and values,
 *   K_l = enc W_xk,l^T,  V_l = enc W_xv,l^T + b_xv,l
 * (the decoder reuses the encoded audio at every step; paper, section 1 and appendix
 * "Draft architecture").  enc is device [frames_cap][d] of the model dtype, sequence b
 * at rows enc_off[b].. (rows outside any sequence are projected too and never read).
 * cross->data is written only; with two or more layers its last layer's part also
 * serves as scratch for a copy of enc (bf16 models) before that layer is written, so
 * enc must not lie inside it.  A tiled model (ad_model_pack) reads its tiled weights.
 * Errors: AD_EINVAL, AD_ERANGE (frames_cap not a positive multiple of 32).
 */
ad_status ad_cross_kv_prefill(const ad_model* model, const void* enc, const ad_cross* cross,
                              void* stream);

/*
 * The verify step (paper, section 3 "Speculative Loop"): embed the block of every
 * sequence at positions n_b .. n_b + k_b, run the decoder over it with self-attention
 * causal inside the block and over the committed cache, write the block's keys/values
 * into the cache (write-through), take g_i = argmax of the float32 logits (lowest index
 * on ties) at every row, accept a_b = max{ j <= k_b : d_i = g_{i-1} for all i <= j } and
 * emit g_0..g_{a_b}.  kv_len is not changed; call ad_kv_commit next.
 * Requires n_b + k_b + 1 <= max_pos, 1 <= T_b <= max_frames.
 * Errors: AD_EINVAL, AD_ERANGE, AD_ENOSPACE, AD_EHIP (see conventions above).
 */
ad_status ad_verify_step(const ad_model* model, const ad_step* step, void* stream);

/*
 * ad_verify_step without a caller workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  step->workspace and step->workspace_bytes are ignored; the step runs in
 * a library-owned static device buffer of 64 MiB (AD_STATIC_SCRATCH_BYTES) that every
 * GPU the library runs on holds until the process ends.  Nothing is allocated or freed
 * by the call.  The results are those of ad_verify_step with a workspace (same kernels).
 * Every call on one GPU shares that GPU's buffer: calls that overlap on one GPU (on
 * different streams, or from different threads) race and give undefined results.  The
 * large-v3 bench step (224 rows, 32 sequences, k_max 6) needs 45.7 MiB.
 * Errors: as ad_verify_step; AD_ENOSPACE when ad_workspace_size() of the step exceeds
 * AD_STATIC_SCRATCH_BYTES; AD_EHIP if the buffer's device address cannot be obtained.
 */
#define AD_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
ad_status ad_verify_step_static(const ad_model* model, const ad_step* step, void* stream);

/*
 * Input rows of the audio-conditioned draft block (paper, section 3 "Models and
 * Protocol": an EAGLE-3 style drafter that also attends to the encoder output;
 * appendix "Draft architecture": the input mixes four target feature vectors with the
 * current token's embedding ahead of a single causal block).  For every sequence b
 *   out[b] = W_in [f_b ; E_tok[t_b]] + b_in                         (float32 [B][d])
 * where f_b = W_fuse [taps_0 ; taps_1 ; taps_2 ; hidden] + b_fuse at sequence b's last
 * verified row of a target step when `taps` is given (a round's first draft step; the
 * row is row accept_len[b] of the step's layout, described by layout / k_max / cu_rows /
 * rows; taps is the step's out_taps [3][rows][d] and hidden its out_hidden), else
 * f_b = feature[b] (later steps: the draft block's previous out_hidden row, [B][d]).
 * t_b = tokens[b * token_stride + (token_index ? token_index[b] : 0)]; a round's first
 * token is the target step's out_tokens[b][a_b] (tokens = out_tokens, token_stride =
 * k_max + 1, token_index = accept_len).  With `anchor` given, window[b] receives
 * {max(0, c - half_window), min(T_b, c + half_window + 1)} around c = anchor[b] (the
 * verification-attention anchor; T_b from enc_len), the draft block's cross_window.
 * W_fuse [d][4d], W_in [d][2d], b_fuse, b_in: device arrays of the target's dtype; the
 * token table is the target's.  Skipped sequences (accept_len < 0) get zero features.
 * workspace: device, >= ad_draft_input_workspace_size() bytes, 256-byte aligned.
 * Errors: AD_EINVAL (NULL argument, bad layout, misaligned workspace), AD_ERANGE (batch
 * < 1, rows < batch, token_stride < 1, half_window < 0), AD_ENOSPACE (workspace too
 * small).
 */
ad_status ad_draft_input_workspace_size(const ad_model* target, int32_t batch, size_t* bytes);
ad_status ad_draft_input(const ad_model* target, const void* w_fuse, const void* b_fuse,
                         const void* w_in, const void* b_in, int32_t batch, const float* taps,
                         const float* hidden, int32_t layout, int32_t k_max,
                         const int32_t* cu_rows, const int32_t* accept_len, int32_t rows,
                         const float* feature, const int32_t* tokens, int32_t token_stride,
                         const int32_t* token_index, const int32_t* anchor,
                         const int32_t* enc_len, int32_t half_window, int32_t* window,
                         float* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Commit / roll back (appendix "Real cached loop"): kv_len[b] += accept_len[b] + 1 for
 * every sequence with accept_len[b] >= 0.  Slots past the new length hold rejected
 * drafts; they are never read and are overwritten by the next round.
 */
ad_status ad_kv_commit(int32_t* kv_len, const int32_t* accept_len, int32_t batch, void* stream);

/*
 * Commit after a draft-tree step (paper, appendix "Tree-decoder implementation check"):
 * for every sequence with accept_len[b] >= 0, the keys / values of accepted path node j
 * (written at slot n_b + path[b * path_stride + j]) are moved to slot n_b + j, every
 * layer and head, for j = 1 .. accept_len[b] (in path order: path rows increase, so no
 * slot is overwritten before it is read), then kv_len[b] += accept_len[b] + 1.  The
 * cache then holds what a chain step over the path's tokens would have written.  path
 * is the step's out_path (path_stride = k_max + 1); kv is the step's cache.
 * Errors: AD_EINVAL (NULL argument), AD_ERANGE (batch, path_stride or the cache sizes
 * not positive).
 */
ad_status ad_kv_commit_tree(const ad_model* model, const ad_kv* kv, const int32_t* accept_len,
                            const int32_t* path, int32_t path_stride, int32_t batch, void* stream);

/*
 * The AnchorDraft training objective (paper, section "Correction and Cost", paragraph
 * "AnchorDraft Training Objective"; appendix "Training Correction with AnchorDraft",
 * eq. anchordraft-supp) over `batch` sequences of rows_per_seq padded rows (row t of
 * sequence b is b * rows_per_seq + t), for a bf16 draft model whose layer `layer` (its
 * first) attends to the audio in `cross` (the draft's own ad_cross_kv_prefill):
 *   A_{t,hj}  = softmax over frames j < T_b of (xq_{t,h} . k_{h,j}) / 8
 *   Abar_t(j) = (1/H) sum_h A_{t,hj}
 *   q_t(j)    = exp(-(j - c_t)^2 / (2 sigma^2)) / sum_{l < T_b} exp(-(l - c_t)^2 / (2 sigma^2))
 *   L_anchor  = -(1/|V|) sum_{t in V} sum_{j < T_b} q_t(j) log Abar_t(j)
 *   L_tok     = (1/|T|) sum_{t in T} (logsumexp(z_t) - z_t[y_t])
 *   L_feat    = (1/(|T| d)) sum_{t in T} sum_i smoothL1(feat_t,i - feat_target_t,i), beta 1
 *   L         = L_tok + 0.5 L_feat + lambda L_anchor
 * with V the rows whose center is >= 0 and T the rows whose target is >= 0 (the paper
 * selects lambda = 0.1, sigma = 5).  Device inputs: xq [rows][d] the layer's
 * cross-attention query rows (ad_step.out_xq; NULL leaves the alignment term out),
 * center [rows] (aligned frame in 0 .. T_b - 1, -1 for none), logits [rows][vocab] and
 * feat / feat_target [rows][d] (optional), targets [rows] (next token, -1 for none;
 * required with logits or feat).  Device outputs: out_terms[4] = {L, L_tok, L_feat,
 * L_anchor}; optional out_row [rows] (-sum_j q_t(j) log Abar_t(j), 0 without
 * alignment), out_dxq [rows][d] = dL/dxq, out_dlogits [rows][vocab] = dL/dlogits and
 * out_dfeat [rows][d] = dL/dfeat.  A centre outside [-1, T_b) or a sequence with bad
 * frames sets AD_ERR_FRAMES, a target outside [-1, vocab) AD_ERR_TOKEN; those rows are
 * left out.  Sums run in a fixed order (repeatable results).
 * workspace: device, >= ad_anchordraft_loss_workspace_size() bytes, 256-byte aligned.
 * Errors: AD_EINVAL (NULL argument, a missing companion input or a misaligned
 * workspace), AD_ERANGE (sizes, layer, sigma <= 0, lambda < 0), AD_ENOSPACE,
 * AD_EUNSUPPORTED (float32 model).
 */
ad_status ad_anchordraft_loss_workspace_size(const ad_model* draft, int32_t batch,
                                             int32_t rows_per_seq, size_t* bytes);
ad_status ad_anchordraft_loss(const ad_model* draft, const ad_cross* cross, int32_t layer,
                              int32_t batch, int32_t rows_per_seq, const float* xq,
                              const int32_t* center, float sigma, float lambda,
                              const float* logits, const int32_t* targets, const float* feat,
                              const float* feat_target, float* out_terms, float* out_row,
                              float* out_dxq, float* out_dlogits, float* out_dfeat,
                              int32_t* err_flag, void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Next draft block from linear draft heads on the final hidden state.  For sequence b
 * take the LN_f output h at row row0_b + a_b (row0_b = first row of b in `layout`),
 * d_i = argmax(W_i h) (float32 logits, lowest index on ties), i = 1..n_heads, and write
 *   next_tokens[b][0] = out_tokens[b][a_b] (the bonus token, the next pending token)
 *   next_tokens[b][i] = d_i
 * heads_w is device [n_heads][vocab][d] of the model dtype.  hidden is the out_hidden
 * of the step ([rows][d] float32).  Sequences with accept_len < 0 get -1 everywhere.
 * workspace: device, >= ad_draft_heads_workspace_size() bytes, 256-byte aligned.
 * Errors: AD_EINVAL (NULL argument, misaligned workspace), AD_ERANGE, AD_ENOSPACE.
 */
ad_status ad_draft_heads(const ad_model* model, const void* heads_w, int32_t n_heads,
                         const float* hidden, int32_t layout, int32_t k_max,
                         const int32_t* cu_rows, const int32_t* accept_len,
                         const int32_t* out_tokens, int32_t batch, int32_t* next_tokens,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace ad_draft_heads needs for n_heads heads over `batch` sequences. */
ad_status ad_draft_heads_workspace_size(const ad_model* model, int32_t n_heads, int32_t batch,
                                        size_t* bytes);

/*
 * Import a committed prefix into the cache: src is device [L][2][n][H][64] (keys then
 * values, model dtype, logical order) and becomes positions 0..n-1 of sequence b.
 * Errors: AD_EINVAL, AD_ERANGE (n > pages_per_seq * 16 or n > max_pos);
 * a page index outside the pool sets AD_ERR_PAGE and writes nothing.
 */
ad_status ad_kv_import(const ad_model* model, const ad_kv* kv, int32_t b, const void* src,
                       int32_t n, int32_t* err_flag, void* stream);

/*
 * Export positions 0..n-1 of sequence b from the cache into dst, device
 * [L][2][n][H][64] (the layout ad_kv_import reads): a snapshot of the decode state that
 * a later ad_kv_import restores.  Errors as for ad_kv_import.
 */
ad_status ad_kv_export(const ad_model* model, const ad_kv* kv, int32_t b, void* dst,
                       int32_t n, int32_t* err_flag, void* stream);

/*
 * Per-kernel timing with HIP events recorded on the step's stream.  After
 * ad_profile_enable(model, kernel, max_launches), every launch of that kernel class made
 * by ad_verify_step on this model is bracketed by a start/stop event pair (up to
 * max_launches pairs; later launches are not timed).  ad_profile_read waits for the
 * recorded events, returns the summed duration in milliseconds and the number of timed
 * launches, and clears the record.  max_launches = 0 disables timing and frees the
 * events.  Host-side state of the model handle: not thread-safe.
 * An event recorded between two kernels delays the second one's start by the launch
 * latency the stream otherwise hides (a few microseconds); the two pair classes bracket
 * the cross-attention query projection with and without the cross-attention kernel that
 * follows it, so the difference of their means is that kernel's duration alone.
 */
#define AD_PROF_CROSS_ATTN 1  /* cross-attention over the encoder K/V              */
#define AD_PROF_SELF_ATTN 2   /* self-attention over the paged cache               */
#define AD_PROF_GEMM 3        /* the per-layer projections                         */
#define AD_PROF_LM_HEAD 4     /* LM head with the fused argmax                     */
#define AD_PROF_XQ_CROSS 5    /* cross-attention query projection + cross-attention */
#define AD_PROF_XQ 6          /* cross-attention query projection alone             */
#define AD_PROF_ANCHOR 7      /* the anchor readout's two kernels (bf16 models)     */
ad_status ad_profile_enable(ad_model* model, int32_t kernel, int32_t max_launches);
ad_status ad_profile_read(ad_model* model, double* total_ms, int32_t* launches);

/* Thread-local text of the last error (never NULL). */
const char* ad_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* AD_H_ */
