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
};

// Where a GEMM's epilogue sends its output.
enum Epi : int {
  EPI_STORE = 0,   // out[m][n] = acc + bias                  (float32)
  EPI_RESID = 1,   // out[m][n] += acc + bias                 (residual stream)
  EPI_GELU = 2,    // out[m][n] = GELU(acc + bias)            (float32)
  EPI_QKV = 3,     // n < d: q; d <= n < 3d: key / value into the paged cache
  EPI_XKV = 4,     // cross-K/V prefill: n < d key, else value, into the cross cache
};

struct EpiArgs {
  float* out;
  size_t ldo;
  // cache writes
  const RowDesc* rows;
  void* cache;
  const int* block_table;
  int pages_per_seq, num_pages, H, d, layer, frames_cap;
};

void launch_prep(const StepArgs& a, SeqDesc* seqs, RowDesc* rows, int* err, hipStream_t st);
template <class S>
void launch_embed(int M, int d, const RowDesc* rows, const void* tok, const void* pos, float* x,
                  hipStream_t st);
template <class S>
void launch_layernorm(int M, int d, const float* x, const void* g, const void* b, float* out,
                      hipStream_t st);
void launch_argmax(int M, int V, const float* logits, size_t ld, const RowDesc* rows, int* greedy,
                   float* margin, int* err, hipStream_t st);
void launch_accept(int B, int k_max, const SeqDesc* seqs, const int* tokens, const int* greedy,
                   int* accept_len, int* out_tokens, hipStream_t st);
void launch_commit(int B, int* kv_len, const int* accept_len, hipStream_t st);
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

// The same product with a bf16 A operand (encoder states of a bf16 model).
void launch_gemm_valu_bf16a(int epi, int M, int N, int K, const void* A, const void* W, const void* bias,
                            const EpiArgs& e, hipStream_t st);

// Attention of every block row over the paged self cache (causal inside the block) or
// over the sequence's encoder frames.  q and out are float32 [rows][d].
template <class S>
void launch_self_attn_valu(int B, int H, int d, int layer, const SeqDesc* seqs, const float* q,
                           float* out, const void* pool, int num_pages, const int* block_table,
                           int pages_per_seq, hipStream_t st);
template <class S>
void launch_cross_attn_valu(int B, int H, int d, int layer, const SeqDesc* seqs, const float* q,
                            float* out, const void* cross, int frames_cap, hipStream_t st);

}  // namespace ad
