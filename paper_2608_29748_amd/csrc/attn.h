// Paged grouped-query attention for blocks of query rows (verify, draft, prefill).
#pragma once
#include "common.h"

namespace rt {

struct AttnArgs {
  const void* q;                 // [row][n_q_heads * head_dim], row = seq * rows_per_seq + token
  const void* kcache;            // this layer: K pages [page][kv head][token][hd]
  const void* vcache;            // this layer: V pages [page][kv head][hd][token]
  const int32_t* page_table; int max_pages;
  const int32_t* pos0;           // [seq * seq_stride] position of query token 0
  const int32_t* nq;             // [seq * seq_stride] valid query tokens (null: rows_per_seq)
  int seq_stride;
  int rows_per_seq;
  int n_seqs;
  int causal;                    // 1: key position <= query position; 0: every key below pos0+nq
  int n_q_heads, n_kv_heads, head_dim;
  int splits;                    // key-range splits per (seq, kv head, row block)
  int row_blocks;                // row blocks of rb_rows (token, head) rows per sequence
  int rb_rows;                   // rows per block: 64, or 96 (bf16) when a sequence has 65..96 rows
  // split partials: per (split, row) the running max and sum (fp32 mlpart) and the
  // split's own normalised output O / sum (opart: fp16 for bf16 models, fp32 otherwise)
  float* opart; float* mlpart;
  int32_t* plan;                 // [2][64] balanced split plan: first partial block, split count per unit
  int span;                      // bf16 kernel without the fused q / k work: balanced launches may
                                 // use the spanning plan (slots cross unit boundaries) when it
                                 // shortens the longest split; 2: whenever it is valid (test hook)
  void* out; int ldo;            // packed GEMM-operand layout of [row][n_q_heads * head_dim]; ldo = group stride
  float scale;                   // 1/sqrt(head_dim)
  // Rounds (at most 16 rows per sequence, one q|k|v slab): the q / k per-head RMSNorm,
  // RoPE and the block's K / V cache write done here instead of by qkv_post.  qkv: the
  // fp32 q|k|v projection [row][ldqkv] (q at column 0, k at q_cols, v at q_cols + kv_cols);
  // null: q comes from `q` and the block's K / V are already cached.  Every workgroup
  // normalises and rotates its own q rows; the workgroups whose chunks hold the block's
  // positions normalise and rotate the block's k rows, write k and v to the caches and
  // into their LDS stages.  Key split 0 of each unit also stores its normalised q rows to
  // q_out ([row][ldq], as qkv_post would).
  const float* qkv; int ldqkv; int q_cols, kv_cols;
  const void* q_norm; const void* k_norm;
  const float* rope; int rope_max_pos; float eps;
  void* q_out; int ldq;
};

// Query (token, head) rows handled by one workgroup: 64, or 96 for bf16 blocks of 65..96
// rows (a GQA group of 5 over a 16-token block), so that every KV head is read once.
constexpr int kAttnRows = 64;
constexpr int kAttnRowsMax = 96;

// attention = attention_partials (per key split) then attention_merge (splits > 1).
template <typename T>
hipError_t attention(const AttnArgs& a, hipStream_t s);
template <typename T>
hipError_t attention_partials(const AttnArgs& a, hipStream_t s);
template <typename T>
hipError_t attention_merge(const AttnArgs& a, hipStream_t s);
size_t attn_partial_floats(int n_seqs, int n_kv_heads, int row_blocks, int splits, int head_dim, int rb_rows);

}  // namespace rt
