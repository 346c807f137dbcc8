// Weight-streaming / tiled bf16 (or fp32) MFMA GEMM  Y = X * W^T  with fused epilogues.
//
// Weights are pre-packed once into 16(n) x 32(k) tiles laid out in MFMA lane order
// (tile (nt, kt) at ((nt * KT) + kt) * 512 elements; lane l holds n = l % 16,
// k = (l / 16) * 8 .. +8), so every wave-wide load of a weight tile is one
// contiguous 1 KiB (bf16) read.  A workgroup of four waves owns a
// (WM*MT*16) x (WN*NT*16) output tile; its k range may be split across
// `ksplit` workgroups whose fp32 partials are summed, in split order, by the
// last workgroup to finish (a per-tile arrival counter), which then runs the
// epilogue on the complete tile.
#pragma once
#include "common.h"

namespace rt {

enum EpiKind : int {
  EPI_STORE_F32 = 0,   // out_f32[m][n] = y
  EPI_STORE_ACT,       // out_act[m][n] = T(y)
  EPI_RESID,           // resid[m][n] += y; optional capture cap[m][n] = T(resid)
  EPI_SWIGLU,          // interleaved gate/up 16-column tiles: out_act[m][n/2] = T(silu(g) * u)
  EPI_ARGMAX,          // keys[m] = max(keys[m], (y, n)); optional out_f32 logits
  EPI_QKV,             // q/k/v heads: per-head RMSNorm + RoPE, q -> out_act, k/v -> paged caches
  EPI_COND_R,          // r = m + beta * y  -> out_f32 (the corrected signal, Eq.8)
  EPI_COND_GATE,       // out_f32 = sigmoid(y)                               (Eq.9 gate)
  EPI_COND_OUT,        // x = e + y * gate on conditioned rows, e elsewhere  (Eq.9)
};

struct EpiArgs {
  int kind;
  int M, N;                      // valid output extent
  // generic outputs
  float* out_f32; void* out_act; int ldo;
  float* resid; int ldr;
  void* cap; int ldcap;          // capture (act type), may be null
  uint64_t* keys;                // argmax keys per row
  // per-row sequence mapping
  int rows_per_seq;              // row m belongs to sequence m / rows_per_seq, block row m % rows_per_seq
  int seq_stride;                // int32 stride between sequences in pos0 / nrows / anchor / cond_len
  const int32_t* pos0;           // [seq] absolute position of block row 0
  const int32_t* nrows;          // [seq] number of valid block rows (null: all)
  // QKV epilogue
  int q_cols, kv_cols;           // column regions [0,q) q, [q,q+kv) k, [q+kv,q+2kv) v (repeats per layer)
  int head_dim, n_kv_heads;
  int layer_cols;                // columns per layer block (q + 2 kv) when several layers share a GEMM
  const void* q_norm; const void* k_norm; int norm_layer_stride;
  void* kcache; void* vcache; size_t cache_layer_stride;   // elements
  const int32_t* page_table; int max_pages;
  const float* rope;             // [pos][hd/2] cos followed by [pos][hd/2] sin at rope + max_pos*hd/2
  int rope_max_pos;
  float eps;
  // conditioning
  const float* cond_m; int ld_cond_m;     // m rows (fp32) for EPI_COND_R
  float beta;
  const float* gate; int ld_gate;
  const void* embed; int mask_token;      // e rows are embedding rows (anchor at block row 0)
  const int32_t* anchor; const int32_t* cond_len;
  float* etilde;                          // copy of the conditioned inputs
};

struct GemmArgs {
  const void* A; int lda; int a_rows;     // A rows allocated (loads are clamped below it)
  const void* B; int Kp;                  // packed weights, K padded to a multiple of 32
  int ksplit;
  float* partial; uint32_t* counters;
  EpiArgs e;
};

// Host-side launch helpers (implemented in gemm.hip).
template <typename T>
void pack_weights(const T* W, int N, int K, int Kp, T* out, hipStream_t s);
template <typename T>
void pack_interleaved(const T* Wa, const T* Wb, int N, int K, int Kp, T* out, hipStream_t s);

enum GemmShape : int { SHAPE_SKINNY = 0, SHAPE_WIDE = 1 };
template <typename T>
hipError_t gemm(const GemmArgs& a, int shape, bool a_f32, hipStream_t s);
int gemm_tile_cols(int shape);
int gemm_tile_rows(int shape);

}  // namespace rt
