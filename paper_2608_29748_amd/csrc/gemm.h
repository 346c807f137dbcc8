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
  EPI_SWIGLU,          // gate|up 8-column halves of each 16-column tile: out_act[m][n/2] = T(silu(g) * u)
  EPI_COND_R,          // r = m + beta * y  -> out_f32 (the corrected signal, Eq.8)
  EPI_COND_GATE,       // out_f32 = sigmoid(y)                               (Eq.9 gate)
  EPI_COND_OUT,        // x = e + y * gate on conditioned rows, e elsewhere  (Eq.9)
  EPI_PARTIAL,         // k slab z of a split reduction: out_f32[z * part_stride + m * ldo + n] = y
  EPI_ARGMAX,          // per row, (max, lowest column) key of each half workgroup -> part_keys;
                       // optional fp32 logits out_f32[m * ldo + n] (mid-size kernel only)
};

struct EpiArgs {
  int kind;
  int M, N;                      // valid output extent
  // generic outputs: out_f32 row-major with ldo, except EPI_COND_R (packed, ldo = group
  // stride, columns offset by out_k0); out_act always packed (ldo = group stride)
  float* out_f32; void* out_act; int ldo; int out_k0;
  size_t part_stride;            // EPI_PARTIAL: elements between the slabs of consecutive k splits
  uint64_t* part_keys;           // EPI_ARGMAX: [2 * gridDim.x][M] keys
  float* resid; int ldr;
  void* cap; int ldcap; int cap_k0;   // packed capture of the updated residual (act type), may be null
  // per-row sequence mapping
  int rows_per_seq;              // row m belongs to sequence m / rows_per_seq, block row m % rows_per_seq
  int seq_stride;                // int32 stride between sequences in pos0 / nrows / anchor / cond_len
  const int32_t* pos0;           // [seq] absolute position of block row 0
  const int32_t* nrows;          // [seq] number of valid block rows (null: all)
  // conditioning
  const float* cond_m; int ld_cond_m;     // m rows (packed fp32, group stride) for EPI_COND_R
  float beta;
  const float* gate; int ld_gate;
  const void* embed; int mask_token;      // e rows are embedding rows (anchor at block row 0)
  const int32_t* anchor; const int32_t* cond_len;
  float* etilde;                          // copy of the conditioned inputs
};

struct GemmArgs {
  const void* A; int lda; int a_rows;     // packed A: lda = group stride (elements); rows allocated
  const void* B; int Kp;                  // packed weights, K padded to a multiple of 32
  int ksplit;                             // wide: k splits summed by the last workgroup; skinny:
                                          // k slabs, only with EPI_PARTIAL (one slab per grid z)
  float* partial; uint32_t* counters;
  size_t partial_floats;                  // capacity of `partial`
  EpiArgs e;
};

// Per-head post-processing of a fused q|k|v projection (fp32 [M][layers*(q+2kv)]):
// q and k get a per-head RMSNorm and rotate-half RoPE at their absolute position; q is
// stored to q_out, k and v to the paged caches (K [page][kv head][token][hd], V
// [page][kv head][hd][token]).  q_cols = 0 processes k|v blocks only (one per layer).
struct QkvPostArgs {
  const float* src; int lds;
  int M;
  int q_cols, kv_cols, layer_cols, n_layers;
  int head_dim, n_kv_heads;
  void* q_out; int ldq;
  const void* q_norm; const void* k_norm; int norm_layer_stride;
  void* kcache; void* vcache; size_t cache_layer_stride;
  const int32_t* page_table; int max_pages;
  const float* rope; int rope_max_pos;
  float eps;
  int rows_per_seq, seq_stride;
  const int32_t* pos0; const int32_t* nrows;
  int n_part; size_t part_stride;   // n_part > 1: src holds k-slab partials, summed in slab order
};

// LM head with a fused argmax: logits = X * W^T over the vocabulary; each workgroup
// reduces its columns to one (value, index) key per row in part_keys[wg][M]
// (max value, lowest index among equal values), reduced by argmax_reduce.
struct LmHeadArgs {
  const void* A; int lda; int a_rows; int M;   // packed A (lda = group stride)
  const void* B; int N; int Kp;
  uint64_t* part_keys;             // [gridDim.x][M]
  float* logits; int ldl;          // optional fp32 logits
};
int lmhead_grid(int N);
constexpr int kLmGrid = 512;   // LDS-staged LM head: two workgroups per CU on 256 CUs (K <= 2560)
// Partial-key rows (workgroups) of one lm_head launch over M rows, and an upper bound
// over every launch for a vocabulary of N.
int lmhead_parts(int M, int N, int Kp, int elem_bytes);
int lmhead_max_parts(int N);

// Host-side launch helpers (implemented in gemm.hip).
template <typename T>
void pack_weights(const T* W, int N, int K, int Kp, T* out, hipStream_t s);
template <typename T>
void pack_interleaved(const T* Wa, const T* Wb, int N, int K, int Kp, T* out, hipStream_t s);

enum GemmShape : int { SHAPE_SKINNY = 0, SHAPE_WIDE = 1 };
// SHAPE_SKINNY: M <= 32 (and 33..64 with bf16 operands), 16, 32 or 64-row tiles, the k
// range split across the workgroup's waves and reduced in LDS (no ksplit except k slabs
// with EPI_PARTIAL).  SHAPE_WIDE: 128x128 tiles, optional ksplit.
// SHAPE_WIDE with bf16 storage goes to the mid-size kernel (gemm_mid.hip) for 33..512
// rows; otherwise (fp32 storage, more rows) 128x128 tiles.
template <typename T>
hipError_t gemm(const GemmArgs& a, int shape, bool a_f32, hipStream_t s);
bool gemm_mid_supports(const GemmArgs& a);
hipError_t gemm_mid(const GemmArgs& a, bool a_f32, hipStream_t s);
// k slabs the mid-size kernel would use for a GEMM with a stored (non-partial)
// epilogue of this shape (1: none); a caller that adds the slabs itself requests them
// with EPI_PARTIAL and this count
int gemm_mid_store_slabs(const GemmArgs& a, bool a_f32);
// k slabs (1..max_slabs) for a GEMM whose fp32 slab partials a later kernel adds: the
// count that fills the chip in the fewest rounds of the cost model
int gemm_mid_partial_slabs(const GemmArgs& a, bool a_f32, int max_slabs);
// Columns per workgroup of the mid-size kernel's argmax (LM head) launch over N columns
// and M rows; it writes two partial keys per workgroup and row.
int gemm_mid_cols(int N, int M);
// Sums ks fp32 slabs part[z][M][N] (row-major, slab stride M*N) in slab order and runs
// epilogue e on the result.
template <typename T>
hipError_t gemm_split_epilogue(const EpiArgs& e, const float* part, int ks, hipStream_t s);
template <typename T>
hipError_t qkv_post(const QkvPostArgs& a, hipStream_t s);
template <typename T>
hipError_t lm_head(const LmHeadArgs& a, hipStream_t s);
// keys[m] = max over part_keys[0..nparts)[m]; optional token ids
hipError_t argmax_reduce(const uint64_t* part_keys, int nparts, int M, uint64_t* keys, hipStream_t s);

}  // namespace rt
