// Small kernels of the round: RMSNorm, embedding gathers, conditioning gather,
// acceptance / rollback, and state set-up.
#pragma once
#include "common.h"

namespace rt {

// Per-sequence round state, one int32 array of kStateFields per sequence.
enum StateField : int {
  ST_SEQ_LEN = 0,    // anchor position P = number of valid target KV rows
  ST_ANCHOR,         // last committed token (block row 0 of the next draft)
  ST_R,              // first rejected block position of the last round (A + 1)
  ST_COND_LEN,       // rows conditioned in the next draft (B - r, or 0)
  ST_BUDGET,         // tokens still to generate
  ST_ROUND_POS,      // P of the round just verified (context-append base)
  ST_APPEND,         // rows of that round to append to the drafter context (A + 1, or 0)
  ST_ACCEPT,         // A of the last round
  ST_ROUND,          // rounds (or target-only steps) completed: the round of the random draws
  kStateFields
};

// Pending k-slab partials of a GEMM whose residual add was deferred to the next norm:
// slab z of row r is part[z * part_stride + r * ldx ..]; cap (optional) receives the
// updated row, packed, at column offset cap_k0 (group stride ldcap).
struct NormFold {
  const float* part; int n_part; size_t part_stride;
  void* cap; int ldcap; int cap_k0;
};
// out: packed GEMM-operand layout with group stride ldg; keep: optional row-major copy.
// With fold.n_part > 0 the partials are summed and added to x first (x is updated).
template <typename T, typename K>
void rmsnorm(float* x, int ldx, const T* w, int d, float eps, int rows, T* out, int ldg,
             K* keep, int ldk, const NormFold& fold, hipStream_t s);
template <typename T>
void embed_rows(const T* embed, int d, const int32_t* tokens, int rows, float* x, int ldx, hipStream_t s);
// Drafter input without gated conditioning: row (s, 0) = E[anchor], rows (s, j>0) =
// E[mask], except that with hD given the conditioned rows 1..cond_len take the aligned
// drafter states m_j = hD[s][r + j] instead (the overwrite ablation of Table 3).
// etilde (a second copy of the rows) may be null.
template <typename T, typename K>
void embed_block(const T* embed, int d, const int32_t* state, int mask_token, int n_seqs, int bk, const K* hD,
                 float* x, float* etilde, int ldx, hipStream_t s);
// Verify input: row (s, 0) = E[anchor], row (s, i) = E[draft token i]; also records the
// draft tokens (decoded from the drafter's argmax keys unless `forced`).
template <typename T>
void embed_verify(const T* embed, int d, const int32_t* state, const uint64_t* dkeys, int forced,
                  int32_t* dtok, int n_seqs, int bk, float* x, int ldx, hipStream_t s);
// Conditioning gather (Eq.5/6): mu = [m | u] rows, er[:, :d] = e rows (both packed fp32,
// group stride ldg).  raw != 0 (gated fusion of the uncorrected signal): er[:, d:2d] = m
// rows and mu is left untouched.
template <typename T, typename K>
void cond_prep(const T* embed, int d, const int32_t* state, int mask_token, const K* hD, const K* hT,
               int n_seqs, int bk, float* mu, float* er, int ldg, int raw, hipStream_t s);
// Low-rank conditioning path: latent rank, correction rank, and the width of the latent
// GEMM's output rows ([A m ; C_down [m; u]]).
constexpr int kLowRankLatent = 64;
constexpr int kLowRankCorr = 32;
constexpr int kLowRankLat = kLowRankLatent + kLowRankCorr;
// x / etilde rows from the latent GEMM output lat [rows][kLowRankLat] (see misc.hip).
template <typename T>
void lowrank_fuse(const float* lat, const T* cup, const T* V, const T* G, const float* ge, float beta, const T* embed,
                  int d, const int32_t* state, int mask, int n_seqs, int bk, float* x, float* etilde, hipStream_t s);
// ge = W_g[:, :d] E[mask] from the unpacked [d][2d] gate weight.
template <typename T>
void lowrank_gate_bias(const T* wg, const T* embed, int d, int mask, float* ge, hipStream_t s);
void accept(int32_t* state, const int32_t* dtok, const uint64_t* tkeys, int32_t* ttok, int n_seqs,
            int bk, int32_t* out_tokens, int32_t* out_n, int32_t* out_a, hipStream_t s);
// Target-only greedy step commit for n_seqs (<= 1024) sequences: tokens go to column
// *step of out (row stride ld_out), then *step is advanced.
// sampled (may be null): the step's drawn tokens per sequence instead of the argmax keys.
void ar_commit(int32_t* state, const uint64_t* tkeys, const int32_t* sampled, int n_seqs, int32_t* out, int ld_out,
               int32_t* step, hipStream_t s);
void set_ints(int32_t* dst, int n, int v0, int v1, int v2, int v3, hipStream_t s);
// sampled (may be null): drawn first tokens per sequence instead of the argmax key.
void first_token(int32_t* state, int seq, const uint64_t* keys, const int32_t* sampled, int prompt_len, int budget,
                 int32_t* first_out, hipStream_t s);
void fill_zero(void* p, size_t bytes, hipStream_t s);
// Plain read of bytes (a multiple of 16) at p by `grid` workgroups of 256 threads.
void stream_read(const void* p, size_t bytes, int grid, uint32_t* sink, hipStream_t s);

}  // namespace rt
