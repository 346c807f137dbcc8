// Temperature sampling of speculative rounds: filtered next-token distributions,
// counter-based draws, and the speculative-sampling acceptance rule.
#pragma once
#include "common.h"

namespace rt {

constexpr int kMaxTopK = 64;   // entries of a filtered distribution (one per lane of a wave)
constexpr int kSelectChunk = 8192;   // logits per workgroup of the first top-k stage

// purposes of a random draw (the counter is (round, sequence, purpose, position))
enum DrawPurpose : int { U_DRAFT = 1, U_ACCEPT = 2, U_RESAMPLE = 3, U_FIRST = 4, U_STEP = 5 };

enum SampleMode : int {
  SAMPLE_NONE = 0,    // distributions only (verify rows)
  SAMPLE_DRAFT = 1,   // rows (s, i) of draft blocks: draw block positions i >= 1 into tok_out[row]
  SAMPLE_FIRST = 2,   // one row of sequence `seq0`: the prefill's first token into tok_out[seq0]
  SAMPLE_STEP = 3,    // row s = sequence s: a target-only step into tok_out[s]
};

struct DistArgs {
  const float* logits; int ldl; int V; int rows;   // fp32 logits [rows][ldl]
  int top_k; float inv_temp; float top_p;
  int32_t* ids; float* probs; int ldd;             // outputs [rows][ldd]: kept ids (-1 after), probabilities
  int mode;
  const int32_t* state; int state_stride; int bk; int seq0;
  uint64_t seed;
  int32_t* tok_out;                                // may be null (draft tokens given by the host)
};

// The top_k largest logits of each row (ties to the lowest id) in two stages -- every
// 8192-logit chunk keeps its top_k keys in `cand` ([rows][topk_chunks(V)][kMaxTopK]
// 64-bit keys), then one wave per row folds those -- followed by the filtered
// distribution (temperature, top-k, top-p on the renormalised top-k probabilities)
// and, per mode, one inverse-CDF draw.
int topk_chunks(int V);
hipError_t filtered_dists(const DistArgs& a, uint64_t* cand, hipStream_t s);

struct AcceptSampleArgs {
  int32_t* state; int state_stride;
  const int32_t* dtok;                 // [seq][bk]: anchor, then the B draft tokens
  const int32_t* q_ids; const float* q_p;   // drafter distributions, rows (s, i)
  const int32_t* p_ids; const float* p_p;   // target distributions, rows (s, i)
  int ldd;
  const uint64_t* tkeys; int32_t* ttok;     // target argmax keys -> ttok (diagnostic)
  int bk;
  uint64_t seed;
  int32_t* out_tok; int32_t* out_n; int32_t* out_a;
};
// One wave per sequence: keep draft i with probability min(1, p_i(y_i) / q_i(y_i)),
// stop at the first rejection and draw the correction from the normalised residual
// max(0, p_i - q_i); after B acceptances draw a bonus token from p_{B+1}; commit,
// roll back and carry as in the greedy acceptance.
hipError_t accept_sampled(const AcceptSampleArgs& a, int n_seqs, hipStream_t s);

}  // namespace rt
