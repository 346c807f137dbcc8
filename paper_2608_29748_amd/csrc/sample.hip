// Temperature sampling of speculative rounds (standard lossless speculative sampling
// with the paper's temperature-1 settings, Section 5): filtered distributions, draws
// from a counter-based generator, and the acceptance rule.
#include "misc.h"
#include "sample.h"

namespace rt {

// ------------------------------------------------------------------ counter-based draws
// Philox4x64 with ten rounds (two 64 x 64 -> 128-bit multiplies and a Weyl key step per
// round), counter (round, sequence, purpose, position), key (seed, 0); word 0 of the
// block, top 53 bits, scaled to [0, 1).
__device__ __forceinline__ double philox_uniform(uint64_t seed, uint64_t rnd, uint64_t seq, uint64_t purpose,
                                                 uint64_t pos) {
  uint64_t c0 = rnd, c1 = seq, c2 = purpose, c3 = pos, k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
    const uint64_t h0 = __umul64hi(m0, c0), l0 = m0 * c0;
    const uint64_t h1 = __umul64hi(m1, c2), l1 = m1 * c2;
    const uint64_t n0 = h1 ^ c1 ^ k0, n2 = h0 ^ c3 ^ k1;
    c0 = n0; c1 = l1; c2 = n2; c3 = l0;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  return (double)(c0 >> 11) * (1.0 / 9007199254740992.0);
}

__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ float wave_scan_f(float v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// ------------------------------------------------------------------ filtered distributions

constexpr int kDistThreads = 256;
constexpr int kChunk = kSelectChunk;

// key of logit i: orderable value above, (0xffffffff - i) below, so that the larger
// key is the larger logit and, among equal logits, the lower id; 0 marks padding
__device__ __forceinline__ uint64_t logit_key(float v, int i) {
  return ((uint64_t)orderable(v) << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
}
__device__ __forceinline__ uint64_t kmax(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t kmin(uint64_t a, uint64_t b) { return a < b ? a : b; }

// Sorts one key per lane into decreasing order across the wave (bitonic network).
__device__ __forceinline__ uint64_t wave_sort_desc(uint64_t v, int lane) {
#pragma unroll
  for (int k2 = 2; k2 <= 64; k2 <<= 1)
#pragma unroll
    for (int j = k2 >> 1; j > 0; j >>= 1) {
      const uint64_t o = __shfl_xor(v, j, 64);
      v = (((lane & k2) == 0) == ((lane & j) == 0)) ? kmax(v, o) : kmin(v, o);
    }
  return v;
}
// The 64 largest of two decreasing wave lists, decreasing: the elementwise maximum of
// one list and the other reversed is a bitonic sequence holding exactly those keys,
// which the half-cleaner cascade then sorts.
__device__ __forceinline__ uint64_t wave_merge_top(uint64_t list, uint64_t batch_sorted, int lane) {
  uint64_t m = kmax(list, __shfl(batch_sorted, 63 - lane, 64));
#pragma unroll
  for (int j = 32; j > 0; j >>= 1) {
    const uint64_t o = __shfl_xor(m, j, 64);
    m = ((lane & j) == 0) ? kmax(m, o) : kmin(m, o);
  }
  return m;
}

// Stage 1: workgroup (c, row) keeps the 64 largest keys of logits c*kChunk .. of its row:
// each wave folds batches of 64 logits into a running top-64, then wave 0 folds the
// other waves' lists and stores its top_k keys.
__global__ __launch_bounds__(kDistThreads) void topk_chunk_kernel(DistArgs a, uint64_t* cand, int n_chunks) {
  __shared__ uint64_t lists[kDistThreads / 64][64];
  const int c = blockIdx.x, row = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const float* z = a.logits + (size_t)row * a.ldl;
  const int i0 = c * kChunk, i1 = min(a.V, i0 + kChunk);
  uint64_t top = 0ull;
  for (int b = i0 + w * 64; b < i1; b += kDistThreads) {
    const int i = b + lane;
    const uint64_t k = i < i1 ? logit_key(z[i], i) : 0ull;
    top = wave_merge_top(top, wave_sort_desc(k, lane), lane);
  }
  lists[w][lane] = top;
  __syncthreads();
  if (w != 0) return;
  for (int v = 1; v < kDistThreads / 64; ++v) top = wave_merge_top(top, lists[v][lane], lane);
  if (lane < a.top_k) cand[((size_t)row * n_chunks + c) * kMaxTopK + lane] = top;
}

// Stage 2: one wave per row folds the chunks' candidates into the row's top_k keys,
// forms the filtered distribution from them and, per mode, draws one token.
__global__ __launch_bounds__(64) void filtered_dist_kernel(DistArgs a, const uint64_t* cand, int n_chunks) {
  const int row = blockIdx.x, lane = threadIdx.x;
  const float* z = a.logits + (size_t)row * a.ldl;
  const int K = a.top_k;
  const int n_cand = n_chunks * K;
  uint64_t key = 0ull;
  for (int b = 0; b < n_cand; b += 64) {
    const int j = b + lane;
    const uint64_t k = j < n_cand ? cand[((size_t)row * n_chunks + j / K) * kMaxTopK + j % K] : 0ull;
    key = wave_merge_top(key, wave_sort_desc(k, lane), lane);
  }
  // the K largest keys in order (value descending, index ascending)
  const bool valid = lane < K && key != 0ull;
  const int id = valid ? key_index(key) : -1;
  const float lg = valid ? z[id] : 0.f;
  const float l0 = __shfl(lg, 0, 64);
  const float e = valid ? expf((lg - l0) * a.inv_temp) : 0.f;
  const float pk = e / wave_sum_f(e);
  const float cum = wave_scan_f(pk, lane);
  const int below = (int)__popcll(__ballot(valid && cum < a.top_p));
  const int n = below + 1 < K ? below + 1 : K;        // shortest prefix reaching top_p
  const bool kept = lane < n;
  const float pz = wave_sum_f(kept ? pk : 0.f);
  const float p = kept ? pk / pz : 0.f;
  a.ids[(size_t)row * a.ldd + lane] = kept ? id : -1;
  a.probs[(size_t)row * a.ldd + lane] = p;

  if (a.mode == SAMPLE_NONE || !a.tok_out) return;
  int s = 0, pos = 0, purpose = U_STEP;
  if (a.mode == SAMPLE_DRAFT) {
    s = row / a.bk;
    pos = row % a.bk;
    purpose = U_DRAFT;
    if (pos == 0) return;                   // the anchor row proposes nothing
  } else if (a.mode == SAMPLE_FIRST) {
    s = a.seq0;
    purpose = U_FIRST;
  } else {
    s = row;
  }
  const int32_t* st = a.state + (size_t)s * a.state_stride;
  const uint64_t rnd = a.mode == SAMPLE_FIRST ? 0ull : (uint64_t)(st[ST_ROUND] + 1);
  const double u = philox_uniform(a.seed, rnd, (uint64_t)s, (uint64_t)purpose, (uint64_t)pos);
  const float c2 = wave_scan_f(p, lane);
  int j = (int)__popcll(__ballot(kept && (double)c2 <= u));
  if (j > n - 1) j = n - 1;
  const int tok = __shfl(id, j, 64);
  if (lane == 0) a.tok_out[a.mode == SAMPLE_DRAFT ? row : s] = tok;
}

int topk_chunks(int V) { return (V + kChunk - 1) / kChunk; }

hipError_t filtered_dists(const DistArgs& a, uint64_t* cand, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.top_k < 1 || a.top_k > kMaxTopK || a.top_k > a.V || a.ldd < kMaxTopK) return hipErrorInvalidValue;
  const int nc = topk_chunks(a.V);
  RT_LAUNCH(topk_chunk_kernel, dim3(nc, a.rows), dim3(kDistThreads), 0, s, a, cand, nc);
  RT_LAUNCH(filtered_dist_kernel, dim3(a.rows), dim3(64), 0, s, a, cand, nc);
  return hipGetLastError();
}

// ------------------------------------------------------------------ acceptance
__global__ __launch_bounds__(64) void accept_sampled_kernel(AcceptSampleArgs a) {
  const int sq = blockIdx.x, lane = threadIdx.x;
  const int bk = a.bk, B = bk - 1;
  int32_t* st = a.state + (size_t)sq * a.state_stride;
  const size_t r0 = (size_t)sq * bk;
  if (lane < bk) a.ttok[r0 + lane] = key_index(a.tkeys[r0 + lane]);
  const int budget = st[ST_BUDGET];
  const uint64_t rnd = (uint64_t)(st[ST_ROUND] + 1);
  int A = B, corr = -1;
  for (int i = 1; i <= B; ++i) {
    const int tok = a.dtok[r0 + i];
    const size_t qrow = (r0 + i) * a.ldd, prow = (r0 + i - 1) * a.ldd;
    const int qid = a.q_ids[qrow + lane], pid = a.p_ids[prow + lane];
    const float qp = a.q_p[qrow + lane], pp = a.p_p[prow + lane];
    const float pt = wave_sum_f(pid == tok ? pp : 0.f), qt = wave_sum_f(qid == tok ? qp : 0.f);
    const double u = philox_uniform(a.seed, rnd, (uint64_t)sq, U_ACCEPT, (uint64_t)i);
    if (u * (double)qt < (double)pt) continue;            // kept with probability min(1, p / q)
    // rejected: the correction comes from the normalised residual max(0, p - q) over
    // p's support, in p's order
    float qx = 0.f;
    for (int m = 0; m < kMaxTopK; ++m) {
      const int qm = __shfl(qid, m, 64);
      const float qpm = __shfl(qp, m, 64);
      if (qm >= 0 && qm == pid) qx = qpm;
    }
    float wgt = pid >= 0 ? fmaxf(pp - qx, 0.f) : 0.f;
    if (wave_sum_f(wgt) <= 0.f) wgt = pid >= 0 ? pp : 0.f;   // p == q: cannot occur in exact arithmetic
    const float tot = wave_sum_f(wgt);
    const float cum = wave_scan_f(wgt, lane);
    const double ur = philox_uniform(a.seed, rnd, (uint64_t)sq, U_RESAMPLE, 0) * (double)tot;
    const uint64_t pos_lanes = __ballot(wgt > 0.f);
    const int last = pos_lanes ? 63 - __builtin_clzll(pos_lanes) : 0;
    int j = (int)__popcll(__ballot(pid >= 0 && (double)cum <= ur));
    if (j > last) j = last;
    corr = __shfl(pid, j, 64);
    if (corr < 0) corr = __shfl(pid, 0, 64);             // p's first entry is always kept
    A = i - 1;
    break;
  }
  if (corr < 0) {                                          // all B kept: bonus from p_{B+1}
    const size_t prow = (r0 + B) * a.ldd;
    const int pid = a.p_ids[prow + lane];
    const float pp = a.p_p[prow + lane];
    const float cum = wave_scan_f(pp, lane);
    const double ur = philox_uniform(a.seed, rnd, (uint64_t)sq, U_RESAMPLE, 0);
    const int n = (int)__popcll(__ballot(pid >= 0));
    int j = (int)__popcll(__ballot(pid >= 0 && (double)cum <= ur));
    if (j > n - 1) j = n - 1;
    if (j < 0) j = 0;
    corr = __shfl(pid, j, 64);
    if (corr < 0) corr = __shfl(pid, 0, 64);
  }
  const int n_new = budget > 0 ? min(A + 1, budget) : 0;
  if (lane < bk) {
    int v = -1;
    if (lane < n_new) v = lane < A ? a.dtok[r0 + lane + 1] : corr;
    a.out_tok[r0 + lane] = v;
  }
  if (lane == 0) {
    a.out_n[sq] = n_new;
    a.out_a[sq] = n_new > 0 ? A : 0;
    if (budget > 0) {
      const int P = st[ST_SEQ_LEN];
      st[ST_ROUND_POS] = P;
      st[ST_APPEND] = A + 1;
      st[ST_ACCEPT] = A;
      st[ST_SEQ_LEN] = P + A + 1;        // rows P+A+1.. of the target KV are rolled back
      st[ST_ANCHOR] = corr;
      st[ST_BUDGET] = budget - n_new;
      st[ST_ROUND] = (int32_t)rnd;
      if (A < B - 1) { st[ST_R] = A + 1; st[ST_COND_LEN] = B - (A + 1); }
      else { st[ST_R] = 0; st[ST_COND_LEN] = 0; }
    } else {
      st[ST_APPEND] = 0;
      st[ST_ROUND_POS] = st[ST_SEQ_LEN];
    }
  }
}

hipError_t accept_sampled(const AcceptSampleArgs& a, int n_seqs, hipStream_t s) {
  if (n_seqs <= 0) return hipSuccess;
  if (a.bk > 64 || a.ldd < kMaxTopK) return hipErrorInvalidValue;
  RT_LAUNCH(accept_sampled_kernel, dim3(n_seqs), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace rt
