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

// Finds, from the top, the bin where the suffix count reaches `need` among nb bins of
// hist (nb / kDistThreads consecutive bins per thread).  Returns the bin in *bin and the
// count of the bins above it in *above.
template <int NB>
__device__ void suffix_find(const uint32_t* hist, uint32_t need, uint32_t* part, int* bin, uint32_t* above) {
  constexpr int PER = NB / kDistThreads;
  const int t = threadIdx.x;
  uint32_t mine = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) mine += hist[t * PER + j];
  part[t] = mine;
  __syncthreads();
  // inclusive suffix sums of the per-thread counts (Hillis-Steele over 256 entries)
  for (int o = 1; o < kDistThreads; o <<= 1) {
    const uint32_t v = t + o < kDistThreads ? part[t + o] : 0u;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  const uint32_t incl = part[t];            // counts of threads t.. (bins >= t*PER)
  const uint32_t excl = incl - mine;        // bins above this thread's range
  if (excl < need && incl >= need) {
    uint32_t acc = excl;
    for (int j = PER - 1; j >= 0; --j) {
      const uint32_t h = hist[t * PER + j];
      if (acc + h >= need) {
        *bin = t * PER + j;
        *above = acc;
        break;
      }
      acc += h;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kDistThreads) void filtered_dist_kernel(DistArgs a) {
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t part[kDistThreads];
  __shared__ int s_bin;
  __shared__ uint32_t s_above, s_ngt, s_base;
  __shared__ uint64_t cand[kMaxTopK];
  __shared__ uint32_t wcnt[kDistThreads / 64];
  const int row = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const float* z = a.logits + (size_t)row * a.ldl;
  const int V = a.V, K = a.top_k;

  if (t == 0) { s_bin = 0; s_above = 0u; }
  __syncthreads();
  // radix selection of the K-th largest orderable key: 12, 12 and 8 bits
  uint32_t prefix = 0u, mask = 0u, need = (uint32_t)K;
  const int shifts[3] = {20, 8, 0}, widths[3] = {12, 12, 8};
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass], nb = 1 << widths[pass];
    for (int b = t; b < nb; b += kDistThreads) hist[b] = 0u;
    __syncthreads();
    for (int i = t; i < V; i += kDistThreads) {
      const uint32_t k = orderable(z[i]);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> sh) & (nb - 1)], 1u);
    }
    __syncthreads();
    if (nb == 4096) suffix_find<4096>(hist, need, part, &s_bin, &s_above);
    else suffix_find<256>(hist, need, part, &s_bin, &s_above);
    prefix |= (uint32_t)s_bin << sh;
    mask |= (uint32_t)(nb - 1) << sh;
    need -= s_above;
    __syncthreads();
  }
  // prefix is now the K-th largest key: K - need keys lie above it, and the `need`
  // lowest indices holding it complete the set; n_eq keys hold it in all
  const uint32_t n_eq = hist[s_bin];
  if (t == 0) { s_ngt = 0u; s_base = 0u; }
  __syncthreads();
  const uint32_t n_gt = (uint32_t)K - need;
  if (n_eq == need) {
    // every key at or above the K-th is taken: no ordering by index needed
    for (int i = t; i < V; i += kDistThreads) {
      const uint32_t k = orderable(z[i]);
      if (k >= prefix) {
        const uint32_t slot = atomicAdd(&s_ngt, 1u);
        if (slot < (uint32_t)kMaxTopK) cand[slot] = ((uint64_t)k << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
      }
    }
  } else {
    // ties at the K-th key: rank the tied indices in index order
    for (int i0 = 0; i0 < V; i0 += kDistThreads) {
      const int i = i0 + t;
      const uint32_t k = i < V ? orderable(z[i]) : 0u;
      if (i < V && k > prefix) {
        const uint32_t slot = atomicAdd(&s_ngt, 1u);
        if (slot < n_gt) cand[slot] = ((uint64_t)k << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
      }
      const bool eq = i < V && k == prefix;
      const uint64_t bal = __ballot(eq);
      if (lane == 0) wcnt[w] = (uint32_t)__popcll(bal);
      __syncthreads();
      uint32_t before = s_base;
      for (int v = 0; v < w; ++v) before += wcnt[v];
      const uint32_t rank = before + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
      if (eq && rank < need) cand[n_gt + rank] = ((uint64_t)k << 32) | (uint64_t)(0xffffffffu - (uint32_t)i);
      __syncthreads();
      if (t == 0) s_base += wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
      __syncthreads();
    }
  }
  __syncthreads();

  if (w != 0) return;
  // wave 0: sort the K keys (value descending, index ascending), then the distribution
  uint64_t key = lane < K ? cand[lane] : 0ull;
#pragma unroll
  for (int k2 = 2; k2 <= 64; k2 <<= 1)
#pragma unroll
    for (int j = k2 >> 1; j > 0; j >>= 1) {
      const uint64_t o = __shfl_xor(key, j, 64);
      const bool keep_max = ((lane & k2) == 0) == ((lane & j) == 0);
      key = keep_max ? (key > o ? key : o) : (key < o ? key : o);
    }
  const bool valid = lane < K;
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

hipError_t filtered_dists(const DistArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.top_k < 1 || a.top_k > kMaxTopK || a.top_k > a.V || a.ldd < kMaxTopK) return hipErrorInvalidValue;
  RT_LAUNCH(filtered_dist_kernel, dim3(a.rows), dim3(kDistThreads), 0, s, a);
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
