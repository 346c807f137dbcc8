// Paged GQA attention with MFMA.  One workgroup owns one sequence, one KV head, one
// block of 64 or 96 (token, head) query rows and one contiguous share of the key range
// (shares sized by the sequence lengths of the batch), walked in 64-key chunks (four
// pages); each wave owns a 16-row MFMA tile of the queries and runs an online softmax.  K pages are stored [token][hd] and V pages
// transposed ([hd][token]), so a K row and a V^T row are contiguous MFMA fragments.
// Split partials (unnormalised O, running max, running sum) are merged by a second
// kernel.
//
// bf16 storage: every wave copies one page of K and one of V per chunk straight from
// HBM into LDS (16-byte direct-to-LDS loads), into a ring of pipeline stages, so the
// copies of the next chunks are in flight while the current one is used; one barrier
// per chunk.  fp32 storage (small configurations): chunks are staged through
// registers.
//
// In rounds and target-only steps (bf16, at most 16 rows per sequence) the same kernel
// also applies the per-head q / k RMSNorm and RoPE to the fp32 q|k|v projection and
// writes the block's K / V rows to the caches (a launch fewer per layer); it rounds
// exactly as the separate post-processing kernel does.
#include "attn.h"

namespace rt {

constexpr int kChunk = 64;      // keys per LDS chunk (four pages)
constexpr int kMaxSplitPages = 1024;   // fp32 path: page ids of one split held in LDS (16384 keys)

// Storage of the split partials' normalised output rows: fp16 for bf16 models (the
// output is rounded to bf16 anyway; fp16 keeps 3 more significand bits), fp32 otherwise.
template <typename T> struct PartOf;
template <> struct PartOf<bf16_t> {
  using P = _Float16;
  // (values are weighted means of V entries; beyond the fp16 range they are clamped)
  __device__ static __forceinline__ _Float16 h(float v) { return (_Float16)fminf(fmaxf(v, -65504.f), 65504.f); }
  __device__ static __forceinline__ void store4(P* p, float a, float b, float c, float d) {
    typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 h4;
    *reinterpret_cast<h4*>(p) = h4{h(a), h(b), h(c), h(d)};
  }
  template <int N>
  __device__ static __forceinline__ void load(const P* p, float (&v)[N]) {
    typedef __attribute__((__vector_size__(N * sizeof(_Float16)))) _Float16 hN;
    const hN x = *reinterpret_cast<const hN*>(p);
#pragma unroll
    for (int e = 0; e < N; ++e) v[e] = (float)x[e];
  }
};
template <> struct PartOf<float> {
  using P = float;
  __device__ static __forceinline__ void store4(P* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
  }
  template <int N>
  __device__ static __forceinline__ void load(const P* p, float (&v)[N]) {
#pragma unroll
    for (int e = 0; e < N; ++e) v[e] = p[e];
  }
};

size_t attn_partial_floats(int n_seqs, int n_kv_heads, int row_blocks, int splits, int head_dim, int rb_rows) {
  return (size_t)n_kv_heads * ((size_t)n_seqs * row_blocks * (splits + 1) - 1) * rb_rows * head_dim;
}

// wave-wide integer reductions and scan of the ROCm device library (DPP based)
extern "C" __device__ int __ockl_wfred_add_i32(int);
extern "C" __device__ int __ockl_wfred_max_i32(int);
extern "C" __device__ int __ockl_wfscan_add_i32(int, bool);

// Key splits.  A work unit is one (sequence, row block), u = seq * row_blocks + rb; the
// workgroups of one KV head are slots 0 .. n_units * splits - 1 (slot = blockIdx.z *
// splits + blockIdx.x), and the partials of slot x of KV head h sit at block
// h * n_slots + x.  Uniform plan: unit u owns slots u*splits .. u*splits + splits-1.
// Balanced plan (2..64 units and splits > 1), for batches of unequal context lengths:
// unit u owns s_u = ceil(n_u / q) consecutive slots, n_u being its number of 64-key
// chunks and q the smallest chunk count per split for which the s_u fit in the slots.
// q never exceeds the uniform plan's ceil(max n_u / splits), so no split is longer than
// under the uniform plan, and s_u <= 64 (one merge lane per split).  Every wave derives
// the plan from the sequence lengths; the workgroup of slot 0 of KV head 0 stores it
// for the merge, which runs after the partial kernel on the same stream.
__device__ __forceinline__ bool attn_balanced(const AttnArgs& a) {
  const int nu = a.n_seqs * a.row_blocks;
  return a.splits > 1 && nu > 1 && nu <= 64;
}
__device__ __forceinline__ int attn_unit_chunks(const AttnArgs& a, int u, int rbr) {
  const int s = u / a.row_blocks, rb = u % a.row_blocks;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int nrows = nq * G, row0 = rb * rbr;
  if (row0 >= nrows) return 0;
  const int P = a.pos0[s * a.seq_stride];
  const int last_tok = min(nrows, row0 + rbr) - 1;
  const int kv_end = a.causal ? P + last_tok / G + 1 : P + nq;
  return (kv_end + kChunk - 1) / kChunk;
}
struct SplitPlan {
  int count;   // lane u: s_u (0 past the units)
  int end;     // lane u: s_0 + .. + s_u
  int q;       // the chunk bound per split
};
// Balanced plan; all 64 lanes of the wave must be active.
__device__ __forceinline__ SplitPlan attn_balanced_plan(const AttnArgs& a, int rbr) {
  const int lane = threadIdx.x & 63;
  const int nu = a.n_seqs * a.row_blocks, slots = nu * a.splits;
  const int n = lane < nu ? attn_unit_chunks(a, lane, rbr) : 0;
  const int tot = __ockl_wfred_add_i32(n), mx = __ockl_wfred_max_i32(n);
  int lo = max(1, max((tot + slots - 1) / slots, (mx + 63) / 64));
  int hi = max(lo, (mx + a.splits - 1) / a.splits);
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (__ockl_wfred_add_i32((n + mid - 1) / mid) <= slots) hi = mid;
    else lo = mid + 1;
  }
  const int cnt = (n + lo - 1) / lo;
  return SplitPlan{cnt, __ockl_wfscan_add_i32(cnt, true), lo};
}
// Work of the workgroup at (blockIdx.x, blockIdx.z): unit, split index within the unit
// and the unit's split count; false for a slot the balanced plan leaves idle.
__device__ __forceinline__ bool attn_slot_work(const AttnArgs& a, int rbr, int& unit, int& split, int& nsplit) {
  if (!attn_balanced(a)) {
    unit = blockIdx.z; split = blockIdx.x; nsplit = a.splits;
    return true;
  }
  const SplitPlan p = attn_balanced_plan(a, rbr);
  const int slot = blockIdx.z * a.splits + blockIdx.x;
  if (slot == 0 && blockIdx.y == 0 && threadIdx.x < 64) {   // hand the plan to the merge
    a.plan[threadIdx.x] = p.end - p.count;
    a.plan[64 + threadIdx.x] = p.count;
  }
  const unsigned long long m = __ballot(slot < p.end);   // units whose slots end past this one
  if (m == 0) return false;
  unit = __builtin_ctzll(m);                                 // the first of them owns it
  nsplit = __builtin_amdgcn_readlane(p.count, unit);
  split = slot - (__builtin_amdgcn_readlane(p.end, unit) - nsplit);
  return true;
}
// Partial blocks per KV head: one per slot, plus one per unit boundary under the
// balanced plans (a spanning slot writes one block per unit it meets).
__device__ __forceinline__ int attn_head_blocks(const AttnArgs& a) {
  const int nu = a.n_seqs * a.row_blocks, slots = nu * a.splits;
  return attn_balanced(a) ? slots + nu - 1 : slots;
}
// First partial block (x) and split count (y) of unit u (merge side): the balanced plan
// as the partial kernel's first workgroup stored it, clamped to this launch's blocks (a
// merge replayed on its own, for timing, may find another launch's plan there).
__device__ __forceinline__ int2 attn_unit_slots(const AttnArgs& a, int u) {
  if (!attn_balanced(a)) return make_int2(u * a.splits, a.splits);
  const int nb = attn_head_blocks(a);
  const int first = min(max(a.plan[u], 0), nb);
  return make_int2(first, min(max(a.plan[64 + u], 0), min(nb - first, 64)));
}
// Spanning plan (bf16 kernel without the fused q / k work; balanced launches): the units'
// chunks are laid end to end, C in all, and slot x takes chunks [b(x), b(x+1)) of that
// sequence, b(x) = floor(x C / S), so every slot gets floor or ceil of C / S chunks.  A
// slot may meet the end of one unit and the start of the next; it then runs one segment
// per unit.  The j-th slot meeting unit u writes partial block seg_first(u) + j.  Usable
// when no unit meets more than 64 slots (one merge lane per split); else the kernel keeps
// the balanced plan.  All 64 lanes of the wave must be active; lane u describes unit u.
struct SpanPlan {
  int start, n;        // unit u's first chunk in the concatenation, its chunk count
  int first, count;    // its first slot, the number of slots meeting it
  int seg_end;         // inclusive prefix sum of count (its blocks end there)
  int total;           // C
  bool ok;             // every count <= 64
};
__device__ __forceinline__ SpanPlan attn_span_plan(const AttnArgs& a, int rbr) {
  const int lane = threadIdx.x & 63;
  const int nu = a.n_seqs * a.row_blocks, S = nu * a.splits;
  SpanPlan p;
  p.n = lane < nu ? attn_unit_chunks(a, lane, rbr) : 0;
  p.start = __ockl_wfscan_add_i32(p.n, true) - p.n;
  p.total = __ockl_wfred_add_i32(p.n);
  const int C = max(p.total, 1);
  // slot holding chunk t: the largest x with floor(x C / S) <= t
  auto slot_of = [&](int t) { return (int)(((long)(t + 1) * S + C - 1) / C) - 1; };
  p.first = p.n > 0 ? slot_of(p.start) : 0;
  p.count = p.n > 0 ? slot_of(p.start + p.n - 1) - p.first + 1 : 0;
  p.seg_end = __ockl_wfscan_add_i32(p.count, true);
  p.ok = __ockl_wfred_max_i32(p.count) <= 64;
  return p;
}

// Scores are computed transposed, S^T = K Q^T: in the accumulator layout a lane holds
// keys 4*(lane/16)+i of one query (column lane%16), so the softmax is a per-lane
// reduction plus two cross-lane steps, and the probabilities feed O^T = V^T P^T as the
// B operand straight from registers (no LDS transpose).  In each 32-key MFMA step a
// lane supplies keys {4g..4g+3} and {16+4g..16+4g+3} of the step (g = lane/16); the
// V^T fragment from LDS uses the same key order.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_staged_kernel(AttnArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int KPAD = HD + 16 / EB;       // LDS row pitch (elements) for K
  constexpr int VPAD = kChunk + 16 / EB;   // LDS row pitch for V^T
  constexpr int NHT = HD / 16;             // output hd tiles
  constexpr int NKS = HD / 32;             // k-steps over hd for S
  constexpr int NSUB = kChunk / 16;        // 16-key score tiles per chunk
  constexpr int PAGES = kChunk / kPage;
  __shared__ __attribute__((aligned(16))) T sK[kChunk][KPAD];
  __shared__ __attribute__((aligned(16))) T sV[HD][VPAD];
  __shared__ int sPage[kMaxSplitPages];
  // bf16: probabilities enter P V as hi + lo bf16 parts (~16 significand bits)
  constexpr bool kSplitP = sizeof(T) == 2;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g4 = lane / 16, c16 = lane % 16;
  const int kvh = blockIdx.y;
  int unit, split, nsplit;
  if (!attn_slot_work(a, kAttnRows, unit, split, nsplit)) return;
  const int s = unit / a.row_blocks, rb = unit % a.row_blocks;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int P = a.pos0[s * a.seq_stride];
  const int nrows = nq * G;                      // valid (token, head) rows of this sequence
  const int row0 = rb * kAttnRows;               // first row of this workgroup
  if (row0 >= nrows) return;
  const int last_tok = min(nrows, row0 + kAttnRows) - 1;
  const int kv_end = a.causal ? P + last_tok / G + 1 : P + nq;   // keys [0, kv_end)
  const int nchunks = (kv_end + kChunk - 1) / kChunk;
  // chunks spread evenly over the splits (counts differ by at most one); the first splits
  // take the extra chunks, so the last one, which holds the newest keys (in rounds the
  // block's, whose K / V it may also write), is never the longest
  const int cq = nchunks / nsplit, cr = nchunks % nsplit;
  const int c_beg = split * cq + min(split, cr), c_end = c_beg + cq + (split < cr ? 1 : 0);
  // page ids of this split's keys (pages past kv_end are never dereferenced)
  const int pg_beg = c_beg * PAGES;
  const int npg = max(0, min((kv_end + kPage - 1) / kPage, c_end * PAGES) - pg_beg);
  for (int i = threadIdx.x; i < npg && i < kMaxSplitPages; i += 256)
    sPage[i] = a.page_table[(size_t)s * a.max_pages + pg_beg + i];

  // This lane's query: row = row0 + w*16 + lane%16 (all four lanes groups share it).
  const int qrow = row0 + w * 16 + c16;
  const bool qvalid = qrow < nrows;
  const int qpos = P + (qvalid ? qrow / G : 0);
  Frag<T> qf[NKS];
  {
    const int r = min(qrow, nrows - 1);
    const int tok = r / G, h = kvh * G + r % G;
    const T* qp = (const T*)a.q + (size_t)(s * a.rows_per_seq + tok) * a.n_q_heads * HD + (size_t)h * HD;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks].load(qp + ks * 32 + g4 * 8);
  }
  const float sl2 = a.scale * 1.4426950408889634f;
  float mrun = -INFINITY, lrun = 0.f;
  f32x4 o[NHT];                                   // O^T tiles: lane holds hd 16t+4g..+4 of its query
#pragma unroll
  for (int t = 0; t < NHT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();   // sPage ready

  const size_t head_page = (size_t)kPage * HD;   // elements of one (page, head) slice
  // Each thread stages NP 16-byte pieces of a chunk (K pieces first, then V^T pieces);
  // the next chunk's pieces are loaded into registers while the current one is used.
  constexpr int KV16 = kChunk * HD * EB / 16;     // 16-byte pieces of K per chunk (same for V)
  constexpr int NP = 2 * KV16 / 256;
  uint4 pf[NP];
  auto fetch = [&](int c) {
    const int key0 = c * kChunk;
    int pid[PAGES];
#pragma unroll
    for (int q = 0; q < PAGES; ++q)
      pid[q] = (c < c_end && key0 + q * kPage < kv_end) ? sPage[(c - c_beg) * PAGES + q] : -1;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int p = threadIdx.x + j * 256;
      const bool isv = p >= KV16;
      const int e0 = (isv ? p - KV16 : p) * (16 / EB);
      const int pg = e0 / (int)head_page, within = e0 % (int)head_page;
      int page = pid[0];
#pragma unroll
      for (int q = 1; q < PAGES; ++q) page = pg == q ? pid[q] : page;
      pf[j] = make_uint4(0, 0, 0, 0);
      if (page >= 0) {
        const T* src = (const T*)(isv ? a.vcache : a.kcache) + ((size_t)page * a.n_kv_heads + kvh) * head_page + within;
        pf[j] = *reinterpret_cast<const uint4*>(src);
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int p = threadIdx.x + j * 256;
      const bool isv = p >= KV16;
      const int e0 = (isv ? p - KV16 : p) * (16 / EB);
      const int pg = e0 / (int)head_page, within = e0 % (int)head_page;
      if (!isv) *reinterpret_cast<uint4*>(&sK[pg * kPage + within / HD][within % HD]) = pf[j];
      else *reinterpret_cast<uint4*>(&sV[within / kPage][pg * kPage + within % kPage]) = pf[j];
    }
  };
  if (c_beg < c_end) fetch(c_beg);
  for (int c = c_beg; c < c_end; ++c) {
    const int key0 = c * kChunk;
    __syncthreads();
    stage();
    __syncthreads();
    fetch(c + 1);
    // S^T = K Q^T, NSUB 16-key tiles
    f32x4 st[NSUB];
#pragma unroll
    for (int sub = 0; sub < NSUB; ++sub) {
      st[sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        Frag<T> kf;
        kf.load(&sK[sub * 16 + c16][ks * 32 + g4 * 8]);
        mma(st[sub], kf, qf[ks]);
      }
    }
    // scale, mask (only chunks that reach the causal edge or kv_end), online softmax
    float mx = -INFINITY;
    if (key0 + kChunk <= P && key0 + kChunk <= kv_end) {
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          st[sub][i] *= sl2;
          mx = fmaxf(mx, st[sub][i]);
        }
    } else {
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kp = key0 + sub * 16 + 4 * g4 + i;
          const bool vis = kp < kv_end && (!a.causal || kp <= qpos);
          st[sub][i] = vis ? st[sub][i] * sl2 : -INFINITY;
          mx = fmaxf(mx, st[sub][i]);
        }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(mrun, mx);
    float alpha = 1.f, rs = 0.f;
    if (mnew != -INFINITY) {
      alpha = __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          st[sub][i] = __builtin_amdgcn_exp2f(st[sub][i] - mnew);
          rs += st[sub][i];
        }
    } else {
#pragma unroll
      for (int sub = 0; sub < NSUB; ++sub)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[sub][i] = 0.f;
    }
    rs += __shfl_xor(rs, 16, 64);
    rs += __shfl_xor(rs, 32, 64);
    lrun = lrun * alpha + rs;
    mrun = mnew;
#pragma unroll
    for (int t = 0; t < NHT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[t][i] *= alpha;
    // O^T += V^T P^T, 32 keys per step: B (P^T) from registers, A (V^T) from LDS
#pragma unroll
    for (int kk = 0; kk < kChunk / 32; ++kk) {
      Frag<T> ph, pl;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x0 = st[2 * kk][i], x1 = st[2 * kk + 1][i];
        ph.set(i, x0);
        ph.set(4 + i, x1);
        if constexpr (kSplitP) {
          pl.set(i, x0 - ph.get(i));
          pl.set(4 + i, x1 - ph.get(4 + i));
        }
      }
#pragma unroll
      for (int t = 0; t < NHT; ++t) {
        Frag<T> vf;
        const T* vrow = &sV[t * 16 + c16][kk * 32];
        vf.load_halves(vrow + 4 * g4, vrow + 16 + 4 * g4);
        mma(o[t], vf, ph);
        if constexpr (kSplitP) mma(o[t], vf, pl);
      }
    }
  }

  // write result (single split) or partials; lane holds hd 16t+4g4+i of query qrow
  if (a.splits == 1) {
    if (qvalid) {
      const int tok = qrow / G, h = kvh * G + qrow % G;
      const float inv = lrun > 0.f ? 1.f / lrun : 0.f;
      T* op = (T*)a.out;
      const int orow = s * a.rows_per_seq + tok;
#pragma unroll
      for (int t = 0; t < NHT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          op[pa_index(orow, h * HD + t * 16 + 4 * g4 + i, a.ldo)] = Elem<T>::from_f32(o[t][i] * inv);
    }
  } else {
    const size_t blk = (size_t)kvh * attn_head_blocks(a) + blockIdx.z * a.splits + blockIdx.x;
    typename PartOf<T>::P* op = reinterpret_cast<typename PartOf<T>::P*>(a.opart) + blk * kAttnRows * HD;
    float* ml = a.mlpart + blk * kAttnRows * 2;
    const int rl = w * 16 + c16;
    const float inv = lrun > 0.f ? 1.f / lrun : 0.f;
#pragma unroll
    for (int t = 0; t < NHT; ++t)
      PartOf<T>::store4(op + (size_t)rl * HD + t * 16 + 4 * g4, o[t][0] * inv, o[t][1] * inv, o[t][2] * inv, o[t][3] * inv);
    if (g4 == 0) { ml[rl * 2] = mrun; ml[rl * 2 + 1] = lrun; }
  }
}

typedef __attribute__((address_space(4))) const int32_t const_i32_t;

__device__ __forceinline__ short bf16_bits(float x) { return __builtin_bit_cast(short, (__bf16)x); }
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// v[l] + v[l ^ 32] and v[l] + v[l ^ 16] in every lane l (both lanes of a pair add the
// same two values, so they agree bit for bit)
__device__ __forceinline__ float xor32_sum(float v) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float xor16_sum(float v) {
  auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// Wait until at most min(N, r) chunks of LPC copies each (this wave's) are in flight.
template <int N, int LPC>
__device__ __forceinline__ void wait_chunks(int r) {
  if constexpr (N <= 0) {
    wait_vm<0>();
  } else {
    if (r >= N) wait_vm<N * LPC>();
    else wait_chunks<N - 1, LPC>(r);
  }
}

// LDS accesses hidden from the compiler's wait insertion, which would otherwise wait
// for every direct-to-LDS copy in flight before them (the next chunk's copies
// included).  lds_wait() waits for them; a value read is used only after lds_wait() and
// lds_hold() on it, and a write is followed by lds_wait() before the barrier that
// publishes it.
__device__ __forceinline__ u32x4 lds_ld16(const void* p) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"((const lds_void_t*)p) : "memory");
  return v;
}
__device__ __forceinline__ void lds_st16(void* p, u32x4 v) {
  asm volatile("ds_write_b128 %0, %1" ::"v"((lds_void_t*)p), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_st2(void* p, uint32_t v) {
  asm volatile("ds_write_b16 %0, %1" ::"v"((lds_void_t*)p), "v"(v) : "memory");
}
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// A 16-byte direct-to-LDS copy per lane (lane l writes ldst + 16 l; ldst wave-uniform)
// the compiler does not see, so that it adds no waits for it (it waits for every such
// copy in flight before any LDS access it cannot tell apart from the copy).  M0 (the
// LDS address) is saved and restored around it; the caller waits with vmcnt.
__device__ __forceinline__ void lds_dma16(const void* gsrc, const void* ldst) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gsrc), "s"((uint32_t)(size_t)(const lds_void_t*)ldst)
      : "memory");
}
__device__ __forceinline__ void lds_hold(u32x4& v) { asm volatile("" : "+v"(v)); }

// Elements ks*32 + g4*8 + e (e = 0..7, ks < NKS) of an fp32 row: the lane's share of a
// 16-row tile in the MFMA fragment layout (g4 = lane / 16), as raw bits: x[ks][e / 4][e % 4].
template <int NKS>
__device__ __forceinline__ void load_frag_u(const float* row, int g4, u32x4 (&x)[NKS][2]) {
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) x[ks][hf] = *reinterpret_cast<const u32x4*>(row + ks * 32 + g4 * 8 + hf * 4);
}

// Per-head RMSNorm and rotate-half RoPE of a 16-row tile in the fragment layout (lane
// (g4, c16) holds elements ks*32 + g4*8 + e of row c16: x as raw fp32 bits, w the bf16
// norm weights of those elements, cs / sn the rotation factors of the pairs kp < NKS/2),
// rounded to bf16 fragments.  The row's sum of squares is added in the order of the
// q|k|v post-processing kernel: the pairs (l, l + hd/2), then over the bits of l from
// the highest down, which here are the pair index kp (bit 5 at hd 128), the lane bits 5
// and 4, and the element bits of e; so the results agree with that kernel bit for bit.
template <int NKS>
__device__ __forceinline__ void qk_tile(const u32x4 (&x)[NKS][2], const u32x4 (&w)[NKS], const u32x4 (&cs)[NKS / 2][2],
                                        const u32x4 (&sn)[NKS / 2][2], float eps, Frag<bf16_t> (&out)[NKS]) {
  constexpr int NKP = NKS / 2;
  auto X = [&](int ks, int e) { return __uint_as_float(x[ks][e >> 2][e & 3]); };
  auto W = [&](int ks, int e) { return __uint_as_float(((w[ks][e >> 1] >> (16 * (e & 1))) & 0xffffu) << 16); };
  float t[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    t[e] = qk_sq(X(0, e), X(NKP, e));
    if constexpr (NKP == 2) t[e] = t[e] + qk_sq(X(1, e), X(3, e));
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = xor32_sum(t[e]);
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = xor16_sum(t[e]);
#pragma unroll
  for (int e = 0; e < 4; ++e) t[e] = t[e] + t[e + 4];
#pragma unroll
  for (int e = 0; e < 2; ++e) t[e] = t[e] + t[e + 2];
  const float inv = qk_inv(t[0] + t[1], NKS * 32, eps);
#pragma unroll
  for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x0 = X(kp, e), x1 = X(kp + NKP, e);
      qk_norm_rope(x0, x1, inv, W(kp, e), W(kp + NKP, e), __uint_as_float(cs[kp][e >> 2][e & 3]),
                   __uint_as_float(sn[kp][e >> 2][e & 3]));
      out[kp].v[e] = bf16_bits(x0);
      out[kp + NKP].v[e] = bf16_bits(x1);
    }
}

// XOR swizzle of the 16-byte pieces of a K row in LDS (row r of chunk page pg), so that
// the 16 lanes reading one fragment column hit distinct banks.
template <int NPR>
__device__ __forceinline__ int kswz(int r, int pg) { return (r ^ ((pg & 1) << 2)) & (NPR - 1); }

// Work split of a workgroup of NW waves: wave w owns query rows rh*16*NRT .. +16*NRT-1
// of the row block (rh = w/2, NRT 16-row MFMA tiles) and keys kh*32..kh*32+31 of every
// 64-key chunk (kh = w%2, two pages); the two key halves of the same rows are merged
// through LDS at the end.  Every K / V byte staged in LDS is read by NW/2 waves.  The
// launches use one query tile per wave (8 or 12 waves): two or three waves per SIMD then
// interleave their dependent chains (LDS reads, score MFMAs, online softmax, PV MFMAs).
//
// Key order inside a wave's 32 keys: score tile tau (0, 1), A-operand row m holds key
// (m/4)*8 + 4*tau + m%4, so that the accumulator lane (g, q) ends up with the eight
// consecutive keys 8g..8g+7 (tau = 0: 8g..8g+3, tau = 1: 8g+4..8g+7).  Those eight
// probabilities are exactly the lane's B operand of O^T += V^T P^T, and its V^T operand
// is one contiguous 16-byte piece of a V page row.
template <int HD, int NSTAGE, int NRT, int NW, bool FUSED>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(AttnArgs a) {
  constexpr int ROWB = HD * 2;                 // bytes of one K row (one token)
  constexpr int NPR = ROWB / 16;               // 16-byte pieces per K row
  constexpr int PGB = kPage * ROWB;            // bytes of one (page, KV head) slice of K or V
  constexpr int NLD = PGB / 1024;              // wave-wide 16-byte-per-lane copies per slice
  constexpr int PAGES = kChunk / kPage;        // one page copied per wave
  constexpr int STG = 2 * PAGES * PGB;         // one stage: 4 K slices, then 4 V slices
  constexpr int NHT = HD / 16, NKS = HD / 32;
  constexpr int OPITCH = HD + 4;               // fp32 row pitch of the key-half merge buffer
  constexpr int RH = 16 * NRT;                 // rows per wave
  constexpr int RBR = NW / 2 * RH;             // rows per workgroup (row block)
  constexpr int MERGE = RBR * OPITCH * 4 + RBR * 2 * 4;
  // copies per chunk: with four waves each copies one K and one V page; with eight or
  // more, waves 0-3 copy the K pages and waves 4-7 the V pages (the rest copy nothing)
  constexpr bool SPREAD = NW >= 8;
  constexpr int LPC = SPREAD ? NLD : 2 * NLD;  // copies per chunk of a copying wave
  static_assert(NW % 2 == 0 && (NW == 4 || NW >= 8), "wave pairs; 4 or at least 8 waves");
  constexpr int SMEM = NSTAGE * STG > MERGE ? NSTAGE * STG : MERGE;
  // Fused q / k post-processing: an LDS area fsm behind the stages / merge buffer holds
  // the block's bf16 K and V rows [2][16][HD].  With eight waves (two stages) the fp32
  // inputs are staged there too by direct-to-LDS copies: the workgroup's 64 q rows, the
  // rotation factors of the 16 block positions, the two norm weights and the block's
  // fp32 k and v rows; so they take one L1 pass per workgroup and the waits for them are
  // explicit.  (One LDS array: with a second one the compiler tracks the chunk copies by
  // object and waits for the next chunk's copies before every read of the current one.)
  constexpr bool STAGED = FUSED && NSTAGE == 2 && NW == 8;
  constexpr int QST = 2 * 16 * ROWB;                // q rows [64][HD] fp32 (pieces swizzled)
  constexpr int RP = QST + 256 * HD;                // rotation factors [cos, sin][16][HD/2] fp32
  constexpr int NWT = RP + 64 * HD;                 // norm weights [q, k][HD] bf16
  constexpr int KVF = NWT + 4 * HD;                 // block rows [k, v][16][HD] fp32 (pieces swizzled)
  constexpr int QFX = KVF + 128 * HD;               // normalised q fragments of key half 0 [NW/2][64][HD/2 B]
  constexpr int FSM = STAGED ? QFX + NW / 2 * 32 * HD : 2 * 16 * ROWB;
  static_assert(!STAGED || NRT == 1, "one query tile per wave");
  static_assert(PAGES == 4, "four 16-token pages per 64-key chunk");
  static_assert(NW * 64 >= 32 * NPR, "one thread per 16-byte piece of the block's K and V rows");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM + (FUSED ? FSM : 0)];
  char* const fsm = smem + SMEM;

  const int lane = threadIdx.x & 63, g4 = lane >> 4, c16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rh = w >> 1, kh = w & 1;
  const int kvh = blockIdx.y;
  // This workgroup's segments: one (unit, chunk range, partial block) under the uniform
  // and balanced plans; under the spanning plan (batches without the fused q / k work)
  // one per unit its slot meets, run one after the other.
  int unit = 0, split = 0, nsplit = 1;
  bool span = false;
  SpanPlan sp{};
  unsigned long long seg_units = 0;   // spanning: units still to run
  const int slot = blockIdx.z * a.splits + blockIdx.x;
  if constexpr (!FUSED) {
    if (a.span && attn_balanced(a)) {
      // span when its slots are shorter than the balanced plan's longest split by more
      // than the pipeline fill of a second segment (about three chunks, measured)
      sp = attn_span_plan(a, RBR);
      const int S = a.n_seqs * a.row_blocks * a.splits;
      span = sp.ok && (a.span == 2 || (sp.total + S - 1) / S + 3 < attn_balanced_plan(a, RBR).q);
    }
  }
  if (span) {
    if (slot == 0 && blockIdx.y == 0 && threadIdx.x < 64) {   // hand the plan to the merge
      a.plan[threadIdx.x] = sp.seg_end - sp.count;
      a.plan[64 + threadIdx.x] = sp.count;
    }
    seg_units = __ballot(sp.count > 0 && slot >= sp.first && slot < sp.first + sp.count);
    if (seg_units == 0) return;
  } else if (!attn_slot_work(a, RBR, unit, split, nsplit)) {
    return;
  }
  for (;;) {
  int seg_c0 = 0, seg_c1 = 0;
  size_t part_blk = (size_t)kvh * attn_head_blocks(a) + slot;
  if (span) {
    unit = __builtin_ctzll(seg_units);
    seg_units &= seg_units - 1;
    const int S = a.n_seqs * a.row_blocks * a.splits;
    const long b0 = (long)slot * sp.total / S, b1 = (long)(slot + 1) * sp.total / S;
    const int ustart = __builtin_amdgcn_readlane(sp.start, unit), un = __builtin_amdgcn_readlane(sp.n, unit);
    const int ufirst = __builtin_amdgcn_readlane(sp.first, unit);
    seg_c0 = (int)max(b0, (long)ustart) - ustart;
    seg_c1 = (int)min(b1, (long)(ustart + un)) - ustart;
    split = slot - ufirst;
    nsplit = __builtin_amdgcn_readlane(sp.count, unit);
    part_blk = (size_t)kvh * attn_head_blocks(a) + (__builtin_amdgcn_readlane(sp.seg_end, unit) - nsplit) + split;
  }
  {
  const int s = unit / a.row_blocks, rb = unit % a.row_blocks;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int P = a.pos0[s * a.seq_stride];
  const int nrows = nq * G;
  const int row0 = rb * RBR;
  if (row0 >= nrows) goto seg_done;
  {
  const int last_tok = min(nrows, row0 + RBR) - 1;
  const int kv_end = a.causal ? P + last_tok / G + 1 : P + nq;   // keys [0, kv_end), kv_end >= 1
  const int nchunks = (kv_end + kChunk - 1) / kChunk;
  // chunks spread evenly over the splits (counts differ by at most one); the first splits
  // take the extra chunks, so the last one, which holds the newest keys (in rounds the
  // block's, whose K / V it may also write), is never the longest
  const int cq = nchunks / nsplit, cr = nchunks % nsplit;
  const int c_beg = span ? seg_c0 : split * cq + min(split, cr);
  const int c_end = span ? seg_c1 : c_beg + cq + (split < cr ? 1 : 0);
  const int last_page = (kv_end - 1) / kPage;
  const_i32_t* pt = (const_i32_t*)(a.page_table + (size_t)s * a.max_pages);
  // page w of chunk c (pages past kv_end are replaced by the last valid one, so every
  // wave issues the same number of copies per chunk; their keys are masked)
  const int cw = w & (PAGES - 1);               // page of the chunk this wave copies
  const bool copies_k = SPREAD ? w < PAGES : true, copies_v = SPREAD ? (w >= PAGES && w < 2 * PAGES) : true;
  auto page_of = [&](int c) { return pt[min(c * PAGES + cw, last_page)]; };

  // per-lane source offsets of the copies (LDS slot j*64+lane of this wave's slice)
  int koff[NLD], voff[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) {
    const int sl = j * 64 + lane;
    const int r = sl / NPR, p = sl % NPR;
    koff[j] = r * ROWB + (p ^ kswz<NPR>(r, cw)) * 16;
    const int h = sl >> 1, vp = sl & 1;
    voff[j] = h * 32 + (vp ^ ((h >> 3) & 1)) * 16;
  }
  // with one row block per sequence every K / V chunk is read by one workgroup:
  // non-temporal copies (several row blocks, as in prefill, share the chunks through cache)
  const bool stream_kv = a.row_blocks == 1;
  // With SPREAD a copying wave copies one page of K or one of V: its cache, per-lane
  // offsets and LDS slice are chosen once here, so that a chunk's copies cost one branch
  // and one page address.  stg_off: the byte offset of the stage.
  const char* const kvsrc = copies_k ? (const char*)a.kcache : (const char*)a.vcache;
  int coff[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) coff[j] = copies_k ? koff[j] : voff[j];
  const int lslice = (copies_k ? 0 : PAGES * PGB) + cw * PGB;
  auto issue = [&](int pg, int stg_off) {
    if constexpr (SPREAD) {
      if (!copies_k && !copies_v) return;
      const char* b = kvsrc + ((size_t)pg * a.n_kv_heads + kvh) * PGB;
      char* l = smem + stg_off + lslice;
      if (stream_kv) {
#pragma unroll
        for (int j = 0; j < NLD; ++j)
          __builtin_amdgcn_global_load_lds((const void*)(b + coff[j]), (lds_void_t*)(l + j * 1024), 16, 0, RT_NT_AUX);
      } else {
#pragma unroll
        for (int j = 0; j < NLD; ++j)
          __builtin_amdgcn_global_load_lds((const void*)(b + coff[j]), (lds_void_t*)(l + j * 1024), 16, 0, 0);
      }
    } else {
      const char* kb = (const char*)a.kcache + ((size_t)pg * a.n_kv_heads + kvh) * PGB;
      const char* vb = (const char*)a.vcache + ((size_t)pg * a.n_kv_heads + kvh) * PGB;
      char* lk = smem + stg_off + cw * PGB;
      char* lv = smem + stg_off + PAGES * PGB + cw * PGB;
#pragma unroll
      for (int j = 0; j < NLD; ++j)
        if (stream_kv) __builtin_amdgcn_global_load_lds((const void*)(kb + koff[j]), (lds_void_t*)(lk + j * 1024), 16, 0, RT_NT_AUX);
        else __builtin_amdgcn_global_load_lds((const void*)(kb + koff[j]), (lds_void_t*)(lk + j * 1024), 16, 0, 0);
#pragma unroll
      for (int j = 0; j < NLD; ++j)
        if (stream_kv) __builtin_amdgcn_global_load_lds((const void*)(vb + voff[j]), (lds_void_t*)(lv + j * 1024), 16, 0, RT_NT_AUX);
        else __builtin_amdgcn_global_load_lds((const void*)(vb + voff[j]), (lds_void_t*)(lv + j * 1024), 16, 0, 0);
    }
  };

  // this wave's queries: tile t2 (0..NRT-1) column c16 is row row0 + rh*RH + t2*16 + c16
  const int nrt = min(NRT, max(0, (nrows - row0 - rh * RH + 15) / 16));   // tiles with valid rows
  Frag<bf16_t> qf[NRT][NKS];
  int qpos[NRT];
  // Fused q / k post-processing (a.qkv set): every wave takes its q rows from the fp32
  // projection (with the norm weights and rotation factors) and normalises them once the
  // first chunk's copies are issued.  The workgroups whose chunks hold block positions
  // [kb_lo, kb_hi) also take the block's k (wave 0) and v (wave 1) rows, as a 16-row
  // tile (row c16 = block row c16); their bf16 values go to the LDS area fsm, into the
  // stage of the chunk that holds them once its copies have landed, and to the caches at
  // the end.  Eight waves stage these inputs in LDS (below); twelve load them directly.
  constexpr bool fused = FUSED;   // a.qkv set (the launch selects this instance)
  constexpr int NKP = NKS / 2;
  u32x4 qx[NRT][NKS][2], qcs[NRT][NKP][2], qsn[NRT][NKP][2], qw[NKS];   // raw fp32 / bf16 bits
#pragma unroll
  for (int t2 = 0; t2 < NRT; ++t2) {
    const int qrow = row0 + rh * RH + t2 * 16 + c16;
    const int r = min(qrow, nrows - 1);
    qpos[t2] = P + r / G;
    const int tok = r / G, h = kvh * G + r % G;
    if constexpr (STAGED) {
    } else if constexpr (fused) {
      load_frag_u<NKS>(a.qkv + (size_t)(s * a.rows_per_seq + tok) * a.ldqkv + (size_t)h * HD, g4, qx[t2]);
      const float* cs = a.rope + (size_t)qpos[t2] * (HD / 2);
      load_frag_u<NKP>(cs, g4, qcs[t2]);
      load_frag_u<NKP>(cs + (size_t)a.rope_max_pos * (HD / 2), g4, qsn[t2]);
    } else {
      const bf16_t* qp = (const bf16_t*)a.q + (size_t)(s * a.rows_per_seq + tok) * a.n_q_heads * HD + (size_t)h * HD;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) qf[t2][ks].load(qp + ks * 32 + g4 * 8);
    }
  }
  const int kb_lo = max(P, c_beg * kChunk), kb_hi = fused ? min(P + a.rows_per_seq, c_end * kChunk) : kb_lo;
  // the waves that take the block's k and v rows: staged, the key-half-1 waves 1 and 3
  // (key half 0 of their row pair normalises the pair's q); else waves 0 and 1
  constexpr int KW = STAGED ? 1 : 0, VW = STAGED ? 3 : 1;
  const bool kv_wave = kb_lo < kb_hi && (w == KW || w == VW);
  const bool q_wave = !STAGED || kh == 0;        // normalises q (staged: shares it through LDS)
  u32x4 kx[NKS][2], kcs[NKP][2], ksn[NKP][2], kw[NKS];
  auto load_kv = [&]() {
    const int i = min(c16, a.rows_per_seq - 1);
    load_frag_u<NKS>(a.qkv + (size_t)(s * a.rows_per_seq + i) * a.ldqkv + a.q_cols + (w == VW ? a.kv_cols : 0) +
                         (size_t)kvh * HD, g4, kx);
    if (w == KW) {
      const float* cs = a.rope + (size_t)(P + i) * (HD / 2);
      load_frag_u<NKP>(cs, g4, kcs);
      load_frag_u<NKP>(cs + (size_t)a.rope_max_pos * (HD / 2), g4, ksn);
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) kw[ks] = *reinterpret_cast<const u32x4*>((const bf16_t*)a.k_norm + ks * 32 + g4 * 8);
    }
  };
  if constexpr (STAGED) {
    // q rows: piece slot ps of row rr holds the row's 16-byte piece ps ^ (rr % 16)
    constexpr int PR = HD / 4;                      // 16-byte pieces of an fp32 row
    constexpr int QI = 64 * PR / 64 / NW;           // copies per wave
#pragma unroll
    for (int j = 0; j < QI; ++j) {
      const int slot = (w * QI + j) * 64 + lane, rr = slot / PR, ps = slot % PR;
      const int r = min(row0 + rr, nrows - 1), tok = r / G, h = kvh * G + r % G;
      const float* src = a.qkv + (size_t)(s * a.rows_per_seq + tok) * a.ldqkv + (size_t)h * HD + (ps ^ (rr & 15)) * 4;
      lds_dma16(src, fsm + QST + (w * QI + j) * 1024);
    }
    if (w == 0 && lane < HD / 4) {                  // q-norm then k-norm weights
      const bf16_t* src = lane < HD / 8 ? (const bf16_t*)a.q_norm + lane * 8 : (const bf16_t*)a.k_norm + (lane - HD / 8) * 8;
      lds_dma16(src, fsm + NWT);
    }
    if (kb_lo < kb_hi) {                            // the block's k and v rows, same piece swizzle
      constexpr int KI = 2 * 16 * PR / 64 / NW;
#pragma unroll
      for (int j = 0; j < KI; ++j) {
        const int slot = (w * KI + j) * 64 + lane, kv = slot / (16 * PR), rr = slot / PR % 16, ps = slot % PR;
        const float* src = a.qkv + (size_t)(s * a.rows_per_seq + min(rr, a.rows_per_seq - 1)) * a.ldqkv + a.q_cols +
                           (kv ? a.kv_cols : 0) + (size_t)kvh * HD + (ps ^ (rr & 15)) * 4;
        lds_dma16(src, fsm + KVF + (w * KI + j) * 1024);
      }
    }
    // rotation factors of positions P .. P+15 (clamped to the table), cos rows then sin rows
    constexpr int RI = 2 * 16 * (HD / 2) * 4 / 1024;   // copies (one per wave)
    if (w < RI) {
      const int slot = w * 64 + lane, tbl = slot / (16 * HD / 8), t = slot / (HD / 8) % 16, ps = slot % (HD / 8);
      const int pos = min(P + t, a.rope_max_pos - 1);
      const float* src = a.rope + (size_t)tbl * a.rope_max_pos * (HD / 2) + (size_t)pos * (HD / 2) + ps * 4;
      lds_dma16(src, fsm + RP + w * 1024);
    }
  } else if constexpr (fused) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qw[ks] = *reinterpret_cast<const u32x4*>((const bf16_t*)a.q_norm + ks * 32 + g4 * 8);
  }
  const float sl2 = a.scale * 1.4426950408889634f;
  // reference max (log2 units), raised lazily.  It starts at a finite sentinel: a masked
  // score (-inf) then still gives exp2(-inf) = 0, and the first visible score of a row
  // raises the reference before any exponential of it is taken.
  constexpr float kMrefInit = -1.0e30f;
  float mref[NRT], lsum[NRT];   // lsum: this lane's share of the row sum
  f32x4 o[NRT][NHT];
#pragma unroll
  for (int t2 = 0; t2 < NRT; ++t2) {
    mref[t2] = kMrefInit;
    lsum[t2] = 0.f;
  }
#pragma unroll
  for (int t2 = 0; t2 < NRT; ++t2)
#pragma unroll
    for (int t = 0; t < NHT; ++t) o[t2][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // prologue: chunks c_beg .. c_beg+NSTAGE-2 in flight
#pragma unroll
  for (int i = 0; i < NSTAGE - 1; ++i)
    if (c_beg + i < c_end) issue(page_of(c_beg + i), i * STG);
  int pg_next = page_of(c_beg + NSTAGE - 1);

  if constexpr (STAGED) {
    // the staged rows have landed once at most this wave's chunk copies remain; the
    // barrier makes every wave's copies visible
    if (c_beg < c_end) wait_vm<LPC>(); else wait_vm<0>();
    lds_barrier();
    auto read_rows = [&](const char* base, int rr, u32x4 (&x)[NKS][2]) {
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) x[ks][hf] = lds_ld16(base + rr * HD * 4 + (((ks * 8 + g4 * 2 + hf) ^ (rr & 15)) * 16));
    };
    auto read_rot = [&](int t, u32x4 (&cs)[NKP][2], u32x4 (&sn)[NKP][2]) {
      const char* rc = fsm + RP + (t * (HD / 2) + g4 * 8) * 4;
#pragma unroll
      for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          cs[kp][hf] = lds_ld16(rc + (kp * 32 + hf * 4) * 4);
          sn[kp][hf] = lds_ld16(rc + (16 * (HD / 2) + kp * 32 + hf * 4) * 4);
        }
    };
    auto hold = [&](auto& arr) {
      for (auto& v : arr) lds_hold(v);
    };
    if (q_wave) {
      const char* wts = fsm + NWT;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) qw[ks] = lds_ld16(wts + (ks * 32 + g4 * 8) * 2);
      const int rr = rh * RH + c16;
      read_rows(fsm + QST, rr, qx[0]);
      read_rot(min(row0 + rr, nrows - 1) / G, qcs[0], qsn[0]);
      lds_wait();
      hold(qw);
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) hold(qx[0][ks]);
#pragma unroll
      for (int kp = 0; kp < NKP; ++kp) {
        hold(qcs[0][kp]);
        hold(qsn[0][kp]);
      }
    }
  }
  if constexpr (fused) {
    // (unstaged: the compiler waits here for every outstanding load, the copies just
    // issued included: it does not order direct-to-LDS copies with other loads)
#pragma unroll
    for (int t2 = 0; t2 < NRT; ++t2) {
      if (!q_wave) break;
      qk_tile<NKS>(qx[t2], qw, qcs[t2], qsn[t2], a.eps, qf[t2]);
      if constexpr (STAGED) {   // for the key-half-1 wave of the pair (read in the first chunk step)
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) lds_st16(fsm + QFX + (rh * 64 + lane) * (HD / 2) + ks * 16, __builtin_bit_cast(u32x4, qf[t2][ks].v));
        lds_wait();
      }
      // key split 0 of the unit keeps the normalised q (one copy per row: key half 0)
      const int qrow = row0 + rh * RH + t2 * 16 + c16;
      if (a.q_out && split == 0 && kh == 0 && qrow < nrows) {
        const int tok = qrow / G, h = kvh * G + qrow % G;
        bf16_t* qo = (bf16_t*)a.q_out + (size_t)(s * a.rows_per_seq + tok) * a.ldq + (size_t)h * HD + g4 * 8;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) qf[t2][ks].store(qo + ks * 32);
      }
    }
    if (kv_wave) {
      if constexpr (STAGED) {
        const char* wts = fsm + NWT;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            kx[ks][hf] = lds_ld16(fsm + KVF + (w == VW ? 16 * HD * 4 : 0) + c16 * HD * 4 + (((ks * 8 + g4 * 2 + hf) ^ c16) * 16));
          }
        if (w == KW) {
          const char* rc = fsm + RP + (c16 * (HD / 2) + g4 * 8) * 4;
#pragma unroll
          for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
              kcs[kp][hf] = lds_ld16(rc + (kp * 32 + hf * 4) * 4);
              ksn[kp][hf] = lds_ld16(rc + (16 * (HD / 2) + kp * 32 + hf * 4) * 4);
            }
#pragma unroll
          for (int ks = 0; ks < NKS; ++ks) kw[ks] = lds_ld16(wts + (HD + ks * 32 + g4 * 8) * 2);
        }
        lds_wait();
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          lds_hold(kx[ks][0]);
          lds_hold(kx[ks][1]);
          lds_hold(kw[ks]);
        }
#pragma unroll
        for (int kp = 0; kp < NKP; ++kp)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            lds_hold(kcs[kp][hf]);
            lds_hold(ksn[kp][hf]);
          }
      } else {   // unstaged (twelve waves, 168 registers per lane): loaded once q is done
        load_kv();
      }
      Frag<bf16_t> kv[NKS];
      if (w == KW) {
        qk_tile<NKS>(kx, kw, kcs, ksn, a.eps, kv);
      } else {
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) kv[ks].v[e] = bf16_bits(__uint_as_float(kx[ks][e >> 2][e & 3]));
      }
      char* side = fsm + (w == VW ? 16 * ROWB : 0) + c16 * ROWB + g4 * 16;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) lds_st16(side + ks * 64, __builtin_bit_cast(u32x4, kv[ks].v));
      lds_wait();   // published by the first chunk step's barrier
    }
  }
  // the block's rows in the side area: thread piece (row i, 16-byte piece p) of K (first
  // 16 * NPR threads) or V (next 16 * NPR threads)
  const int bt = threadIdx.x % (16 * NPR), bi = bt / NPR, bp = bt % NPR;
  const bool b_v = threadIdx.x >= 16 * NPR, b_any = threadIdx.x < 32 * NPR;
  const char* bside = fsm + (b_v ? 16 * ROWB : 0) + bi * ROWB + bp * 16;
  const bool b_mine = fused && b_any && P + bi >= kb_lo && P + bi < kb_hi;   // a row this workgroup caches
  const int b_page = b_mine ? pt[(P + bi) / kPage] : 0;

  // byte offsets of chunk c's stage and of the stage its step fills (chunk c+NSTAGE-1),
  // advanced by one stage per chunk with a wrap
  int off_c = 0, off_n = (NSTAGE - 1) * STG;
  for (int c = c_beg; c < c_end; ++c) {
    const int cur = off_c, nxt = off_n;
    off_c = off_c + STG == NSTAGE * STG ? 0 : off_c + STG;
    off_n = off_n + STG == NSTAGE * STG ? 0 : off_n + STG;
    // this wave's copies of chunk c have landed once at most the later chunks' remain
    wait_chunks<NSTAGE - 2, LPC>(c_end - 1 - c);
    lds_barrier();   // every wave's copies of chunk c are visible; chunk c-1's stage is free
    if (STAGED && !q_wave && c == c_beg) {   // the pair's normalised q from key half 0
      u32x4 qr[NKS];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) qr[ks] = lds_ld16(fsm + QFX + (rh * 64 + lane) * (HD / 2) + ks * 16);
      lds_wait();
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        lds_hold(qr[ks]);
        qf[0][ks].v = __builtin_bit_cast(bf16x8, qr[ks]);
      }
    }
    if (fused && kb_lo < kb_hi && c * kChunk < kb_hi && (c + 1) * kChunk > kb_lo) {
      // the block's rows in this chunk replace what the copies brought from the caches
      // (before the next chunk's copies are issued: the wait for these LDS accesses also
      // waits for the scalar page lookup issued with them)
      const int pos = P + bi;
      if (b_any && pos >= max(kb_lo, c * kChunk) && pos < min(kb_hi, (c + 1) * kChunk)) {
        const int pg = pos / kPage - c * PAGES, r = pos % kPage;
        char* st = smem + cur + (b_v ? PAGES * PGB : 0) + pg * PGB;
        u32x4 v = lds_ld16(bside);
        lds_wait();
        lds_hold(v);
        if (!b_v) {
          lds_st16(st + r * ROWB + (bp ^ kswz<NPR>(r, pg)) * 16, v);
        } else {   // V^T: hd row h = bp*8 + e, token r at piece (r / 8) ^ ((h / 8) & 1)
          char* vt = st + ((r >> 3) ^ (bp & 1)) * 16 + (r & 7) * 2;
#pragma unroll
          for (int e = 0; e < 8; ++e) lds_st2(vt + (bp * 8 + e) * 32, (v[e / 2] >> (16 * (e & 1))) & 0xffff);
        }
        lds_wait();
      }
      lds_barrier();
    }
    if (c + NSTAGE - 1 < c_end) {
      issue(pg_next, nxt);
      pg_next = page_of(c + NSTAGE);
    }
    if (nrt == 0) continue;
    const char* sk = smem + cur;
    const char* sv = sk + PAGES * PGB;
    const int kbase = c * kChunk + kh * 32;
    // fragments of this wave's 32 keys: K (2 score tiles x NKS), V^T (NHT)
    Frag<bf16_t> kf[2][NKS], vf[NHT];
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      const int kis = (c16 >> 2) * 8 + tau * 4 + (c16 & 3);
      const int pg = kh * 2 + (kis >> 4), r = kis & 15;
      const char* rowp = sk + pg * PGB + r * ROWB;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        kf[tau][ks].v = *reinterpret_cast<const bf16x8*>(rowp + ((ks * 4 + g4) ^ kswz<NPR>(r, pg)) * 16);
    }
#pragma unroll
    for (int t = 0; t < NHT; ++t) {
      const int pg = kh * 2 + (g4 >> 1), h = t * 16 + c16;
      vf[t].v = *reinterpret_cast<const bf16x8*>(sv + pg * PGB + h * 32 + ((g4 & 1) ^ ((h >> 3) & 1)) * 16);
    }
#pragma unroll
    for (int t2 = 0; t2 < NRT; ++t2) {
      if (t2 >= nrt) break;
      // S^T = K Q^T: two 16-key tiles of this query tile
      f32x4 st[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
        for (int tau = 0; tau < 2; ++tau) mma(st[tau], kf[tau][ks], qf[t2][ks]);
      if (kbase + 32 > P) {   // keys that reach the block: causal / end mask
#pragma unroll
        for (int tau = 0; tau < 2; ++tau)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int kp = kbase + g4 * 8 + tau * 4 + e;
            const bool vis = kp < kv_end && (!a.causal || kp <= qpos[t2]);
            st[tau][e] = vis ? st[tau][e] : -INFINITY;
          }
      }
      float mx = fmaxf(fmaxf(fmaxf(st[0][0], st[0][1]), fmaxf(st[0][2], st[0][3])),
                       fmaxf(fmaxf(st[1][0], st[1][1]), fmaxf(st[1][2], st[1][3])));
      mx = group4_max(mx);
      const float mxs = mx * sl2;
      // raise the reference only when a score exceeds it by more than 2^8 (exponentials
      // stay below 256; the final ratio is unchanged); rescale O and the sum then
      if (__builtin_amdgcn_ballot_w64(mxs > mref[t2] + 8.f)) {
        const float mnew = fmaxf(mref[t2], mxs);
        const float alpha = __builtin_amdgcn_exp2f(mref[t2] - mnew);   // 0 when leaving the sentinel
#pragma unroll
        for (int t = 0; t < NHT; ++t)
#pragma unroll
          for (int e = 0; e < 4; ++e) o[t2][t][e] *= alpha;
        lsum[t2] *= alpha;
        mref[t2] = mnew;
      }
      const float mr = mref[t2];
      // P as a bf16 high part plus the bf16 rounding of its remainder (about 16
      // significand bits), two MFMAs per tile: the weights entering O are the fp32
      // exponentials to within 2^-16 relative, and the row sum adds the fp32 values
      Frag<bf16_t> ph, pl;
#pragma unroll
      for (int tau = 0; tau < 2; ++tau)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = __builtin_amdgcn_exp2f(fmaf(st[tau][e], sl2, -mr));
          lsum[t2] += x;
          const short hb = bf16_bits(x);
          ph.v[tau * 4 + e] = hb;
          pl.v[tau * 4 + e] = bf16_bits(x - __uint_as_float((uint32_t)(uint16_t)hb << 16));
        }
      // O^T += V^T P^T
#pragma unroll
      for (int t = 0; t < NHT; ++t) mma(o[t2][t], vf[t], ph);
#pragma unroll
      for (int t = 0; t < NHT; ++t) mma(o[t2][t], vf[t], pl);
    }
  }
#pragma unroll
  for (int t2 = 0; t2 < NRT; ++t2) lsum[t2] = group4_sum(lsum[t2]);
  // fused: the block's K / V rows into the caches (last, so that no wait for a chunk's
  // copies also waits for these stores; the loop's barriers made the side area visible)
  if (b_mine) {
    const int tok = (P + bi) % kPage;
    const size_t pb = ((size_t)b_page * a.n_kv_heads + kvh) * (size_t)(kPage * HD);
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(bside);
    if (!b_v) {
      *reinterpret_cast<bf16x8*>((bf16_t*)a.kcache + pb + (size_t)tok * HD + bp * 8) = v;
    } else {
      short* vc = (short*)a.vcache + pb + tok;
#pragma unroll
      for (int e = 0; e < 8; ++e) vc[(size_t)(bp * 8 + e) * kPage] = v[e];
    }
  }

  // merge the two key halves of each row pair of waves through LDS (stages are free
  // once every wave has passed this barrier)
  lds_barrier();
  float* mo = reinterpret_cast<float*>(smem) + rh * RH * OPITCH;             // [RH][OPITCH] O^T rows
  float* mml = reinterpret_cast<float*>(smem) + RBR * OPITCH + rh * RH * 2;    // [RH][2] (m, l)
  if (kh == 1) {
#pragma unroll
    for (int t2 = 0; t2 < NRT; ++t2) {
      const int rl = t2 * 16 + c16;
#pragma unroll
      for (int t = 0; t < NHT; ++t)
        *reinterpret_cast<float4*>(mo + rl * OPITCH + t * 16 + 4 * g4) =
            make_float4(o[t2][t][0], o[t2][t][1], o[t2][t][2], o[t2][t][3]);
      if (g4 == 0) { mml[rl * 2] = mref[t2]; mml[rl * 2 + 1] = lsum[t2]; }
    }
  }
  lds_barrier();
  if (kh == 1) goto seg_done;
#pragma unroll
  for (int t2 = 0; t2 < NRT; ++t2) {
    const int rl = t2 * 16 + c16;
    const float m1 = mml[rl * 2], l1 = mml[rl * 2 + 1];
    const float m0 = mref[t2];
    const float M = fmaxf(m0, m1);
    const float f0 = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m0 - M);
    const float f1 = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
    // explicit fused forms: every wave layout rounds the merge identically
    const float L = fmaf(f0, lsum[t2], f1 * l1);
#pragma unroll
    for (int t = 0; t < NHT; ++t) {
      const float4 v1 = *reinterpret_cast<const float4*>(mo + rl * OPITCH + t * 16 + 4 * g4);
      o[t2][t][0] = fmaf(f1, v1.x, f0 * o[t2][t][0]);
      o[t2][t][1] = fmaf(f1, v1.y, f0 * o[t2][t][1]);
      o[t2][t][2] = fmaf(f1, v1.z, f0 * o[t2][t][2]);
      o[t2][t][3] = fmaf(f1, v1.w, f0 * o[t2][t][3]);
    }
    const int qrow = row0 + rh * RH + rl;
    if (a.splits == 1) {
      if (qrow < nrows) {
        const int tok = qrow / G, h = kvh * G + qrow % G;
        const float inv = L > 0.f ? 1.f / L : 0.f;
        bf16_t* op = (bf16_t*)a.out;
        const int orow = s * a.rows_per_seq + tok;
#pragma unroll
        for (int t = 0; t < NHT; ++t)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            op[pa_index(orow, h * HD + t * 16 + 4 * g4 + e, a.ldo)] = f32_to_bf16(o[t2][t][e] * inv);
      }
    } else {
      const size_t blk = part_blk;
      _Float16* op = reinterpret_cast<_Float16*>(a.opart) + blk * RBR * HD;
      float* ml = a.mlpart + blk * RBR * 2;
      const int rw = rh * RH + rl;
      const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
      for (int t = 0; t < NHT; ++t)
        PartOf<bf16_t>::store4(op + (size_t)rw * HD + t * 16 + 4 * g4, o[t2][t][0] * inv, o[t2][t][1] * inv,
                               o[t2][t][2] * inv, o[t2][t][3] * inv);
      if (g4 == 0) { ml[rw * 2] = M; ml[rw * 2 + 1] = L; }
    }
  }
  }
  }
seg_done:
  if (!span || seg_units == 0) break;
  lds_barrier();   // the key-half merge buffer is read before the next segment's copies land
  }
}

// One wave per (sequence, kv head, row).  Lane j holds split j's running max and sum;
// lane l keeps hd elements l*PL .. l*PL+PL-1 of every split's normalised partial row,
// loaded in batches of 32 splits before the split weights are known, then summed with
// the weights exp2(m_j - M) * sum_j read from lane j.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  using P = typename PartOf<T>::P;
  constexpr int PL = HD / 64;                 // hd elements per lane (1 or 2)
  constexpr int NB = 32;                      // splits per batch of loads
  const int lane = threadIdx.x & 63;
  const int rl = blockIdx.x * 4 + (threadIdx.x >> 6);        // row within the row block
  const int s = blockIdx.z / a.row_blocks, rb = blockIdx.z % a.row_blocks, kvh = blockIdx.y;
  const int RBR = a.rb_rows;
  if (rl >= RBR) return;
  const int2 us = attn_unit_slots(a, blockIdx.z);
  const int S = us.y;                         // <= 64
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int r = rb * RBR + rl;
  if (r >= nq * G) return;
  const int tok = r / G, h = kvh * G + r % G;
  T* out = (T*)a.out;
  const int orow = s * a.rows_per_seq + tok;
  if (S <= 0) {   // no split holds keys of this unit (not produced by the plans)
#pragma unroll
    for (int e = 0; e < PL; ++e) out[pa_index(orow, h * HD + lane * PL + e, a.ldo)] = Elem<T>::from_f32(0.f);
    return;
  }
  const size_t blk0 = (size_t)kvh * attn_head_blocks(a) + us.x;
  const P* opp = reinterpret_cast<const P*>(a.opart) + (blk0 * RBR + rl) * HD + lane * PL;   // split j: + j * RBR * HD
  const float* mlp = a.mlpart + (blk0 * RBR + rl) * 2;          // split j: + j * RBR * 2
  // loads past the last split read split S-1 again (no branch, so all stay in flight);
  // their weights are zero
  float ob[NB][PL];
#pragma unroll
  for (int j = 0; j < NB; ++j) PartOf<T>::template load<PL>(opp + (size_t)(j < S ? j : S - 1) * RBR * HD, ob[j]);
  float mj = -INFINITY, lj = 0.f;
  if (lane < S) {
    const float2 v = *reinterpret_cast<const float2*>(mlp + (size_t)lane * RBR * 2);
    mj = v.x;
    lj = v.y;
  }
  const float M = warp_max(mj);
  const float f = (M == -INFINITY || mj == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mj - M) * lj;
  const float den = warp_sum(f);
  float num[PL];
#pragma unroll
  for (int e = 0; e < PL; ++e) num[e] = 0.f;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const float fj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), j));
#pragma unroll
    for (int e = 0; e < PL; ++e) num[e] += fj * ob[j][e];
  }
  for (int j0 = NB; j0 < S; j0 += NB) {
#pragma unroll
    for (int j = 0; j < NB; ++j)
      PartOf<T>::template load<PL>(opp + (size_t)(j0 + j < S ? j0 + j : S - 1) * RBR * HD, ob[j]);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const float fj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), j0 + j));
#pragma unroll
      for (int e = 0; e < PL; ++e) num[e] += (j0 + j < S ? fj : 0.f) * ob[j][e];
    }
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
  for (int e = 0; e < PL; ++e) out[pa_index(orow, h * HD + lane * PL + e, a.ldo)] = Elem<T>::from_f32(num[e] * inv);
}

// One query tile per wave: 64-row blocks 8 waves with two LDS stages (64 KB at hd 128,
// two workgroups per compute unit), or three (96 KB) where every split holds long key
// ranges: 8B batch-8 rounds 34.2 -> 32.6 us per layer (four stages 33.3), while the
// short contexts of a 16-sequence serving batch ran 0.6 us slower with three; the kernel
// that stages the q / k work's inputs keeps two (they take the third stage's room); 96-row
// blocks 12 waves, three stages (96 KB; 15% faster than 4 waves of three tiles at the 14B
// verify shape, where four stages measured no faster).  Results do not depend on the wave layout (the key-half
// merge is written in explicit fused form).
template <typename T>
hipError_t attention_partials(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.splits, a.n_kv_heads, a.n_seqs * a.row_blocks);
  // the fused q / k post-processing: bf16 kernels, blocks of at most 16 rows per sequence
  if (a.qkv && (sizeof(T) != 2 || a.rows_per_seq > 16 || a.nq)) return hipErrorInvalidValue;
  if constexpr (sizeof(T) == 2) {
    const bool f = a.qkv != nullptr;
    if (a.rb_rows == 96) {
      if (a.head_dim == 128 && f) RT_LAUNCH((attn_bf16_kernel<128, 3, 1, 12, true>), grid, dim3(768), 0, s, a);
      else if (a.head_dim == 128) RT_LAUNCH((attn_bf16_kernel<128, 3, 1, 12, false>), grid, dim3(768), 0, s, a);
      else if (a.head_dim == 64 && f) RT_LAUNCH((attn_bf16_kernel<64, 3, 1, 12, true>), grid, dim3(768), 0, s, a);
      else if (a.head_dim == 64) RT_LAUNCH((attn_bf16_kernel<64, 3, 1, 12, false>), grid, dim3(768), 0, s, a);
      else return hipErrorInvalidValue;
    } else if (a.rb_rows == 64) {
      // a third stage where each split holds long key ranges (16 or more chunks at the
      // longest context, one row block per sequence); otherwise two stages keep two
      // workgroups per compute unit
      const bool deep = a.row_blocks == 1 && a.max_pages / 4 >= 16 * a.splits;
      if (a.head_dim == 128 && f) RT_LAUNCH((attn_bf16_kernel<128, 2, 1, 8, true>), grid, dim3(512), 0, s, a);
      else if (a.head_dim == 128 && deep) RT_LAUNCH((attn_bf16_kernel<128, 3, 1, 8, false>), grid, dim3(512), 0, s, a);
      else if (a.head_dim == 128) RT_LAUNCH((attn_bf16_kernel<128, 2, 1, 8, false>), grid, dim3(512), 0, s, a);
      else if (a.head_dim == 64 && f) RT_LAUNCH((attn_bf16_kernel<64, 2, 1, 8, true>), grid, dim3(512), 0, s, a);
      else if (a.head_dim == 64 && deep) RT_LAUNCH((attn_bf16_kernel<64, 3, 1, 8, false>), grid, dim3(512), 0, s, a);
      else if (a.head_dim == 64) RT_LAUNCH((attn_bf16_kernel<64, 2, 1, 8, false>), grid, dim3(512), 0, s, a);
      else return hipErrorInvalidValue;
    } else {
      return hipErrorInvalidValue;
    }
  } else {
    if (a.rb_rows != kAttnRows) return hipErrorInvalidValue;
    if (a.head_dim == 128) RT_LAUNCH((attn_staged_kernel<T, 128>), grid, dim3(256), 0, s, a);
    else if (a.head_dim == 64) RT_LAUNCH((attn_staged_kernel<T, 64>), grid, dim3(256), 0, s, a);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
// Sixteen lanes per (token, head) row: lane c of the row owns hd elements c*PL ..
// c*PL + PL-1.  Each lane reads the (max, sum) pairs of splits c, c+16, .. for the row's
// maximum and denominator (two DPP row reductions), then walks all splits in order,
// loading a batch of partial O pieces and their maxima before weighting them, so the
// split weights need no cross-lane exchange.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_merge16_kernel(AttnArgs a) {
  constexpr int PL = HD / 16;                 // hd elements per lane
  constexpr int NB = 8;                       // splits per batch of loads
  const int c = threadIdx.x & 15;
  const int rl = blockIdx.x * 16 + (threadIdx.x >> 4);       // row within the row block
  const int s = blockIdx.z / a.row_blocks, rb = blockIdx.z % a.row_blocks, kvh = blockIdx.y;
  const int RBR = a.rb_rows;
  if (rl >= RBR) return;                      // whole rows leave together
  const int2 us = attn_unit_slots(a, blockIdx.z);
  const int S = us.y;                         // <= 64
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int r = rb * RBR + rl;
  if (r >= nq * G) return;
  if (S <= 0) {   // no split holds keys of this unit (not produced by the plans)
    const int tok = r / G, h = kvh * G + r % G;
#pragma unroll
    for (int e = 0; e < PL; ++e)
      ((T*)a.out)[pa_index(s * a.rows_per_seq + tok, h * HD + c * PL + e, a.ldo)] = Elem<T>::from_f32(0.f);
    return;
  }
  const size_t blk0 = (size_t)kvh * attn_head_blocks(a) + us.x;
  using P = typename PartOf<T>::P;
  const P* opp = reinterpret_cast<const P*>(a.opart) + (blk0 * RBR + rl) * HD + c * PL;   // split j: + j * RBR * HD
  const float* mlp = a.mlpart + (blk0 * RBR + rl) * 2;            // split j: + j * RBR * 2
  float mj[4], lj[4];
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = c + 16 * i;
    mj[i] = -INFINITY;
    lj[i] = 0.f;
    if (j < S) {
      const float2 v = *reinterpret_cast<const float2*>(mlp + (size_t)j * RBR * 2);
      mj[i] = v.x;
      lj[i] = v.y;
    }
    M = fmaxf(M, mj[i]);
  }
  M = row16_max(M);
  float den = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    den += (M == -INFINITY || mj[i] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mj[i] - M) * lj[i];
  den = row16_sum(den);
  float num[PL];
#pragma unroll
  for (int e = 0; e < PL; ++e) num[e] = 0.f;
  for (int j0 = 0; j0 < S; j0 += NB) {
    // loads past the last split read split S-1 again (all in flight); their weights are zero
    float ob[NB][PL];
    float2 mb[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int jj = j0 + j < S ? j0 + j : S - 1;
      PartOf<T>::template load<PL>(opp + (size_t)jj * RBR * HD, ob[j]);
      mb[j] = *reinterpret_cast<const float2*>(mlp + (size_t)jj * RBR * 2);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (j0 + j >= S) mb[j].x = -INFINITY;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      // weight of split j: its share exp2(m_j - M) * sum_j of the denominator
      const float f = (M == -INFINITY || mb[j].x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mb[j].x - M) * mb[j].y;
#pragma unroll
      for (int e = 0; e < PL; ++e) num[e] += f * ob[j][e];
    }
  }
  const int tok = r / G, h = kvh * G + r % G;
  T* out = (T*)a.out;
  const int orow = s * a.rows_per_seq + tok;
  const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
  for (int e = 0; e < PL; ++e) out[pa_index(orow, h * HD + c * PL + e, a.ldo)] = Elem<T>::from_f32(num[e] * inv);
}

template <typename T>
hipError_t attention_merge(const AttnArgs& a, hipStream_t s) {
  if (a.splits <= 1) return hipSuccess;
  // few splits (batches): sixteen lanes per row, one batch of loads (8B-shape batch 8:
  // 7.3 -> 3.5 us, 14B batch 16: 13.6 -> 4.4 us); many splits (batch 1, 32 splits): one
  // wave per row with all 32 splits' loads in flight at once (3.6 us against 5.8)
  if (a.splits <= 8) {
    dim3 grid(kAttnRowsMax / 16, a.n_kv_heads, a.n_seqs * a.row_blocks);
    if (a.head_dim == 128) RT_LAUNCH((attn_merge16_kernel<T, 128>), grid, dim3(256), 0, s, a);
    else if (a.head_dim == 64) RT_LAUNCH((attn_merge16_kernel<T, 64>), grid, dim3(256), 0, s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  dim3 grid(kAttnRowsMax / 4, a.n_kv_heads, a.n_seqs * a.row_blocks);
  if (a.head_dim == 128) RT_LAUNCH((attn_merge_kernel<T, 128>), grid, dim3(256), 0, s, a);
  else if (a.head_dim == 64) RT_LAUNCH((attn_merge_kernel<T, 64>), grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}
template <typename T>
hipError_t attention(const AttnArgs& a, hipStream_t s) {
  hipError_t e = attention_partials<T>(a, s);
  return e != hipSuccess ? e : attention_merge<T>(a, s);
}
template hipError_t attention<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attention<float>(const AttnArgs&, hipStream_t);
template hipError_t attention_partials<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attention_partials<float>(const AttnArgs&, hipStream_t);
template hipError_t attention_merge<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attention_merge<float>(const AttnArgs&, hipStream_t);

}  // namespace rt
