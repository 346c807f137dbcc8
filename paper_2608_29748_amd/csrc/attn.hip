// Paged GQA attention with MFMA.  One workgroup (4 waves) owns one sequence, one KV
// head, one block of 64 (token, head) query rows and one contiguous share of the key
// range; each wave owns a 16-row MFMA tile and runs an online softmax over 32-key
// chunks staged in LDS.  K pages are stored [token][hd] so a K row is a contiguous
// B-operand fragment of S = Q K^T; V pages are stored transposed ([hd][token]) so a
// V^T row is a contiguous B-operand fragment of O = P V.  Split partials
// (unnormalised O, running max, running sum) are merged by a second kernel.
#include "attn.h"

namespace rt {

constexpr int kChunk = 64;      // keys per LDS chunk (four pages)
constexpr int kMaxSplitPages = 1024;   // page ids of one split held in LDS (16384 keys)

size_t attn_partial_floats(int n_seqs, int n_kv_heads, int row_blocks, int splits, int head_dim) {
  return (size_t)n_seqs * n_kv_heads * row_blocks * splits * kAttnRows * head_dim;
}
int attn_min_splits(int max_keys) { return (max_keys + kMaxSplitPages * kPage - 1) / (kMaxSplitPages * kPage); }

// Scores are computed transposed, S^T = K Q^T: in the accumulator layout a lane holds
// keys 4*(lane/16)+i of one query (column lane%16), so the softmax is a per-lane
// reduction plus two cross-lane steps, and the probabilities feed O^T = V^T P^T as the
// B operand straight from registers (no LDS transpose).  In each 32-key MFMA step a
// lane supplies keys {4g..4g+3} and {16+4g..16+4g+3} of the step (g = lane/16); the
// V^T fragment from LDS uses the same key order.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
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
  const int split = blockIdx.x, kvh = blockIdx.y;
  const int s = blockIdx.z / a.row_blocks, rb = blockIdx.z % a.row_blocks;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int P = a.pos0[s * a.seq_stride];
  const int nrows = nq * G;                      // valid (token, head) rows of this sequence
  const int row0 = rb * kAttnRows;               // first row of this workgroup
  if (row0 >= nrows) return;
  const int last_tok = min(nrows, row0 + kAttnRows) - 1;
  const int kv_end = a.causal ? P + last_tok / G + 1 : P + nq;   // keys [0, kv_end)
  const int nchunks = (kv_end + kChunk - 1) / kChunk;
  const int cps = (nchunks + a.splits - 1) / a.splits;
  const int c_beg = split * cps, c_end = min(nchunks, c_beg + cps);
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
    const size_t blk = (((size_t)s * a.n_kv_heads + kvh) * a.row_blocks + rb) * a.splits + split;
    float* op = a.opart + blk * kAttnRows * HD;
    float* ml = a.mlpart + blk * kAttnRows * 2;
    const int rl = w * 16 + c16;
#pragma unroll
    for (int t = 0; t < NHT; ++t)
      *reinterpret_cast<float4*>(op + (size_t)rl * HD + t * 16 + 4 * g4) = make_float4(o[t][0], o[t][1], o[t][2], o[t][3]);
    if (g4 == 0) { ml[rl * 2] = mrun; ml[rl * 2 + 1] = lrun; }
  }
}

// One wave per (sequence, kv head, row).  Lane j reads split j's running max and sum
// (64 splits per pass); the weights exp2(m_j - M) are broadcast by shuffles while the
// lanes accumulate the head dimension, eight splits' partial rows in flight at a time.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int PL = HD / 64;                 // hd elements per lane
  const int lane = threadIdx.x & 63;
  const int rl = blockIdx.x * 4 + (threadIdx.x >> 6);        // row within the row block
  const int s = blockIdx.z / a.row_blocks, rb = blockIdx.z % a.row_blocks, kvh = blockIdx.y;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int nq = a.nq ? a.nq[s * a.seq_stride] : a.rows_per_seq;
  const int r = rb * kAttnRows + rl;
  if (r >= nq * G) return;
  const size_t blk0 = (((size_t)s * a.n_kv_heads + kvh) * a.row_blocks + rb) * a.splits;
  float M = -INFINITY;
  for (int sp = lane; sp < a.splits; sp += 64) M = fmaxf(M, a.mlpart[((blk0 + sp) * kAttnRows + rl) * 2]);
  M = warp_max(M);
  float num[PL], den = 0.f;
#pragma unroll
  for (int j = 0; j < PL; ++j) num[j] = 0.f;
  if (M != -INFINITY) {
    for (int base = 0; base < a.splits; base += 64) {
      const int sp = base + lane;
      float f = 0.f;
      if (sp < a.splits) {
        const float* ml = a.mlpart + ((blk0 + sp) * kAttnRows + rl) * 2;
        f = (ml[0] == -INFINITY) ? 0.f : exp2f(ml[0] - M);
        den += f * ml[1];
      }
      const int n = min(64, a.splits - base);
      for (int j0 = 0; j0 < n; j0 += 8) {
        float o[8][PL], fw[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int jj = j0 + u < n ? j0 + u : n - 1;
          fw[u] = __shfl(f, jj, 64) * (j0 + u < n ? 1.f : 0.f);
          const float* op = a.opart + ((blk0 + base + jj) * kAttnRows + rl) * HD;
#pragma unroll
          for (int j = 0; j < PL; ++j) o[u][j] = op[lane + 64 * j];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int j = 0; j < PL; ++j) num[j] += fw[u] * o[u][j];
      }
    }
  }
  den = warp_sum(den);
  const int tok = r / G, h = kvh * G + r % G;
  T* out = (T*)a.out;
  const int orow = s * a.rows_per_seq + tok;
  const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
  for (int j = 0; j < PL; ++j) out[pa_index(orow, h * HD + lane + 64 * j, a.ldo)] = Elem<T>::from_f32(num[j] * inv);
}

template <typename T>
hipError_t attention(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.splits, a.n_kv_heads, a.n_seqs * a.row_blocks);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL((attn_kernel<T, 128>), grid, dim3(256), 0, s, a);
    if (a.splits > 1)
      hipLaunchKernelGGL((attn_merge_kernel<T, 128>), dim3(kAttnRows / 4, a.n_kv_heads, a.n_seqs * a.row_blocks),
                         dim3(256), 0, s, a);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL((attn_kernel<T, 64>), grid, dim3(256), 0, s, a);
    if (a.splits > 1)
      hipLaunchKernelGGL((attn_merge_kernel<T, 64>), dim3(kAttnRows / 4, a.n_kv_heads, a.n_seqs * a.row_blocks),
                         dim3(256), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t attention<bf16_t>(const AttnArgs&, hipStream_t);
template hipError_t attention<float>(const AttnArgs&, hipStream_t);

}  // namespace rt
