// Paged GQA attention with MFMA.  One workgroup (4 waves) owns one sequence, one KV
// head, one block of 64 (token, head) query rows and one contiguous share of the key
// range; each wave owns a 16-row MFMA tile and runs an online softmax over 32-key
// chunks staged in LDS.  K pages are stored [token][hd] so a K row is a contiguous
// B-operand fragment of S = Q K^T; V pages are stored transposed ([hd][token]) so a
// V^T row is a contiguous B-operand fragment of O = P V.  Split partials
// (unnormalised O, running max, running sum) are merged by a second kernel.
#include "attn.h"

namespace rt {

constexpr int kChunk = 32;      // keys per LDS chunk (two pages)

size_t attn_partial_floats(int n_seqs, int n_kv_heads, int row_blocks, int splits, int head_dim) {
  return (size_t)n_seqs * n_kv_heads * row_blocks * splits * kAttnRows * head_dim;
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  constexpr int EB = Elem<T>::kBytes;
  constexpr int KPAD = HD + 16 / EB;       // LDS row pitch (elements) for K
  constexpr int VPAD = kChunk + 16 / EB;   // LDS row pitch for V^T and P
  constexpr int NHT = HD / 16;             // output hd tiles
  constexpr int NKS = HD / 32;             // k-steps over hd for S
  __shared__ __attribute__((aligned(16))) T sK[kChunk][KPAD];
  __shared__ __attribute__((aligned(16))) T sV[HD][VPAD];
  __shared__ __attribute__((aligned(16))) T sP[4][16][VPAD];
  // bf16: probabilities enter P V as hi + lo bf16 parts (~16 significand bits)
  constexpr bool kSplitP = sizeof(T) == 2;
  __shared__ __attribute__((aligned(16))) T sPl[kSplitP ? 4 : 1][16][VPAD];

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

  // This wave's 16 rows: row = row0 + w*16 + (lane%16) for A fragments;
  // accumulator rows are row0 + w*16 + 4*g4 + i.
  const int arow = row0 + w * 16 + c16;
  Frag<T> qf[NKS];
  {
    const int r = min(arow, nrows - 1);
    const int tok = r / G, h = kvh * G + r % G;
    const T* qp = (const T*)a.q + (size_t)(s * a.rows_per_seq + tok) * a.n_q_heads * HD + (size_t)h * HD;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks].load(qp + ks * 32 + g4 * 8);
  }
  int qpos[4];
  bool rvalid[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = row0 + w * 16 + 4 * g4 + i;
    rvalid[i] = r < nrows;
    qpos[i] = P + (rvalid[i] ? r / G : 0);
  }
  const float sl2 = a.scale * 1.4426950408889634f;
  float mrun[4], lrun[4];
  f32x4 o[NHT];
#pragma unroll
  for (int i = 0; i < 4; ++i) { mrun[i] = -INFINITY; lrun[i] = 0.f; }
#pragma unroll
  for (int t = 0; t < NHT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t head_page = (size_t)kPage * HD;   // elements of one (page, head) slice
  // Each thread stages NP 16-byte pieces of a chunk (K pieces first, then V^T pieces);
  // the next chunk's pieces are loaded into registers while the current one is used.
  constexpr int KV16 = kChunk * HD * EB / 16;     // 16-byte pieces of K per chunk (same for V)
  constexpr int NP = 2 * KV16 / 256;
  uint4 pf[NP];
  auto fetch = [&](int c) {
    const int key0 = c * kChunk;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int p = threadIdx.x + j * 256;
      const bool isv = p >= KV16;
      const int e0 = (isv ? p - KV16 : p) * (16 / EB);
      const int pg = e0 / (int)head_page, within = e0 % (int)head_page;
      const int tok0 = key0 + pg * kPage;
      pf[j] = make_uint4(0, 0, 0, 0);
      if (c < c_end && tok0 < kv_end) {
        const int page = a.page_table[(size_t)s * a.max_pages + tok0 / kPage];
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
    // S = Q K^T for two 16-key subtiles
    f32x4 sacc[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      sacc[sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        Frag<T> kf;
        kf.load(&sK[sub * 16 + c16][ks * 32 + g4 * 8]);
        mma(sacc[sub], qf[ks], kf);
      }
    }
    // mask, online softmax
    float p[2][4], alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = -INFINITY;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        const int kp = key0 + sub * 16 + c16;
        const bool vis = rvalid[i] && kp < kv_end && (!a.causal || kp <= qpos[i]);
        const float v = vis ? sacc[sub][i] * sl2 : -INFINITY;
        p[sub][i] = v;
        mx = fmaxf(mx, v);
      }
      for (int off = 8; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      const float mnew = fmaxf(mrun[i], mx);
      if (mnew == -INFINITY) {
        alpha[i] = 1.f;
        p[0][i] = 0.f; p[1][i] = 0.f;
      } else {
        alpha[i] = exp2f(mrun[i] - mnew);
        p[0][i] = exp2f(p[0][i] - mnew);
        p[1][i] = exp2f(p[1][i] - mnew);
      }
      float rs = p[0][i] + p[1][i];
      for (int off = 8; off > 0; off >>= 1) rs += __shfl_xor(rs, off, 64);
      lrun[i] = lrun[i] * alpha[i] + rs;
      mrun[i] = mnew;
    }
#pragma unroll
    for (int t = 0; t < NHT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[t][i] *= alpha[i];
    // P: accumulator layout -> A-operand layout through this wave's LDS slot
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const T hi = Elem<T>::from_f32(p[sub][i]);
        sP[w][4 * g4 + i][sub * 16 + c16] = hi;
        if constexpr (kSplitP)
          sPl[w][4 * g4 + i][sub * 16 + c16] = Elem<T>::from_f32(p[sub][i] - Elem<T>::to_f32(hi));
      }
    __syncthreads();
    Frag<T> pf, pfl;
    pf.load(&sP[w][c16][g4 * 8]);
    if constexpr (kSplitP) pfl.load(&sPl[w][c16][g4 * 8]);
#pragma unroll
    for (int t = 0; t < NHT; ++t) {
      Frag<T> vf;
      vf.load(&sV[t * 16 + c16][g4 * 8]);
      mma(o[t], pf, vf);
      if constexpr (kSplitP) mma(o[t], pfl, vf);
    }
  }

  // write result (single split) or partials
  if (a.splits == 1) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = row0 + w * 16 + 4 * g4 + i;
      if (r >= nrows) continue;
      const int tok = r / G, h = kvh * G + r % G;
      const float inv = lrun[i] > 0.f ? 1.f / lrun[i] : 0.f;
      T* op = (T*)a.out;
      const int orow = s * a.rows_per_seq + tok;
#pragma unroll
      for (int t = 0; t < NHT; ++t) op[pa_index(orow, h * HD + t * 16 + c16, a.ldo)] = Elem<T>::from_f32(o[t][i] * inv);
    }
  } else {
    const size_t blk = (((size_t)s * a.n_kv_heads + kvh) * a.row_blocks + rb) * a.splits + split;
    float* op = a.opart + blk * kAttnRows * HD;
    float* ml = a.mlpart + blk * kAttnRows * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rl = w * 16 + 4 * g4 + i;
#pragma unroll
      for (int t = 0; t < NHT; ++t) op[(size_t)rl * HD + t * 16 + c16] = o[t][i];
      if (c16 == 0) { ml[rl * 2] = mrun[i]; ml[rl * 2 + 1] = lrun[i]; }
    }
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
