#include "misc.h"

namespace rt {

// ------------------------------------------------------------------ RMSNorm
template <typename K> struct KeepT;
template <> struct KeepT<uint16_t> { __device__ static uint16_t of(float v) { return f32_to_f16(v); } };
template <> struct KeepT<float> { __device__ static float of(float v) { return v; } };

// One workgroup per row, single pass: each thread keeps its 8-element chunks of the row
// in registers (hidden <= 8192), and writes the normalised row in the packed GEMM-operand
// layout (one 8-element run per chunk) plus an optional row-major retained copy.  With a
// fold, the pending k-slab partials of the producing GEMM are first summed (slab order)
// and added to the row, which is written back (and optionally captured, packed).  Every
// load of the row (x, partials, weight) is issued before the first use, so the row costs
// one memory latency; NP is the partial count when known at compile time (-1: runtime,
// at most 8), NTH the threads of the workgroup (1024 / NTH chunks per thread).
template <typename T, typename K, int NP, int NTH>
__global__ __launch_bounds__(NTH) void rmsnorm_kernel(float* __restrict__ x, int ldx,
                                                      const T* __restrict__ w, int d, float eps,
                                                      T* __restrict__ out, int ldg, K* keep, int ldk,
                                                      NormFold fold) {
  constexpr int MAXP = NP >= 0 ? NP : 8;
  constexpr int JM = 1024 / NTH;            // 8-float chunks per thread (d <= 8192)
  constexpr int NWV = NTH / 64;
  __shared__ float red[NWV];
  const int row = blockIdx.x;
  float* xr = x + (size_t)row * ldx;
  const int nch = d / 8;
  const int np = NP >= 0 ? NP : fold.n_part;
  float4 xa[JM][2], pa[JM][MAXP > 0 ? MAXP : 1][2];
  Frag<T> wf[JM];
#pragma unroll
  for (int j = 0; j < JM; ++j) {
    const int c = threadIdx.x + j * NTH;
    if (c < nch) {
      wf[j].load(w + 8 * c);
      xa[j][0] = *reinterpret_cast<const float4*>(xr + 8 * c);
      xa[j][1] = *reinterpret_cast<const float4*>(xr + 8 * c + 4);
#pragma unroll
      for (int z = 0; z < MAXP; ++z)
        if (z < np) {
          const float* pz = fold.part + z * fold.part_stride + (size_t)row * ldx + 8 * c;
          pa[j][z][0] = *reinterpret_cast<const float4*>(pz);
          pa[j][z][1] = *reinterpret_cast<const float4*>(pz + 4);
        }
    }
  }
  float v[JM][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < JM; ++j) {
    const int c = threadIdx.x + j * NTH;
    if (c < nch) {
      v[j][0] = xa[j][0].x; v[j][1] = xa[j][0].y; v[j][2] = xa[j][0].z; v[j][3] = xa[j][0].w;
      v[j][4] = xa[j][1].x; v[j][5] = xa[j][1].y; v[j][6] = xa[j][1].z; v[j][7] = xa[j][1].w;
      if (np > 0) {
        float t[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = 0.f;
#pragma unroll
        for (int z = 0; z < MAXP; ++z)
          if (z < np) {
            t[0] += pa[j][z][0].x; t[1] += pa[j][z][0].y; t[2] += pa[j][z][0].z; t[3] += pa[j][z][0].w;
            t[4] += pa[j][z][1].x; t[5] += pa[j][z][1].y; t[6] += pa[j][z][1].z; t[7] += pa[j][z][1].w;
          }
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] += t[e];
        *reinterpret_cast<float4*>(xr + 8 * c) = make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
        *reinterpret_cast<float4*>(xr + 8 * c + 4) = make_float4(v[j][4], v[j][5], v[j][6], v[j][7]);
        if (fold.cap) {
          Frag<T> cf;
#pragma unroll
          for (int e = 0; e < 8; ++e) cf.set(e, v[j][e]);
          cf.store((T*)fold.cap + pa_index(row, fold.cap_k0 + 8 * c, (size_t)fold.ldcap));
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[j][e] * v[j][e];
    }
  }
  ss = warp_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = red[0];
#pragma unroll
  for (int i = 1; i < NWV; ++i) tot += red[i];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int j = 0; j < JM; ++j) {
    const int c = threadIdx.x + j * NTH;
    if (c < nch) {
      Frag<T> f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float y = v[j][e] * inv * wf[j].get(e);
        f.set(e, y);
        if (keep) keep[(size_t)row * ldk + 8 * c + e] = KeepT<K>::of(y);
      }
      f.store(out + pa_index(row, 8 * c, (size_t)ldg));
    }
  }
}

template <typename T, typename K>
void rmsnorm(float* x, int ldx, const T* w, int d, float eps, int rows, T* out, int ldg,
             K* keep, int ldk, const NormFold& fold, hipStream_t s) {
  if (rows <= 0) return;
  // 256 threads with up to four 8-float chunks each; more than four partials (up to 8,
  // the mid-size kernel's slabs): 1024 threads with one chunk each, so that every load
  // of a row stays in flight within the register budget
  if (fold.n_part == 0)
    RT_LAUNCH((rmsnorm_kernel<T, K, 0, 256>), dim3(rows), dim3(256), 0, s, x, ldx, w, d, eps, out, ldg, keep, ldk, fold);
  else if (fold.n_part == 4)
    RT_LAUNCH((rmsnorm_kernel<T, K, 4, 256>), dim3(rows), dim3(256), 0, s, x, ldx, w, d, eps, out, ldg, keep, ldk, fold);
  else
    RT_LAUNCH((rmsnorm_kernel<T, K, -1, 1024>), dim3(rows), dim3(1024), 0, s, x, ldx, w, d, eps, out, ldg, keep, ldk, fold);
}
template void rmsnorm<bf16_t, uint16_t>(float*, int, const bf16_t*, int, float, int, bf16_t*, int,
                                        uint16_t*, int, const NormFold&, hipStream_t);
template void rmsnorm<float, float>(float*, int, const float*, int, float, int, float*, int,
                                    float*, int, const NormFold&, hipStream_t);

// ------------------------------------------------------------------ embeddings
template <typename K> struct KeepRead;
template <> struct KeepRead<uint16_t> { __device__ static float of(uint16_t v) { return f16_to_f32(v); } };
template <> struct KeepRead<float> { __device__ static float of(float v) { return v; } };

template <typename T>
__global__ void embed_rows_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ tok,
                                  float* __restrict__ x, int ldx) {
  const int row = blockIdx.x;
  const T* er = E + (size_t)tok[row] * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)row * ldx + i] = Elem<T>::to_f32(er[i]);
}
template <typename T>
void embed_rows(const T* embed, int d, const int32_t* tokens, int rows, float* x, int ldx, hipStream_t s) {
  if (rows <= 0) return;
  RT_LAUNCH((embed_rows_kernel<T>), dim3(rows), dim3(256), 0, s, embed, d, tokens, x, ldx);
}

// Rows (s, j) with 1 <= j <= cond_len take m_j = hD[s][r + j] when hD is given (the
// overwrite ablation); every other row is E[anchor] (j = 0) or E[mask].
template <typename T, typename K>
__global__ void embed_block_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ st,
                                   int mask, int bk, const K* __restrict__ hD, float* x, float* et, int ldx) {
  const int row = blockIdx.x, sq = row / bk, j = row % bk;
  const bool cond = hD && j >= 1 && j <= st[sq * kStateFields + ST_COND_LEN];
  if (cond) {
    const K* pm = hD + ((size_t)sq * bk + st[sq * kStateFields + ST_R] + j) * d;
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
      const float v = KeepRead<K>::of(pm[i]);
      x[(size_t)row * ldx + i] = v;
      et[(size_t)row * ldx + i] = v;
    }
    return;
  }
  const int tok = j == 0 ? st[sq * kStateFields + ST_ANCHOR] : mask;
  const T* er = E + (size_t)tok * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = Elem<T>::to_f32(er[i]);
    x[(size_t)row * ldx + i] = v;
    if (et) et[(size_t)row * ldx + i] = v;
  }
}
template <typename T, typename K>
void embed_block(const T* embed, int d, const int32_t* state, int mask_token, int n_seqs, int bk, const K* hD,
                 float* x, float* etilde, int ldx, hipStream_t s) {
  RT_LAUNCH((embed_block_kernel<T, K>), dim3(n_seqs * bk), dim3(256), 0, s, embed, d, state,
                     mask_token, bk, hD, x, etilde, ldx);
}

template <typename T>
__global__ void embed_verify_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ st,
                                    const uint64_t* __restrict__ dkeys, int forced, int32_t* dtok, int bk,
                                    float* x, int ldx) {
  const int row = blockIdx.x, sq = row / bk, j = row % bk;
  int tok;
  if (j == 0) tok = st[sq * kStateFields + ST_ANCHOR];
  else tok = forced ? dtok[row] : key_index(dkeys[row]);
  __syncthreads();
  if (threadIdx.x == 0) dtok[row] = tok;
  const T* er = E + (size_t)tok * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)row * ldx + i] = Elem<T>::to_f32(er[i]);
}
template <typename T>
void embed_verify(const T* embed, int d, const int32_t* state, const uint64_t* dkeys, int forced,
                  int32_t* dtok, int n_seqs, int bk, float* x, int ldx, hipStream_t s) {
  RT_LAUNCH((embed_verify_kernel<T>), dim3(n_seqs * bk), dim3(256), 0, s, embed, d, state, dkeys,
                     forced, dtok, bk, x, ldx);
}

// ------------------------------------------------------------------ conditioning gather

// row (s, j): m_j = hD[s][r + j], u_j = hT[s][r + j - 1] for 1 <= j <= cond_len, else 0.
// raw: the uncorrected signal r_j = m_j goes straight into er[:, d:2d] and mu is not used.
template <typename T, typename K>
__global__ void cond_prep_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ st, int mask,
                                 const K* __restrict__ hD, const K* __restrict__ hT, int bk,
                                 float* __restrict__ mu, float* __restrict__ er, int ldg, int raw) {
  const int row = blockIdx.x, sq = row / bk, j = row % bk;
  const int r = st[sq * kStateFields + ST_R], cl = st[sq * kStateFields + ST_COND_LEN];
  const bool cond = j >= 1 && j <= cl;
  const K* pm = hD + ((size_t)sq * bk + (cond ? r + j : 0)) * d;
  const K* pu = hT + ((size_t)sq * bk + (cond ? r + j - 1 : 0)) * d;
  const int tok = j == 0 ? st[sq * kStateFields + ST_ANCHOR] : mask;
  const T* pe = E + (size_t)tok * d;
  if (raw) {
    for (int i = threadIdx.x; i < d; i += blockDim.x) {
      er[pa_index(row, i, ldg)] = Elem<T>::to_f32(pe[i]);
      er[pa_index(row, d + i, ldg)] = cond ? KeepRead<K>::of(pm[i]) : 0.f;
    }
    return;
  }
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    mu[pa_index(row, i, ldg)] = cond ? KeepRead<K>::of(pm[i]) : 0.f;
    mu[pa_index(row, d + i, ldg)] = cond ? KeepRead<K>::of(pu[i]) : 0.f;
    er[pa_index(row, i, ldg)] = Elem<T>::to_f32(pe[i]);
  }
}
template <typename T, typename K>
void cond_prep(const T* embed, int d, const int32_t* state, int mask_token, const K* hD, const K* hT,
               int n_seqs, int bk, float* mu, float* er, int ldg, int raw, hipStream_t s) {
  RT_LAUNCH((cond_prep_kernel<T, K>), dim3(n_seqs * bk), dim3(256), 0, s, embed, d, state,
                     mask_token, hD, hT, bk, mu, er, ldg, raw);
}

// ------------------------------------------------------------------ low-rank conditioning
// Rows (s, j), four per workgroup, 64 output columns per workgroup:
//   rho = lat[:64] + beta * C_up lat[64:96]   (lat = [A m ; C_down [m; u]], fp32)
//   x = e + (V rho) * sigmoid(ge + G rho) on conditioned rows 1..cond_len, else e,
// with ge = W_g[:, :d] E[mask] precomputed (every conditioned row is a mask row).
template <typename T>
__global__ __launch_bounds__(256) void lowrank_fuse_kernel(const float* __restrict__ lat, const T* __restrict__ cup,
                                                           const T* __restrict__ V, const T* __restrict__ G,
                                                           const float* __restrict__ ge, float beta,
                                                           const T* __restrict__ E, int d, const int32_t* st,
                                                           int mask, int rows, int bk, float* x, float* et) {
  __shared__ float rho[4][kLowRankLatent];
  const int t = threadIdx.x, r = t >> 6, o = t & 63;
  const int row = blockIdx.y * 4 + r;
  const bool live = row < rows;
  const int sq = live ? row / bk : 0, j = live ? row % bk : 0;
  const bool cond = live && j >= 1 && j <= st[sq * kStateFields + ST_COND_LEN];
  if (live) {
    const float* lr = lat + (size_t)row * kLowRankLat;
    float c = 0.f;
#pragma unroll 8
    for (int k = 0; k < kLowRankCorr; ++k) c += Elem<T>::to_f32(cup[o * kLowRankCorr + k]) * lr[kLowRankLatent + k];
    rho[r][o] = lr[o] + beta * c;
  }
  __syncthreads();
  const int i = blockIdx.x * 64 + o;
  if (!live || i >= d) return;
  const int tok = j == 0 ? st[sq * kStateFields + ST_ANCHOR] : mask;
  float v = Elem<T>::to_f32(E[(size_t)tok * d + i]);
  if (cond) {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll 8
    for (int k = 0; k < kLowRankLatent; ++k) {
      s1 += Elem<T>::to_f32(V[(size_t)i * kLowRankLatent + k]) * rho[r][k];
      s2 += Elem<T>::to_f32(G[(size_t)i * kLowRankLatent + k]) * rho[r][k];
    }
    v += s1 / (1.0f + expf(-(ge[i] + s2)));
  }
  x[(size_t)row * d + i] = v;
  et[(size_t)row * d + i] = v;
}
template <typename T>
void lowrank_fuse(const float* lat, const T* cup, const T* V, const T* G, const float* ge, float beta, const T* embed,
                  int d, const int32_t* state, int mask, int n_seqs, int bk, float* x, float* etilde, hipStream_t s) {
  const int rows = n_seqs * bk;
  RT_LAUNCH((lowrank_fuse_kernel<T>), dim3((d + 63) / 64, (rows + 3) / 4), dim3(256), 0, s, lat, cup, V, G, ge, beta,
            embed, d, state, mask, rows, bk, x, etilde);
}

// ge[i] = sum_k W_g[i][k] E[mask][k] over the first d columns of W_g (row-major [d][2d]).
template <typename T>
__global__ void lowrank_gate_bias_kernel(const T* __restrict__ wg, const T* __restrict__ E, int d, int mask,
                                         float* ge) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= d) return;
  const T* w = wg + (size_t)i * 2 * d;
  const T* e = E + (size_t)mask * d;
  float acc = 0.f;
  for (int k = 0; k < d; ++k) acc += Elem<T>::to_f32(w[k]) * Elem<T>::to_f32(e[k]);
  ge[i] = acc;
}
template <typename T>
void lowrank_gate_bias(const T* wg, const T* embed, int d, int mask, float* ge, hipStream_t s) {
  RT_LAUNCH((lowrank_gate_bias_kernel<T>), dim3((d + 255) / 256), dim3(256), 0, s, wg, embed, d, mask, ge);
}

// ------------------------------------------------------------------ acceptance / rollback
// One wave per sequence.  Draft tokens y^_i (i = 1..B) sit in dtok[s][i]; the target's
// token for block position i is the argmax of verify row i-1.
__global__ void accept_kernel(int32_t* st_all, const int32_t* __restrict__ dtok,
                              const uint64_t* __restrict__ tkeys, int32_t* ttok, int bk,
                              int32_t* out_tok, int32_t* out_n, int32_t* out_a) {
  const int sq = blockIdx.x, lane = threadIdx.x;
  const int B = bk - 1;
  int32_t* st = st_all + sq * kStateFields;
  const int yt = lane < bk ? key_index(tkeys[(size_t)sq * bk + lane]) : -1;   // y^T_{lane+1}
  if (lane < bk) ttok[(size_t)sq * bk + lane] = yt;
  // mismatch at block position i = lane + 1 (1..B)
  const bool mis = (lane < B) && (dtok[(size_t)sq * bk + lane + 1] != yt);
  const unsigned long long ball = __ballot(mis);
  const int A = ball ? __ffsll((long long)ball) - 1 : B;
  const int budget = st[ST_BUDGET];
  const int n_new = budget > 0 ? min(A + 1, budget) : 0;
  const int corr = __shfl(yt, A, 64);                               // y^T_{A+1}
  if (lane < bk) {
    int v = -1;
    if (lane < n_new) v = (lane < A) ? dtok[(size_t)sq * bk + lane + 1] : corr;
    out_tok[(size_t)sq * bk + lane] = v;
  }
  if (lane == 0) {
    out_n[sq] = n_new;
    out_a[sq] = n_new > 0 ? A : 0;
    if (budget > 0) {
      const int P = st[ST_SEQ_LEN];
      st[ST_ROUND_POS] = P;
      st[ST_APPEND] = A + 1;
      st[ST_ACCEPT] = A;
      st[ST_SEQ_LEN] = P + A + 1;        // rows P+A+1.. of the target KV are rolled back
      st[ST_ANCHOR] = corr;
      st[ST_BUDGET] = budget - n_new;
      st[ST_ROUND] += 1;
      if (A < B - 1) { st[ST_R] = A + 1; st[ST_COND_LEN] = B - (A + 1); }
      else { st[ST_R] = 0; st[ST_COND_LEN] = 0; }
    } else {
      st[ST_APPEND] = 0;
      st[ST_ROUND_POS] = st[ST_SEQ_LEN];
    }
  }
}
void accept(int32_t* state, const int32_t* dtok, const uint64_t* tkeys, int32_t* ttok, int n_seqs, int bk,
            int32_t* out_tokens, int32_t* out_n, int32_t* out_a, hipStream_t s) {
  RT_LAUNCH(accept_kernel, dim3(n_seqs), dim3(64), 0, s, state, dtok, tkeys, ttok, bk, out_tokens,
                     out_n, out_a);
}

// Target-only greedy step: one thread per sequence commits the argmax of its row (the
// K/V of the anchor row were written at position seq_len by this step's layers).  The
// token goes to out[s * ld_out + k], k = *step, which the last thread advances.
__global__ __launch_bounds__(1024) void ar_commit_kernel(int32_t* st_all, const uint64_t* __restrict__ tkeys,
                                                         const int32_t* sampled, int n_seqs, int32_t* out, int ld_out,
                                                         int32_t* step) {
  const int k = *step;
  const int sq = threadIdx.x;
  if (sq < n_seqs) {
    int32_t* st = st_all + sq * kStateFields;
    const int budget = st[ST_BUDGET];
    int v = -1;
    if (budget > 0) {
      v = sampled ? sampled[sq] : key_index(tkeys[sq]);
      st[ST_ROUND] += 1;
      const int P = st[ST_SEQ_LEN] + 1;
      st[ST_SEQ_LEN] = P;
      st[ST_ANCHOR] = v;
      st[ST_BUDGET] = budget - 1;
      st[ST_ROUND_POS] = P;
      st[ST_APPEND] = 0;
      st[ST_ACCEPT] = 0;
      st[ST_R] = 0;
      st[ST_COND_LEN] = 0;
    }
    out[(size_t)sq * ld_out + k] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) *step = k + 1;
}
void ar_commit(int32_t* state, const uint64_t* tkeys, const int32_t* sampled, int n_seqs, int32_t* out, int ld_out,
               int32_t* step, hipStream_t s) {
  const int threads = (n_seqs + 63) / 64 * 64;
  RT_LAUNCH(ar_commit_kernel, dim3(1), dim3(threads), 0, s, state, tkeys, sampled, n_seqs, out, ld_out, step);
}

__global__ void set_ints_kernel(int32_t* dst, int n, int v0, int v1, int v2, int v3) {
  const int v[4] = {v0, v1, v2, v3};
  if (threadIdx.x < n && threadIdx.x < 4) dst[threadIdx.x] = v[threadIdx.x];
}
void set_ints(int32_t* dst, int n, int v0, int v1, int v2, int v3, hipStream_t s) {
  RT_LAUNCH(set_ints_kernel, dim3(1), dim3(64), 0, s, dst, n, v0, v1, v2, v3);
}

__global__ void first_token_kernel(int32_t* st_all, int sq, const uint64_t* keys, const int32_t* sampled, int plen,
                                   int budget, int32_t* first_out) {
  if (threadIdx.x != 0) return;
  int32_t* st = st_all + sq * kStateFields;
  const int tok = sampled ? sampled[sq] : key_index(keys[0]);
  st[ST_SEQ_LEN] = plen;
  st[ST_ANCHOR] = tok;
  st[ST_R] = 0;
  st[ST_COND_LEN] = 0;
  st[ST_BUDGET] = budget - 1;
  st[ST_ROUND_POS] = plen;
  st[ST_APPEND] = 0;
  st[ST_ACCEPT] = 0;
  st[ST_ROUND] = 0;
  first_out[sq] = tok;
}
void first_token(int32_t* state, int seq, const uint64_t* keys, const int32_t* sampled, int prompt_len, int budget,
                 int32_t* first_out, hipStream_t s) {
  RT_LAUNCH(first_token_kernel, dim3(1), dim3(64), 0, s, state, seq, keys, sampled, prompt_len, budget,
                     first_out);
}

__global__ void fill_zero_kernel(uint4* p, size_t n16) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}
void fill_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return;
  size_t g = (n16 + 255) / 256;
  if (g > 8192) g = 8192;
  RT_LAUNCH(fill_zero_kernel, dim3((unsigned)g), dim3(256), 0, s, (uint4*)p, n16);
}

// Plain read of a buffer: every byte loaded once with non-temporal 16-byte loads (as the
// weight streams), workgroup b reading the b-th contiguous share, eight loads in flight
// per lane; the values feed a store guarded by a runtime flag (passed as 0), so no load
// can be dropped and nothing is written.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* __restrict__ p, size_t n16, uint32_t* sink,
                                                          int store) {
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t b0 = blockIdx.x * per, b1 = b0 + per < n16 ? b0 + per : n16;
  const v4u* q = reinterpret_cast<const v4u*>(p);
  uint32_t acc = 0;
  for (size_t i = b0 + threadIdx.x; i < b1; i += 8 * (size_t)blockDim.x) {
    v4u v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const size_t j = i + (size_t)u * blockDim.x;
      v[u] = __builtin_nontemporal_load(q + (j < b1 ? j : i));
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (store) sink[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}
void stream_read(const void* p, size_t bytes, int grid, uint32_t* sink, hipStream_t s) {
  RT_LAUNCH(stream_read_kernel, dim3((unsigned)grid), dim3(256), 0, s, (const uint4*)p, bytes / 16, sink, 0);
}

template void embed_rows<bf16_t>(const bf16_t*, int, const int32_t*, int, float*, int, hipStream_t);
template void embed_rows<float>(const float*, int, const int32_t*, int, float*, int, hipStream_t);
template void embed_block<bf16_t, uint16_t>(const bf16_t*, int, const int32_t*, int, int, int, const uint16_t*,
                                            float*, float*, int, hipStream_t);
template void embed_block<float, float>(const float*, int, const int32_t*, int, int, int, const float*, float*,
                                        float*, int, hipStream_t);
template void embed_verify<bf16_t>(const bf16_t*, int, const int32_t*, const uint64_t*, int, int32_t*, int,
                                   int, float*, int, hipStream_t);
template void embed_verify<float>(const float*, int, const int32_t*, const uint64_t*, int, int32_t*, int,
                                  int, float*, int, hipStream_t);
template void lowrank_fuse<bf16_t>(const float*, const bf16_t*, const bf16_t*, const bf16_t*, const float*, float,
                                   const bf16_t*, int, const int32_t*, int, int, int, float*, float*, hipStream_t);
template void lowrank_fuse<float>(const float*, const float*, const float*, const float*, const float*, float,
                                  const float*, int, const int32_t*, int, int, int, float*, float*, hipStream_t);
template void lowrank_gate_bias<bf16_t>(const bf16_t*, const bf16_t*, int, int, float*, hipStream_t);
template void lowrank_gate_bias<float>(const float*, const float*, int, int, float*, hipStream_t);
template void cond_prep<bf16_t, uint16_t>(const bf16_t*, int, const int32_t*, int, const uint16_t*,
                                          const uint16_t*, int, int, float*, float*, int, int, hipStream_t);
template void cond_prep<float, float>(const float*, int, const int32_t*, int, const float*, const float*, int,
                                      int, float*, float*, int, int, hipStream_t);

}  // namespace rt
