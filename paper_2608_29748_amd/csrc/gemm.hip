// Packed-weight MFMA GEMM with split-K fixup and fused epilogues (see gemm.h).
#include "gemm.h"

namespace rt {

// ------------------------------------------------------------------ packing

// out tile (nt, kt), lane l, element e  <-  W[n = src_tile*16 + l%16][k = kt*32 + (l/16)*8 + e]
// (zero for k >= K).  With Wb set, output tiles alternate Wa tile j / Wb tile j.
template <typename T>
__global__ void pack_kernel(const T* __restrict__ Wa, const T* __restrict__ Wb, int N, int K, int Kp,
                            T* __restrict__ out) {
  const int KT = Kp / kTileK;
  const int ntiles = (Wb ? 2 : 1) * (N / kTileN);
  const size_t total = (size_t)ntiles * KT * kWave;
  for (size_t c = blockIdx.x * (size_t)blockDim.x + threadIdx.x; c < total;
       c += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(c % kWave);
    const size_t tile = c / kWave;
    const int kt = (int)(tile % KT);
    const int nt = (int)(tile / KT);
    const T* src = Wa;
    int st = nt;
    if (Wb) { src = (nt & 1) ? Wb : Wa; st = nt >> 1; }
    const int n = st * kTileN + (lane % 16);
    const int k0 = kt * kTileK + (lane / 16) * 8;
    T* dst = out + c * 8;
    for (int e = 0; e < 8; ++e) {
      const int k = k0 + e;
      dst[e] = (k < K) ? src[(size_t)n * K + k] : (T)0;
    }
  }
}

template <typename T>
void pack_weights(const T* W, int N, int K, int Kp, T* out, hipStream_t s) {
  size_t total = (size_t)(N / kTileN) * (Kp / kTileK) * kWave;
  int grid = (int)((total + 255) / 256);
  if (grid > 65535 * 4) grid = 65535 * 4;
  hipLaunchKernelGGL(pack_kernel<T>, dim3(grid), dim3(256), 0, s, W, (const T*)nullptr, N, K, Kp, out);
}
template <typename T>
void pack_interleaved(const T* Wa, const T* Wb, int N, int K, int Kp, T* out, hipStream_t s) {
  size_t total = (size_t)2 * (N / kTileN) * (Kp / kTileK) * kWave;
  int grid = (int)((total + 255) / 256);
  if (grid > 65535 * 4) grid = 65535 * 4;
  hipLaunchKernelGGL(pack_kernel<T>, dim3(grid), dim3(256), 0, s, Wa, Wb, N, K, Kp, out);
}
template void pack_weights<bf16_t>(const bf16_t*, int, int, int, bf16_t*, hipStream_t);
template void pack_weights<float>(const float*, int, int, int, float*, hipStream_t);
template void pack_interleaved<bf16_t>(const bf16_t*, const bf16_t*, int, int, int, bf16_t*, hipStream_t);
template void pack_interleaved<float>(const float*, const float*, int, int, int, float*, hipStream_t);

// ------------------------------------------------------------------ A-operand fragments

// Loads eight consecutive k-values of an A row.  For AF32 with bf16 weights the fp32
// values are split as hi = bf16(x), lo = bf16(x - hi) and both are multiplied, so the
// product keeps ~16 significand bits of the fp32 input.
template <typename T, bool AF32> struct AFrag;
template <typename T> struct AFrag<T, false> {
  Frag<T> f;
  __device__ __forceinline__ void load(const void* p) { f.load((const T*)p); }
  __device__ __forceinline__ void mma_into(f32x4& acc, const Frag<T>& b) const { mma(acc, f, b); }
};
template <> struct AFrag<bf16_t, true> {
  Frag<bf16_t> hi, lo;
  __device__ __forceinline__ void load(const void* p) {
    const float4 x0 = *reinterpret_cast<const float4*>(p);
    const float4 x1 = *(reinterpret_cast<const float4*>(p) + 1);
    const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    for (int i = 0; i < 8; ++i) {
      const bf16_t h = f32_to_bf16(xs[i]);
      hi.v[i] = (short)h;
      lo.v[i] = (short)f32_to_bf16(xs[i] - bf16_to_f32(h));
    }
  }
  __device__ __forceinline__ void mma_into(f32x4& acc, const Frag<bf16_t>& b) const {
    mma(acc, hi, b);
    mma(acc, lo, b);
  }
};
template <> struct AFrag<float, true> : AFrag<float, false> {};

// ------------------------------------------------------------------ epilogues

template <typename T, int ROWS, int COLS, int LDT>
__device__ void run_epilogue(const EpiArgs& e, float (*t)[LDT], int m0, int n0) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  switch (e.kind) {
    case EPI_STORE_F32:
    case EPI_STORE_ACT:
    case EPI_RESID:
    case EPI_COND_R:
    case EPI_COND_GATE:
    case EPI_COND_OUT: {
      for (int idx = tid; idx < ROWS * COLS; idx += 256) {
        const int r = idx / COLS, c = idx % COLS;
        const int m = m0 + r, n = n0 + c;
        if (m >= e.M || n >= e.N) continue;
        const float y = t[r][c];
        if (e.kind == EPI_STORE_F32) {
          e.out_f32[(size_t)m * e.ldo + n] = y;
        } else if (e.kind == EPI_STORE_ACT) {
          ((T*)e.out_act)[(size_t)m * e.ldo + n] = Elem<T>::from_f32(y);
        } else if (e.kind == EPI_RESID) {
          float* px = e.resid + (size_t)m * e.ldr + n;
          const float x = *px + y;
          *px = x;
          if (e.cap) ((T*)e.cap)[(size_t)m * e.ldcap + n] = Elem<T>::from_f32(x);
        } else if (e.kind == EPI_COND_R) {
          e.out_f32[(size_t)m * e.ldo + n] = e.cond_m[(size_t)m * e.ld_cond_m + n] + e.beta * y;
        } else if (e.kind == EPI_COND_GATE) {
          e.out_f32[(size_t)m * e.ldo + n] = 1.0f / (1.0f + expf(-y));
        } else {  // EPI_COND_OUT
          const int s = m / e.rows_per_seq, j = m % e.rows_per_seq;
          const int tok = (j == 0) ? e.anchor[s * e.seq_stride] : e.mask_token;
          const float ev = Elem<T>::to_f32(((const T*)e.embed)[(size_t)tok * e.N + n]);
          const bool cond = (j >= 1) && (j <= e.cond_len[s * e.seq_stride]);
          const float x = cond ? ev + y * e.gate[(size_t)m * e.ld_gate + n] : ev;
          e.resid[(size_t)m * e.ldr + n] = x;
          e.etilde[(size_t)m * e.ldr + n] = x;
        }
      }
      break;
    }
    case EPI_SWIGLU: {
      // LDS columns: per 32-column group g, [g*32, g*32+16) gate tile, [g*32+16, g*32+32) up tile.
      constexpr int OC = COLS / 2;
      for (int idx = tid; idx < ROWS * OC; idx += 256) {
        const int r = idx / OC, j = idx % OC;
        const int m = m0 + r;
        const int cg = (j / 16) * 32 + (j % 16);
        if (m >= e.M || n0 + cg >= e.N) continue;
        const float g = t[r][cg], u = t[r][cg + 16];
        const float a = g / (1.0f + expf(-g)) * u;
        ((T*)e.out_act)[(size_t)m * e.ldo + n0 / 2 + j] = Elem<T>::from_f32(a);
      }
      break;
    }
    case EPI_ARGMAX: {
      for (int r = w; r < ROWS; r += 4) {
        const int m = m0 + r;
        if (m >= e.M) continue;
        uint64_t best = 0;
        for (int c = lane; c < COLS; c += 64) {
          const int n = n0 + c;
          if (n >= e.N) continue;
          const float y = t[r][c];
          if (e.out_f32) e.out_f32[(size_t)m * e.ldo + n] = y;
          const uint64_t k = argmax_key(y, (uint32_t)n);
          best = k > best ? k : best;
        }
        for (int o = 32; o > 0; o >>= 1) {
          const uint64_t other = __shfl_xor(best, o, 64);
          best = other > best ? other : best;
        }
        if (lane == 0) atomicMax((unsigned long long*)&e.keys[m], (unsigned long long)best);
      }
      break;
    }
    case EPI_QKV: {
      const int hd = e.head_dim, half = hd / 2;
      const int heads_per_item = 64 / half;          // 1 (hd 128) or 2 (hd 64)
      const int hh = lane / half, ei = lane % half;
      const int layer = n0 / e.layer_cols;
      const int cin = n0 % e.layer_cols;
      int region, hbase;                              // 0 q, 1 k, 2 v; first head of the tile
      if (cin < e.q_cols) { region = 0; hbase = cin / hd; }
      else if (cin < e.q_cols + e.kv_cols) { region = 1; hbase = (cin - e.q_cols) / hd; }
      else { region = 2; hbase = (cin - e.q_cols - e.kv_cols) / hd; }
      const int items_per_row = COLS / (hd * heads_per_item);
      for (int it = w; it < ROWS * items_per_row; it += 4) {
        const int r = it / items_per_row;
        const int c0 = (it % items_per_row) * hd * heads_per_item + hh * hd;
        const int m = m0 + r;
        if (m >= e.M) continue;
        const int s = m / e.rows_per_seq, i = m % e.rows_per_seq;
        if (e.nrows && i >= e.nrows[s * e.seq_stride]) continue;
        const int pos = e.pos0[s * e.seq_stride] + i;
        float x0 = t[r][c0 + ei], x1 = t[r][c0 + ei + half];
        const int head = hbase + (c0 / hd);
        if (region < 2) {
          float ss = x0 * x0 + x1 * x1;
          for (int o = half / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
          const float inv = 1.0f / sqrtf(ss / (float)hd + e.eps);
          const T* nw = (const T*)(region == 0 ? e.q_norm : e.k_norm) + (size_t)layer * e.norm_layer_stride;
          x0 = x0 * inv * Elem<T>::to_f32(nw[ei]);
          x1 = x1 * inv * Elem<T>::to_f32(nw[ei + half]);
          const float cs = e.rope[(size_t)pos * half + ei];
          const float sn = e.rope[(size_t)e.rope_max_pos * half + (size_t)pos * half + ei];
          const float y0 = x0 * cs - x1 * sn, y1 = x1 * cs + x0 * sn;
          x0 = y0; x1 = y1;
        }
        if (region == 0) {
          T* q = (T*)e.out_act + (size_t)m * e.ldo + (size_t)head * hd;
          q[ei] = Elem<T>::from_f32(x0);
          q[ei + half] = Elem<T>::from_f32(x1);
        } else {
          const int page = e.page_table[(size_t)s * e.max_pages + pos / kPage];
          const int tok = pos % kPage;
          const size_t pbase = ((size_t)page * e.n_kv_heads + head) * (size_t)kPage * hd;
          if (region == 1) {   // K page layout [page][kv head][token][hd]
            T* k = (T*)e.kcache + (size_t)layer * e.cache_layer_stride + pbase + (size_t)tok * hd;
            k[ei] = Elem<T>::from_f32(x0);
            k[ei + half] = Elem<T>::from_f32(x1);
          } else {             // V page layout [page][kv head][hd][token]
            T* v = (T*)e.vcache + (size_t)layer * e.cache_layer_stride + pbase + tok;
            v[(size_t)ei * kPage] = Elem<T>::from_f32(x0);
            v[(size_t)(ei + half) * kPage] = Elem<T>::from_f32(x1);
          }
        }
      }
      break;
    }
  }
}

// ------------------------------------------------------------------ kernel

template <typename T, bool AF32, int MT, int NT, int WM, int WN, int U>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  constexpr int ROWS = WM * MT * 16, COLS = WN * NT * 16, LDT = COLS + 4;
  __shared__ float tile[ROWS][LDT];
  __shared__ int s_last;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / WN, wn = w % WN;
  const int bx = blockIdx.x, by = blockIdx.y, kz = blockIdx.z;
  const int m0 = by * ROWS, n0 = bx * COLS;
  const int KT = a.Kp / kTileK;
  const int kb = (int)((long long)KT * kz / a.ksplit);
  const int ke = (int)((long long)KT * (kz + 1) / a.ksplit);
  const int n_tiles_valid = a.e.N / kTileN;
  constexpr int AB = AF32 ? 4 : Elem<T>::kBytes;     // bytes per A element

  const T* bptr[NT];
  bool bval[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int ntg = (n0 + wn * NT * 16) / kTileN + nt;
    bval[nt] = ntg < n_tiles_valid;
    bptr[nt] = (const T*)a.B + ((size_t)(bval[nt] ? ntg : 0) * KT) * 512 + lane * 8;
  }
  const char* aptr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int row = m0 + wm * MT * 16 + mt * 16 + (lane % 16);
    if (row >= a.a_rows) row = a.a_rows - 1;
    aptr[mt] = (const char*)a.A + ((size_t)row * a.lda + (lane / 16) * 8) * AB;
  }

  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kt = kb; kt < ke; kt += U) {
    Frag<T> bf[U][NT];
    AFrag<T, AF32> af[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kt + u < ke) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          if (bval[nt]) bf[u][nt].load(bptr[nt] + (size_t)(kt + u) * 512);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) af[u][mt].load(aptr[mt] + (size_t)(kt + u) * kTileK * AB);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kt + u < ke) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            if (bval[nt]) af[u][mt].mma_into(acc[mt][nt], bf[u][nt]);
      }
    }
  }

  const int tile_id = by * gridDim.x + bx;
  if (a.ksplit == 1) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          tile[wm * MT * 16 + mt * 16 + 4 * (lane / 16) + i][wn * NT * 16 + nt * 16 + (lane % 16)] =
              acc[mt][nt][i];
    __syncthreads();
  } else {
    float* part = a.partial + ((size_t)tile_id * a.ksplit + kz) * (ROWS * COLS);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          part[(wm * MT * 16 + mt * 16 + 4 * (lane / 16) + i) * COLS + wn * NT * 16 + nt * 16 +
               (lane % 16)] = acc[mt][nt][i];
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
      const unsigned prev = __hip_atomic_fetch_add(&a.counters[tile_id], 1u, __ATOMIC_ACQ_REL,
                                                   __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (unsigned)(a.ksplit - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* base = a.partial + (size_t)tile_id * a.ksplit * (ROWS * COLS);
    for (int idx = threadIdx.x; idx < ROWS * COLS; idx += 256) {
      float sum = 0.f;
      for (int z = 0; z < a.ksplit; ++z)
        sum += __hip_atomic_load(base + (size_t)z * ROWS * COLS + idx, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      tile[idx / COLS][idx % COLS] = sum;
    }
    if (threadIdx.x == 0) a.counters[tile_id] = 0u;
    __syncthreads();
  }
  run_epilogue<T, ROWS, COLS, LDT>(a.e, tile, m0, n0);
}

int gemm_tile_cols(int) { return 128; }
int gemm_tile_rows(int shape) { return shape == SHAPE_SKINNY ? 16 : 128; }

template <typename T>
hipError_t gemm(const GemmArgs& a, int shape, bool a_f32, hipStream_t s) {
  const int rows = gemm_tile_rows(shape);
  dim3 grid((a.e.N + 127) / 128, (a.e.M + rows - 1) / rows, a.ksplit);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  if (shape == SHAPE_SKINNY) {
    if (a_f32) hipLaunchKernelGGL((gemm_kernel<T, true, 1, 2, 1, 4, 4>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<T, false, 1, 2, 1, 4, 8>), grid, dim3(256), 0, s, a);
  } else {
    if (a_f32) hipLaunchKernelGGL((gemm_kernel<T, true, 4, 4, 2, 2, 1>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((gemm_kernel<T, false, 4, 4, 2, 2, 2>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}
template hipError_t gemm<bf16_t>(const GemmArgs&, int, bool, hipStream_t);
template hipError_t gemm<float>(const GemmArgs&, int, bool, hipStream_t);

}  // namespace rt
