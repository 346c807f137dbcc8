// Packed-weight MFMA GEMM with split-K fixup and fused epilogues (see gemm.h).
#include "gemm.h"

namespace rt {

// ------------------------------------------------------------------ packing

// out tile (nt, kt), lane l, element e  <-  W[n = nt*16 + l%16][k = kt*32 + (l/16)*8 + e]
// (zero for k >= K).  With Wb set, output tile nt holds rows nt*8..nt*8+7 of Wa in its
// columns 0..7 and the same rows of Wb in columns 8..15 (gate | up pairs side by side).
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
    int n = nt * kTileN + (lane % 16);
    if (Wb) {
      const int c = lane % 16;
      src = c < 8 ? Wa : Wb;
      n = nt * 8 + (c % 8);
    }
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
  RT_LAUNCH(pack_kernel<T>, dim3(grid), dim3(256), 0, s, W, (const T*)nullptr, N, K, Kp, out);
}
template <typename T>
void pack_interleaved(const T* Wa, const T* Wb, int N, int K, int Kp, T* out, hipStream_t s) {
  size_t total = (size_t)2 * (N / kTileN) * (Kp / kTileK) * kWave;
  int grid = (int)((total + 255) / 256);
  if (grid > 65535 * 4) grid = 65535 * 4;
  RT_LAUNCH(pack_kernel<T>, dim3(grid), dim3(256), 0, s, Wa, Wb, N, K, Kp, out);
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

// Runs on a complete fp32 output tile t[ROWS][COLS] held in LDS (NTH threads).
template <typename T, int ROWS, int COLS, int LDT, int NTH>
__device__ void run_epilogue(const EpiArgs& e, float (*t)[LDT], int m0, int n0) {
  const int tid = threadIdx.x;
  if (e.kind == EPI_SWIGLU) {
    // per 16-column tile: columns 0..7 gate, 8..15 up, for 8 consecutive outputs
    constexpr int OC = COLS / 2;
    for (int idx = tid; idx < ROWS * OC; idx += NTH) {
      const int r = idx / OC, j = idx % OC;
      const int m = m0 + r;
      const int cg = (j / 8) * 16 + (j % 8);
      if (m >= e.M || n0 + cg >= e.N) continue;
      const float g = t[r][cg], u = t[r][cg + 8];
      const float act = g / (1.0f + expf(-g)) * u;
      ((T*)e.out_act)[pa_index(m, n0 / 2 + j, e.ldo)] = Elem<T>::from_f32(act);
    }
    return;
  }
  for (int idx = tid; idx < ROWS * COLS; idx += NTH) {
    const int r = idx / COLS, c = idx % COLS;
    const int m = m0 + r, n = n0 + c;
    if (m >= e.M || n >= e.N) continue;
    const float y = t[r][c];
    switch (e.kind) {
      case EPI_STORE_F32: e.out_f32[(size_t)m * e.ldo + n] = y; break;
      case EPI_STORE_ACT: ((T*)e.out_act)[pa_index(m, n, e.ldo)] = Elem<T>::from_f32(y); break;
      case EPI_RESID: {
        float* px = e.resid + (size_t)m * e.ldr + n;
        const float x = *px + y;
        *px = x;
        if (e.cap) ((T*)e.cap)[pa_index(m, e.cap_k0 + n, e.ldcap)] = Elem<T>::from_f32(x);
        break;
      }
      case EPI_COND_R:
        e.out_f32[pa_index(m, e.out_k0 + n, e.ldo)] = e.cond_m[pa_index(m, n, e.ld_cond_m)] + e.beta * y;
        break;
      case EPI_COND_GATE: e.out_f32[(size_t)m * e.ldo + n] = 1.0f / (1.0f + expf(-y)); break;
      case EPI_PARTIAL: e.out_f32[(size_t)blockIdx.z * e.part_stride + (size_t)m * e.ldo + n] = y; break;
      default: {  // EPI_COND_OUT
        const int s = m / e.rows_per_seq, j = m % e.rows_per_seq;
        const int tok = (j == 0) ? e.anchor[s * e.seq_stride] : e.mask_token;
        const float ev = Elem<T>::to_f32(((const T*)e.embed)[(size_t)tok * e.N + n]);
        const bool cond = (j >= 1) && (j <= e.cond_len[s * e.seq_stride]);
        const float x = cond ? ev + y * e.gate[(size_t)m * e.ld_gate + n] : ev;
        e.resid[(size_t)m * e.ldr + n] = x;
        e.etilde[(size_t)m * e.ldr + n] = x;
      }
    }
  }
}

// ------------------------------------------------------------------ split-slab epilogue
// One workgroup per 16 x 64 output tile: sums the k slabs in slab order into LDS, then
// runs the epilogue on the complete tile.
template <typename T>
__global__ __launch_bounds__(256) void split_epilogue_kernel(EpiArgs e, const float* __restrict__ part, int ks) {
  __shared__ float tile[16][65];
  const int m0 = blockIdx.y * 16, n0 = blockIdx.x * 64;
  const size_t slab = (size_t)e.M * e.N;
  for (int idx = threadIdx.x; idx < 16 * 64; idx += 256) {
    const int r = idx / 64, c = idx % 64;
    const int m = m0 + r, n = n0 + c;
    float sum = 0.f;
    if (m < e.M && n < e.N) {
      const float* p = part + (size_t)m * e.N + n;
      for (int z = 0; z < ks; ++z) sum += p[z * slab];
    }
    tile[r][c] = sum;
  }
  __syncthreads();
  run_epilogue<T, 16, 64, 65, 256>(e, tile, m0, n0);
}
template <typename T>
hipError_t gemm_split_epilogue(const EpiArgs& e, const float* part, int ks, hipStream_t s) {
  if (e.M <= 0 || e.N <= 0) return hipSuccess;
  if (e.kind == EPI_PARTIAL || e.kind == EPI_ARGMAX || ks < 1) return hipErrorInvalidValue;
  RT_LAUNCH((split_epilogue_kernel<T>), dim3((e.N + 63) / 64, (e.M + 15) / 16), dim3(256), 0, s, e, part, ks);
  return hipGetLastError();
}
template hipError_t gemm_split_epilogue<bf16_t>(const EpiArgs&, const float*, int, hipStream_t);
template hipError_t gemm_split_epilogue<float>(const EpiArgs&, const float*, int, hipStream_t);

// ------------------------------------------------------------------ skinny GEMM (M <= 32)
// Workgroup tile (MT*16) x (NT*16); its NW waves split the reduction into contiguous
// k ranges (each streams its own run of packed weight tiles) and the partial tiles are
// summed in wave order through LDS.

template <typename T, bool AF32, int MT, int NT, int NW, int U>
__global__ __launch_bounds__(NW * 64) void gemm16_kernel(GemmArgs a) {
  constexpr int ROWS = MT * 16, COLS = NT * 16, LDT = COLS + 1;
  constexpr int AB = AF32 ? 4 : Elem<T>::kBytes;
  __shared__ float red[NW][ROWS][COLS];
  __shared__ float tile[ROWS][LDT];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m0 = blockIdx.y * ROWS, n0 = blockIdx.x * COLS;
  const int KT = a.Kp / kTileK;
  // k slab blockIdx.z of gridDim.z, split again over the waves
  const int part = blockIdx.z * NW + w, parts = gridDim.z * NW;
  const int kb = KT * part / parts, ke = KT * (part + 1) / parts;
  const int n_tiles_valid = a.e.N / kTileN;
  const T* bptr[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int ntg = n0 / kTileN + nt;
    bptr[nt] = (const T*)a.B + ((size_t)(ntg < n_tiles_valid ? ntg : 0) * KT) * 512 + lane * 8;
  }
  const int max_group = (a.a_rows - 1) >> 4;
  const char* aptr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int grp = (m0 >> 4) + mt;
    if (grp > max_group) grp = max_group;
    aptr[mt] = (const char*)a.A + ((size_t)grp * a.lda + lane * 8) * AB;
  }
  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // groups of U k tiles; the last group's loads are clamped to ke-1 and its extra MFMAs
  // skipped, so the tail costs no additional round trip
  for (int kt = kb; kt < ke; kt += U) {
    Frag<T> bf[U][NT];
    AFrag<T, AF32> af[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kt + u < ke ? kt + u : ke - 1;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bf[u][nt].load_stream(bptr[nt] + (size_t)k * 512);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) af[u][mt].load(aptr[mt] + (size_t)k * 512 * AB);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep all U tiles' loads in flight before the MFMAs
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kt + u < ke) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) af[u][mt].mma_into(acc[mt][nt], bf[u][nt]);
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[w][mt * 16 + 4 * (lane / 16) + i][nt * 16 + (lane % 16)] = acc[mt][nt][i];
  __syncthreads();
  for (int idx = threadIdx.x; idx < ROWS * COLS; idx += NW * 64) {
    const int r = idx / COLS, c = idx % COLS;
    float sum = 0.f;
#pragma unroll
    for (int v = 0; v < NW; ++v) sum += red[v][r][c];
    tile[r][c] = sum;
  }
  __syncthreads();
  run_epilogue<T, ROWS, COLS, LDT, NW * 64>(a.e, tile, m0, n0);
}

// ------------------------------------------------------------------ k-slab partials, A in LDS
// Split reductions of at most 32 rows (bf16; the o and down projections of a round): grid
// (G, 1, slabs).  Workgroup (g, z) copies the A rows of k slab z into LDS once and computes
// the slab's partial tiles of column tiles g, g + G, g + 2G, ..: TP of them at a time, each
// by KW waves over consecutive k ranges of the slab, summed in wave order through LDS.  So
// A crosses from L2 into a compute unit once per slab instead of once per column tile.
template <int MT, int KTSMAX, int U>
__global__ __launch_bounds__(1024) void gemm16_slab_kernel(GemmArgs a, int tp_n, int kw_n) {
  constexpr int ROWS = MT * 16;
  __shared__ __attribute__((aligned(1024))) char sa[MT * KTSMAX * 1024];
  __shared__ float red[16][ROWS][16];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  const int KT = a.Kp / kTileK;
  const int z = blockIdx.z, S = gridDim.z;
  const int kb = KT * z / S, ke = KT * (z + 1) / S, kts = ke - kb;
  // the slab's A fragments (16-row group mt, k tile kb + j at sa + (mt * KTSMAX + j) KiB)
  const int max_group = (a.a_rows - 1) >> 4;
  for (int c = w; c < MT * kts; c += nw) {
    const int mt = c / kts, j = c % kts;
    const int grp = mt < max_group ? mt : max_group;
    const char* src = (const char*)a.A + ((size_t)grp * a.lda + (size_t)(kb + j) * 512) * 2 + lane * 16;
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_void_t*)(sa + (mt * KTSMAX + j) * 1024), 16, 0, 0);
  }
  const int tp = w / kw_n, kw = w % kw_n;
  const int n_tiles = (a.e.N + 15) / 16, n_valid = a.e.N / kTileN;
  const int k0 = kb + kts * kw / kw_n, k1 = kb + kts * (kw + 1) / kw_n;
  bool first = true;
  for (int base = blockIdx.x; base < n_tiles; base += gridDim.x * tp_n) {
    const int t = base + tp * gridDim.x;            // this wave's column tile
    f32x4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tp < tp_n && t < n_tiles && k0 < k1) {
      const bf16_t* bptr = (const bf16_t*)a.B + ((size_t)(t < n_valid ? t : 0) * KT) * 512 + lane * 8;
      for (int kt = k0; kt < k1; kt += U) {
        Frag<bf16_t> bf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) bf[u].load_stream(bptr + (size_t)(kt + u < k1 ? kt + u : k1 - 1) * 512);
        __builtin_amdgcn_sched_barrier(0);   // all U weight tiles in flight before the MFMAs
        if (first) {   // the A copies have landed once at most the U weight loads remain
          wait_vm<U>();
          lds_barrier();
          first = false;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (kt + u < k1) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              Frag<bf16_t> af;
              af.v = *reinterpret_cast<const bf16x8*>(sa + (mt * KTSMAX + kt + u - kb) * 1024 + lane * 16);
              mma(acc[mt], af, bf[u]);
            }
          }
      }
    }
    if (first) {       // waves without work still wait for the shared copies
      wait_vm<0>();
      lds_barrier();
      first = false;
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[w][mt * 16 + 4 * (lane / 16) + i][lane % 16] = acc[mt][i];
    __syncthreads();
    // tile group g2 sums its KW k ranges in order
    if (a.e.kind == EPI_SWIGLU) {
      // 8 gate and the matching 8 up columns per 16-column tile: out[m][n/2 + j]
      for (int idx = threadIdx.x; idx < tp_n * ROWS * 8; idx += blockDim.x) {
        const int g2 = idx / (ROWS * 8), r = idx / 8 % ROWS, j = idx % 8;
        const int tt = base + g2 * gridDim.x, m = r;
        if (tt >= n_tiles || m >= a.e.M || tt * 16 + j >= a.e.N) continue;
        float g = 0.f, u = 0.f;
        for (int v = 0; v < kw_n; ++v) {
          g += red[g2 * kw_n + v][r][j];
          u += red[g2 * kw_n + v][r][j + 8];
        }
        const float act = g / (1.0f + expf(-g)) * u;
        ((bf16_t*)a.e.out_act)[pa_index(m, tt * 8 + j, a.e.ldo)] = f32_to_bf16(act);
      }
    } else {
      for (int idx = threadIdx.x; idx < tp_n * ROWS * 16; idx += blockDim.x) {
        const int g2 = idx / (ROWS * 16), r = idx / 16 % ROWS, c = idx % 16;
        const int tt = base + g2 * gridDim.x, m = r, n = tt * 16 + c;
        if (tt >= n_tiles || m >= a.e.M || n >= a.e.N) continue;
        float sum = 0.f;
        for (int v = 0; v < kw_n; ++v) sum += red[g2 * kw_n + v][r][c];
        a.e.out_f32[(size_t)z * a.e.part_stride + (size_t)m * a.e.ldo + n] = sum;
      }
    }
    __syncthreads();
  }
  if (first) wait_vm<0>();   // no tile at all: leave no copy in flight
}

// Launch parameters of gemm16_slab_kernel for M rows, N columns and a padded K with `slabs`
// k slabs: workgroups per slab (so that about 256 run), column tiles in flight per
// workgroup and waves per tile (16 at most in all); false if the slab's A rows do not fit.
struct SlabPlan { int G, tp, kw, kpw; };
static bool slab_plan(int M, int N, int Kp, int slabs, SlabPlan* sp) {
  const int MT = M > 16 ? 2 : 1, KT = Kp / kTileK, n_tiles = (N + 15) / 16;
  const int kts = (KT + slabs - 1) / slabs;
  if (M > 32 || kts > (MT == 1 ? 80 : 48) || slabs < 1 || KT < slabs) return false;
  int G = 256 / slabs;
  if (G > n_tiles) G = n_tiles;
  if (G < 1) G = 1;
  const int per = (n_tiles + G - 1) / G;          // column tiles of the busiest workgroup
  // one column tile per workgroup reuses nothing: the plain kernels are faster there
  // (Qwen3-0.6B shape o / down: 3.0 / 3.5 us against 4.4 / 4.7 us on this kernel)
  if (per < 2) return false;
  int tp = per < 16 ? per : 16;
  int kw = 16 / tp;                                 // waves per tile: enough for ~8 k tiles each
  const int want = (kts + 7) / 8;
  if (kw > want) kw = want;
  if (kw < 1) kw = 1;
  sp->G = G; sp->tp = tp; sp->kw = kw;
  sp->kpw = (kts + kw - 1) / kw;
  return true;
}
// Weight tiles in flight per wave: batches of 8 up to 16 k tiles per wave, else of 14
// (measured at the Qwen3-4B shape: down, 16 tiles per wave, 11.8 us with two batches of
// 8 against 12.6 with one of 16; gate|up, 27 tiles, 19.4 us with 14 against 19.9 with 8)
static void slab_launch(const GemmArgs& a, const SlabPlan& sp, int M, int slabs, hipStream_t s) {
  const dim3 g3(sp.G, 1, slabs), blk(64 * sp.tp * sp.kw);
  if (M > 16) RT_LAUNCH((gemm16_slab_kernel<2, 48, 8>), g3, blk, 0, s, a, sp.tp, sp.kw);
  else if (sp.kpw <= 16) RT_LAUNCH((gemm16_slab_kernel<1, 80, 8>), g3, blk, 0, s, a, sp.tp, sp.kw);
  else RT_LAUNCH((gemm16_slab_kernel<1, 80, 14>), g3, blk, 0, s, a, sp.tp, sp.kw);
}

// ------------------------------------------------------------------ wide GEMM (large M)

template <typename T, bool AF32, int MT, int NT, int WM, int WN, int U>
__global__ __launch_bounds__(256) void gemm_wide_kernel(GemmArgs a) {
  constexpr int ROWS = WM * MT * 16, COLS = WN * NT * 16, LDT = COLS + 4;
  __shared__ float tile[ROWS][LDT];
  __shared__ int s_last;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w / WN, wn = w % WN;
  const int bx = blockIdx.x, by = blockIdx.y, kz = blockIdx.z;
  const int m0 = by * ROWS, n0 = bx * COLS;
  const int KT = a.Kp / kTileK;
  const int kb = (int)((long long)KT * kz / a.ksplit);
  const int ke = (int)((long long)KT * (kz + 1) / a.ksplit);
  const int n_tiles_valid = a.e.N / kTileN;
  constexpr int AB = AF32 ? 4 : Elem<T>::kBytes;
  const T* bptr[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int ntg = (n0 + wn * NT * 16) / kTileN + nt;
    bptr[nt] = (const T*)a.B + ((size_t)(ntg < n_tiles_valid ? ntg : 0) * KT) * 512 + lane * 8;
  }
  const int max_group = (a.a_rows - 1) >> 4;
  const char* aptr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int grp = ((m0 + wm * MT * 16) >> 4) + mt;
    if (grp > max_group) grp = max_group;
    aptr[mt] = (const char*)a.A + ((size_t)grp * a.lda + lane * 8) * AB;
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
      const int k = kt + u < ke ? kt + u : ke - 1;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bf[u][nt].load(bptr[nt] + (size_t)k * 512);   // re-read by every row tile
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) af[u][mt].load(aptr[mt] + (size_t)k * 512 * AB);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kt + u < ke) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) af[u][mt].mma_into(acc[mt][nt], bf[u][nt]);
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
    // split k: fp32 partial tiles; the last workgroup of a tile sums them in split order
    float* part = a.partial + ((size_t)tile_id * a.ksplit + kz) * (ROWS * COLS);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          part[(wm * MT * 16 + mt * 16 + 4 * (lane / 16) + i) * COLS + wn * NT * 16 + nt * 16 + (lane % 16)] =
              acc[mt][nt][i];
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
      const unsigned prev = __hip_atomic_fetch_add(&a.counters[tile_id], 1u, __ATOMIC_ACQ_REL,
                                                   __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (unsigned)(a.ksplit - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();   // acquire: every split's partial tile is visible
    constexpr int PER = ROWS * COLS / 256;
    float sum[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) sum[i] = 0.f;
    const float* base = a.partial + (size_t)tile_id * a.ksplit * (ROWS * COLS);
    for (int z = 0; z < a.ksplit; ++z) {
      const float* pz = base + (size_t)z * ROWS * COLS + threadIdx.x;
#pragma unroll
      for (int i = 0; i < PER; ++i) sum[i] += pz[i * 256];
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = threadIdx.x + i * 256;
      tile[idx / COLS][idx % COLS] = sum[i];
    }
    if (threadIdx.x == 0) a.counters[tile_id] = 0u;
    __syncthreads();
  }
  run_epilogue<T, ROWS, COLS, LDT, 256>(a.e, tile, m0, n0);
}

template <typename T>
hipError_t gemm(const GemmArgs& a, int shape, bool a_f32, hipStream_t s) {
  const int M = a.e.M, N = a.e.N;
  if (M <= 0 || N <= 0) return hipSuccess;
  if (shape == SHAPE_SKINNY) {
    if (M > 32) {
      // 33..64 rows (bf16 operands): 64-row tiles, eight waves over k, two k tiles in
      // flight per wave; 32 columns, or 64 per k slab of a split reduction
      if constexpr (sizeof(T) != 2) return hipErrorInvalidValue;
      if (M > 64 || a_f32) return hipErrorInvalidValue;
      if ((a.e.kind == EPI_PARTIAL) != (a.ksplit > 1) || a.ksplit < 1) return hipErrorInvalidValue;
      if (a.ksplit > 1) RT_LAUNCH((gemm16_kernel<T, false, 4, 4, 8, 2>), dim3((N + 63) / 64, 1, a.ksplit), dim3(512), 0, s, a);
      else RT_LAUNCH((gemm16_kernel<T, false, 4, 2, 8, 2>), dim3((N + 31) / 32, 1, 1), dim3(512), 0, s, a);
      return hipGetLastError();
    }
    // tile width, waves and loads in flight per shape class (measured on the Qwen3 layer
    // shapes): split reductions (bf16) on the slab kernel, A staged once per slab and
    // workgroup; N >= 16384 (gate|up, SwiGLU) on the slab kernel with one slab (4B shape
    // 20.3 -> 19.4 us; the 16-column kernel with 2 waves x 8 loads at 32 rows); N >= 5120
    // 32 columns (two loads in flight per wave at 16 rows: 5% faster than four at the 4B
    // q|k|v); otherwise 16 columns with 8 loads in flight
    if ((a.e.kind == EPI_PARTIAL) != (a.ksplit > 1) || a.ksplit < 1) return hipErrorInvalidValue;
    dim3 grid((N + 15) / 16, 1, a.ksplit);
    if (a_f32) {
      if (M > 16) RT_LAUNCH((gemm16_kernel<T, true, 2, 1, 4, 8>), grid, dim3(256), 0, s, a);
      else RT_LAUNCH((gemm16_kernel<T, true, 1, 1, 4, 8>), grid, dim3(256), 0, s, a);
    } else if (a.ksplit > 1) {
      SlabPlan sp;
      if (sizeof(T) == 2 && slab_plan(M, N, a.Kp, a.ksplit, &sp)) {
        // A rows of each slab staged once per workgroup
        slab_launch(a, sp, M, a.ksplit, s);
      } else if (M > 16) {
        RT_LAUNCH((gemm16_kernel<T, false, 2, 1, 4, 4>), grid, dim3(256), 0, s, a);
      } else {
        RT_LAUNCH((gemm16_kernel<T, false, 1, 1, 4, 4>), grid, dim3(256), 0, s, a);
      }
    } else if (N >= 16384) {
      SlabPlan sp;
      if (sizeof(T) == 2 && a.e.kind == EPI_SWIGLU && slab_plan(M, N, a.Kp, 1, &sp)) {
        slab_launch(a, sp, M, 1, s);
      }
      else if (M > 16) RT_LAUNCH((gemm16_kernel<T, false, 2, 1, 8, 4>), grid, dim3(512), 0, s, a);
      else RT_LAUNCH((gemm16_kernel<T, false, 1, 1, 2, 8>), grid, dim3(128), 0, s, a);
    } else if (N >= 5120) {
      dim3 g2((N + 31) / 32, 1, 1);
      if (M > 16) RT_LAUNCH((gemm16_kernel<T, false, 2, 2, 8, 4>), g2, dim3(512), 0, s, a);
      else RT_LAUNCH((gemm16_kernel<T, false, 1, 2, 8, 2>), g2, dim3(512), 0, s, a);
    } else {
      if (M > 16) RT_LAUNCH((gemm16_kernel<T, false, 2, 1, 8, 8>), grid, dim3(512), 0, s, a);
      else RT_LAUNCH((gemm16_kernel<T, false, 1, 1, 8, 8>), grid, dim3(512), 0, s, a);
    }
  } else {
    if constexpr (sizeof(T) == 2) {
      if (gemm_mid_supports(a)) return gemm_mid(a, a_f32, s);
    }
    if (a.e.kind == EPI_PARTIAL) return hipErrorInvalidValue;
    dim3 grid((N + 127) / 128, (M + 127) / 128, a.ksplit);
    if (a_f32) RT_LAUNCH((gemm_wide_kernel<T, true, 4, 4, 2, 2, 1>), grid, dim3(256), 0, s, a);
    else RT_LAUNCH((gemm_wide_kernel<T, false, 4, 4, 2, 2, 2>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}
template hipError_t gemm<bf16_t>(const GemmArgs&, int, bool, hipStream_t);
template hipError_t gemm<float>(const GemmArgs&, int, bool, hipStream_t);

// ------------------------------------------------------------------ q/k/v post-processing

template <typename T>
__global__ __launch_bounds__(256) void qkv_post_kernel(QkvPostArgs a) {
  const int lane = threadIdx.x & 63;
  const int hd = a.head_dim, half = hd / 2;
  const int heads_per_layer = a.layer_cols / hd;
  const int heads = heads_per_layer * a.n_layers;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= a.M * heads) return;
  const int m = item / heads, hid = item % heads;
  const int layer = hid / heads_per_layer, hin = hid % heads_per_layer;
  const int s = m / a.rows_per_seq, i = m % a.rows_per_seq;
  if (a.nrows && i >= a.nrows[s * a.seq_stride]) return;
  const int pos = a.pos0[s * a.seq_stride] + i;
  const int qh = a.q_cols / hd, kvh = a.kv_cols / hd;
  const int region = hin < qh ? 0 : (hin < qh + kvh ? 1 : 2);
  const int head = region == 0 ? hin : (region == 1 ? hin - qh : hin - qh - kvh);
  if (lane >= half) return;
  const float* src = a.src + (size_t)m * a.lds + (size_t)layer * a.layer_cols + (size_t)hin * hd;
  float x0, x1;
  if (a.n_part > 1) {   // k-slab partials, added in slab order
    x0 = 0.f;
    x1 = 0.f;
    for (int z = 0; z < a.n_part; ++z) {
      x0 += src[(size_t)z * a.part_stride + lane];
      x1 += src[(size_t)z * a.part_stride + lane + half];
    }
  } else {
    x0 = src[lane];
    x1 = src[lane + half];
  }
  if (region < 2) {
    float ss = qk_sq(x0, x1);
    for (int o = half / 2; o > 0; o >>= 1) ss = ss + __shfl_xor(ss, o, 64);
    const float inv = qk_inv(ss, hd, a.eps);
    const T* nw = (const T*)(region == 0 ? a.q_norm : a.k_norm) + (size_t)layer * a.norm_layer_stride;
    const float cs = a.rope[(size_t)pos * half + lane];
    const float sn = a.rope[(size_t)a.rope_max_pos * half + (size_t)pos * half + lane];
    qk_norm_rope(x0, x1, inv, Elem<T>::to_f32(nw[lane]), Elem<T>::to_f32(nw[lane + half]), cs, sn);
  }
  if (region == 0) {
    T* q = (T*)a.q_out + (size_t)m * a.ldq + (size_t)head * hd;
    q[lane] = Elem<T>::from_f32(x0);
    q[lane + half] = Elem<T>::from_f32(x1);
    return;
  }
  const int page = a.page_table[(size_t)s * a.max_pages + pos / kPage];
  const int tok = pos % kPage;
  const size_t pbase = (size_t)layer * a.cache_layer_stride + ((size_t)page * a.n_kv_heads + head) * (size_t)kPage * hd;
  if (region == 1) {   // K page layout [page][kv head][token][hd]
    T* k = (T*)a.kcache + pbase + (size_t)tok * hd;
    k[lane] = Elem<T>::from_f32(x0);
    k[lane + half] = Elem<T>::from_f32(x1);
  } else {             // V page layout [page][kv head][hd][token]
    T* v = (T*)a.vcache + pbase + tok;
    v[(size_t)lane * kPage] = Elem<T>::from_f32(x0);
    v[(size_t)(lane + half) * kPage] = Elem<T>::from_f32(x1);
  }
}

template <typename T>
hipError_t qkv_post(const QkvPostArgs& a, hipStream_t s) {
  const int heads = (a.layer_cols / a.head_dim) * a.n_layers;
  const long long items = (long long)a.M * heads;
  if (items <= 0) return hipSuccess;
  RT_LAUNCH(qkv_post_kernel<T>, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}
template hipError_t qkv_post<bf16_t>(const QkvPostArgs&, hipStream_t);
template hipError_t qkv_post<float>(const QkvPostArgs&, hipStream_t);

// ------------------------------------------------------------------ LM head + argmax

constexpr int kLmTilesPerWave = 2;
int lmhead_grid(int N) {
  const int tiles = (N + 31) / 32;
  return (tiles + 4 * kLmTilesPerWave - 1) / (4 * kLmTilesPerWave);
}

// Each wave owns 32-column tiles (two 16-column MFMA tiles) over the full reduction and
// keeps, per row, the best (value, index) key seen; the workgroup's four waves then
// combine their keys through LDS.
template <typename T, int MT, int U>
__global__ __launch_bounds__(256) void lmhead_kernel(LmHeadArgs a) {
  constexpr int ROWS = MT * 16;
  __shared__ uint64_t wkeys[4][ROWS];
  const int lane = threadIdx.x & 63, g4 = lane / 16, c16 = lane % 16;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KT = a.Kp / kTileK;
  const int n_tiles16 = a.N / kTileN;
  const int max_group = (a.a_rows - 1) >> 4;
  const T* aptr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) aptr[mt] = (const T*)a.A + (size_t)(mt < max_group ? mt : max_group) * a.lda + lane * 8;
  uint64_t best[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) best[mt][i] = 0ull;
  const int tiles32 = (a.N + 31) / 32;
  for (int t = blockIdx.x * 4 + w; t < tiles32; t += gridDim.x * 4) {
    const T* bptr[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int ntg = t * 2 + nt;
      bptr[nt] = (const T*)a.B + ((size_t)(ntg < n_tiles16 ? ntg : 0) * KT) * 512 + lane * 8;
    }
    f32x4 acc[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt][0] = acc[mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    int kt = 0;
    for (; kt + U <= KT; kt += U) {
      Frag<T> bf[U][2];
      Frag<T> af[U][MT];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        bf[u][0].load_stream(bptr[0] + (size_t)(kt + u) * 512);
        bf[u][1].load_stream(bptr[1] + (size_t)(kt + u) * 512);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) af[u][mt].load(aptr[mt] + (size_t)(kt + u) * 512);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          mma(acc[mt][0], af[u][mt], bf[u][0]);
          mma(acc[mt][1], af[u][mt], bf[u][1]);
        }
    }
    for (; kt < KT; ++kt) {
      Frag<T> b0, b1, af[MT];
      b0.load_stream(bptr[0] + (size_t)kt * 512);
      b1.load_stream(bptr[1] + (size_t)kt * 512);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) af[mt].load(aptr[mt] + (size_t)kt * 512);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        mma(acc[mt][0], af[mt], b0);
        mma(acc[mt][1], af[mt], b1);
      }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mt * 16 + 4 * g4 + i;
        uint64_t k = 0ull;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int n = t * 32 + nt * 16 + c16;
          if (n < a.N) {
            const float y = acc[mt][nt][i];
            if (a.logits && row < a.M) a.logits[(size_t)row * a.ldl + n] = y;
            const uint64_t kk = argmax_key(y, (uint32_t)n);
            k = kk > k ? kk : k;
          }
        }
        best[mt][i] = k > best[mt][i] ? k : best[mt][i];
      }
  }
  // reduce over the 16 lanes holding the same rows, then over the four waves
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint64_t k = best[mt][i];
      for (int o = 8; o > 0; o >>= 1) {
        const uint64_t other = __shfl_xor(k, o, 64);
        k = other > k ? other : k;
      }
      if (c16 == 0) wkeys[w][mt * 16 + 4 * g4 + i] = k;
    }
  __syncthreads();
  if (threadIdx.x < ROWS && (int)threadIdx.x < a.M) {
    uint64_t k = wkeys[0][threadIdx.x];
#pragma unroll
    for (int v = 1; v < 4; ++v) k = wkeys[v][threadIdx.x] > k ? wkeys[v][threadIdx.x] : k;
    a.part_keys[(size_t)blockIdx.x * a.M + threadIdx.x] = k;
  }
}

// LM head for at most 16 rows of bf16 activations with K <= 4096: the workgroup copies
// the 16 x K activation block into LDS once (direct-to-LDS, 1 KiB per k tile) and its
// eight waves then stream 16-column weight tiles over the vocabulary (grid stride),
// taking A fragments from LDS.  The activations are read from L2 once per workgroup
// instead of once per column tile, which leaves the L1 miss path to the weight stream.
constexpr int kLmWaves = 8;

static bool lm_lds_ok(int M, int Kp, int elem_bytes) { return elem_bytes == 2 && M <= 16 && Kp <= 4096; }

template <int KTMAX, int U>
__global__ __launch_bounds__(kLmWaves * 64) void lmhead_lds_kernel(LmHeadArgs a) {
  static_assert(KTMAX * 1024 >= kLmWaves * 16 * 8, "the keys reuse the activation buffer");
  __shared__ __attribute__((aligned(1024))) char sa[KTMAX * 1024];
  const int lane = threadIdx.x & 63, g4 = lane / 16, c16 = lane % 16;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KT = a.Kp / kTileK;
  const int n_tiles = a.N / kTileN;
  for (int t = w; t < KT; t += kLmWaves)
    __builtin_amdgcn_global_load_lds((const void*)((const char*)a.A + (size_t)t * 1024 + lane * 16),
                                     (lds_void_t*)(sa + t * 1024), 16, 0, 0);
  wait_vm<0>();
  lds_barrier();
  uint64_t best[4] = {0ull, 0ull, 0ull, 0ull};
  for (int t = blockIdx.x * kLmWaves + w; t < n_tiles; t += gridDim.x * kLmWaves) {
    const bf16_t* bptr = (const bf16_t*)a.B + ((size_t)t * KT) * 512 + lane * 8;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int kt = 0; kt < KT; kt += U) {
      Frag<bf16_t> bf[U];
#pragma unroll
      for (int u = 0; u < U; ++u) bf[u].load_stream(bptr + (size_t)(kt + u < KT ? kt + u : KT - 1) * 512);
      __builtin_amdgcn_sched_barrier(0);   // all U weight tiles in flight before the MFMAs
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (kt + u < KT) {
          Frag<bf16_t> af;
          af.v = *reinterpret_cast<const bf16x8*>(sa + (kt + u) * 1024 + lane * 16);
          mma(acc, af, bf[u]);
        }
    }
    // lane (g4, c16) holds rows 4 g4 .. 4 g4 + 3 of column t * 16 + c16
    const int n = t * kTileN + c16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * g4 + i;
      if (a.logits && row < a.M) a.logits[(size_t)row * a.ldl + n] = acc[i];
      const uint64_t kk = argmax_key(acc[i], (uint32_t)n);
      best[i] = kk > best[i] ? kk : best[i];
    }
  }
  __syncthreads();   // every wave is done with the activations: the keys take their place
  uint64_t* wkeys = reinterpret_cast<uint64_t*>(sa);   // [kLmWaves][16]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint64_t k = best[i];
    for (int o = 8; o > 0; o >>= 1) {
      const uint64_t other = __shfl_xor(k, o, 64);
      k = other > k ? other : k;
    }
    if (c16 == 0) wkeys[w * 16 + 4 * g4 + i] = k;
  }
  __syncthreads();
  if (threadIdx.x < 16 && (int)threadIdx.x < a.M) {
    uint64_t k = wkeys[threadIdx.x];
#pragma unroll
    for (int v = 1; v < kLmWaves; ++v) k = wkeys[v * 16 + threadIdx.x] > k ? wkeys[v * 16 + threadIdx.x] : k;
    a.part_keys[(size_t)blockIdx.x * a.M + threadIdx.x] = k;
  }
}

int lmhead_parts(int M, int N, int Kp, int elem_bytes) {
  if (!lm_lds_ok(M, Kp, elem_bytes)) return lmhead_grid(N);
  const int grid = Kp / kTileK <= 80 ? kLmGrid : kLmGrid / 2;   // 80 KiB: two per CU; 128 KiB: one
  const int need = (N / kTileN + kLmWaves - 1) / kLmWaves;
  return grid < need ? grid : need;
}
int lmhead_max_parts(int N) { return lmhead_grid(N) > kLmGrid ? lmhead_grid(N) : kLmGrid; }

template <typename T>
hipError_t lm_head(const LmHeadArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.M > 32) return hipErrorInvalidValue;
  if (lm_lds_ok(a.M, a.Kp, (int)sizeof(T))) {
    const dim3 grid(lmhead_parts(a.M, a.N, a.Kp, (int)sizeof(T)));
    if (a.Kp / kTileK <= 80) RT_LAUNCH((lmhead_lds_kernel<80, 8>), grid, dim3(kLmWaves * 64), 0, s, a);
    else RT_LAUNCH((lmhead_lds_kernel<128, 8>), grid, dim3(kLmWaves * 64), 0, s, a);
    return hipGetLastError();
  }
  dim3 grid(lmhead_grid(a.N));
  if (a.M > 16) RT_LAUNCH((lmhead_kernel<T, 2, 8>), grid, dim3(256), 0, s, a);
  else RT_LAUNCH((lmhead_kernel<T, 1, 8>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}
template hipError_t lm_head<bf16_t>(const LmHeadArgs&, hipStream_t);
template hipError_t lm_head<float>(const LmHeadArgs&, hipStream_t);

__global__ __launch_bounds__(256) void argmax_reduce_kernel(const uint64_t* __restrict__ part, int nparts, int M,
                                                            uint64_t* keys) {
  __shared__ uint64_t red[4];
  const int row = blockIdx.x;
  uint64_t k = 0ull;
  for (int j = threadIdx.x; j < nparts; j += 256) {
    const uint64_t v = part[(size_t)j * M + row];
    k = v > k ? v : k;
  }
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t other = __shfl_xor(k, o, 64);
    k = other > k ? other : k;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = k;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t b = red[0];
    for (int v = 1; v < 4; ++v) b = red[v] > b ? red[v] : b;
    keys[row] = b;
  }
}
hipError_t argmax_reduce(const uint64_t* part_keys, int nparts, int M, uint64_t* keys, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  RT_LAUNCH(argmax_reduce_kernel, dim3(M), dim3(256), 0, s, part_keys, nparts, M, keys);
  return hipGetLastError();
}

}  // namespace rt
