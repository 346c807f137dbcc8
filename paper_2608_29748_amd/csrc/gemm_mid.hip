// Weight-streaming bf16 MFMA GEMM for 33..512 rows (batched verify / draft blocks and
// prefill chunks): Y = X * W^T with the packed operands of gemm.h.
//
// A workgroup (4 waves) owns MB rows x NB columns of the output and one k slab.  Per
// 32-wide k tile it copies the MB/16 packed A fragments and NB/16 packed weight tiles
// (1 KiB each, already in MFMA lane order) straight from memory into a ring of LDS
// stages (16-byte direct-to-LDS loads, NSTAGE-1 k tiles in flight), so every weight
// byte is read from HBM once per workgroup and every A byte once per workgroup.  Waves
// split the tile 2 x 2: wave (wm, wn) accumulates MB/2 rows x NB/2 columns, reading its
// fragments from LDS at consecutive 16-byte lane offsets (conflict free).  The
// epilogue runs on the accumulators in registers.
#include "gemm.h"

namespace rt {

// Epilogue of one wave's accumulators: tile (m, n) covers rows rbase + 16 m + 0..3
// (this lane) and column cbase + 16 n + c16.
template <int KIND, int MT, int NT>
__device__ __forceinline__ void mid_store(const EpiArgs& e, const f32x4 (&acc)[MT][NT], int rbase, int cbase,
                                          int c16) {
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      const int ct = cbase + n * 16;   // first column of the 16-column tile
      const int col = ct + c16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + m * 16 + r;
        const float y = acc[m][n][r];
        if constexpr (KIND == EPI_SWIGLU) {
          // columns 0..7 of the tile are gate, 8..15 the matching up values
          const float u = __shfl_xor(y, 8, 64);
          if (c16 < 8 && row < e.M && ct < e.N) {
            const float act = y / (1.0f + expf(-y)) * u;
            ((bf16_t*)e.out_act)[pa_index(row, ct / 2 + c16, e.ldo)] = f32_to_bf16(act);
          }
        } else {
          if (row >= e.M || col >= e.N) continue;
          if constexpr (KIND == EPI_STORE_F32) {
            e.out_f32[(size_t)row * e.ldo + col] = y;
          } else if constexpr (KIND == EPI_STORE_ACT) {
            ((bf16_t*)e.out_act)[pa_index(row, col, e.ldo)] = f32_to_bf16(y);
          } else if constexpr (KIND == EPI_PARTIAL) {
            e.out_f32[(size_t)blockIdx.z * e.part_stride + (size_t)row * e.ldo + col] = y;
          } else {
            float* px = e.resid + (size_t)row * e.ldr + col;
            const float x = *px + y;
            *px = x;
            if (e.cap) ((bf16_t*)e.cap)[pa_index(row, e.cap_k0 + col, e.ldcap)] = f32_to_bf16(x);
          }
        }
      }
    }
}

// Argmax epilogue: for every row, the (value, lowest column) key over this wave's
// columns goes to part_keys[2 * blockIdx.x + wn][row] (reduced by argmax_reduce).
template <int MT, int NT>
__device__ __forceinline__ void mid_argmax(const EpiArgs& e, const f32x4 (&acc)[MT][NT], int rbase, int cbase,
                                           int c16, int part) {
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = rbase + m * 16 + r;
      uint64_t key = 0ull;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int col = cbase + n * 16 + c16;
        const float v = acc[m][n][r];
        if (col < e.N) {
          const uint64_t k = argmax_key(v, (uint32_t)col);
          key = k > key ? k : key;
          if (e.out_f32 && row < e.M) e.out_f32[(size_t)row * e.ldo + col] = v;
        }
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const uint64_t other = __shfl_xor(key, o, 64);
        key = other > key ? other : key;
      }
      if (c16 == 0 && row < e.M) e.part_keys[(size_t)part * e.M + row] = key;
    }
}

template <int MB, int NB, int NSTAGE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2))) void gemm_mid_kernel(GemmArgs a) {
  constexpr int MT = MB / 32;           // 16-row tiles per wave
  constexpr int NT = NB / 32;           // 16-column tiles per wave
  constexpr int AG = MB / 16;           // packed A groups per k tile (1 KiB each)
  constexpr int BT = NB / 16;           // packed weight tiles per k tile (1 KiB each)
  constexpr int LPW = (AG + BT) / 4;    // direct-to-LDS copies per wave per k tile
  constexpr int STG = (AG + BT) * 1024;
  static_assert((AG + BT) % 4 == 0, "copies must spread evenly over the four waves");
  __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STG];

  const int lane = threadIdx.x & 63, g4 = lane >> 4, c16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int m0 = blockIdx.y * MB, n0 = blockIdx.x * NB;
  const int KT = a.Kp / kTileK;
  const int kb = (int)((long)KT * blockIdx.z / gridDim.z), ke = (int)((long)KT * (blockIdx.z + 1) / gridDim.z);
  const int max_group = (a.a_rows - 1) >> 4;
  const int n_tiles_valid = a.e.N / kTileN;

  // copy j of this wave per k tile: item it = w + 4 j (A groups first, then weight
  // tiles); sources and destinations are uniform per wave
  auto item_src = [&](int j) -> const bf16_t* {
    const int it = w + 4 * j;
    if (it < AG) {
      int grp = (m0 >> 4) + it;
      if (grp > max_group) grp = max_group;
      return (const bf16_t*)a.A + (size_t)grp * a.lda;
    }
    int nt = (n0 >> 4) + (it - AG);
    if (nt >= n_tiles_valid) nt = n_tiles_valid - 1;
    return (const bf16_t*)a.B + (size_t)nt * KT * 512;
  };
  auto issue = [&](int kt, int stg) {
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(item_src(j) + (size_t)kt * 512 + lane * 8),
                                       (lds_void_t*)(smem + stg * STG + (w + 4 * j) * 1024), 16, 0, 0);
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < NSTAGE - 1; ++i)
    if (kb + i < ke) issue(kb + i, i);
  for (int kt = kb; kt < ke; ++kt) {
    const int i = kt - kb;
    // this wave's copies of k tile kt have landed once at most the later tiles' remain
    if constexpr (NSTAGE == 4) {
      if (kt + 2 < ke) wait_vm<2 * LPW>(); else if (kt + 1 < ke) wait_vm<LPW>(); else wait_vm<0>();
    } else if constexpr (NSTAGE == 3) {
      if (kt + 1 < ke) wait_vm<LPW>(); else wait_vm<0>();
    } else {
      wait_vm<0>();
    }
    lds_barrier();   // every wave's copies of tile kt are visible; tile kt-1's stage is free
    if (kt + NSTAGE - 1 < ke) issue(kt + NSTAGE - 1, (i + NSTAGE - 1) % NSTAGE);
    const char* st = smem + (i % NSTAGE) * STG;
    Frag<bf16_t> af[MT], bf[NT];
#pragma unroll
    for (int m = 0; m < MT; ++m) af[m].v = *reinterpret_cast<const bf16x8*>(st + (wm * MT + m) * 1024 + lane * 16);
#pragma unroll
    for (int n = 0; n < NT; ++n)
      bf[n].v = *reinterpret_cast<const bf16x8*>(st + (AG + wn * NT + n) * 1024 + lane * 16);
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < NT; ++n) mma(acc[m][n], af[m], bf[n]);
  }

  // epilogue from the accumulators: lane (g4, c16) of tile (m, n) holds rows
  // 4*g4 .. 4*g4+3 of column c16
  const EpiArgs& e = a.e;
  const int rbase = m0 + wm * MT * 16 + 4 * g4, cbase = n0 + wn * NT * 16;
  switch (e.kind) {
    case EPI_ARGMAX: mid_argmax<MT, NT>(e, acc, rbase, cbase, c16, 2 * blockIdx.x + wn); break;
    case EPI_SWIGLU: mid_store<EPI_SWIGLU, MT, NT>(e, acc, rbase, cbase, c16); break;
    case EPI_STORE_F32: mid_store<EPI_STORE_F32, MT, NT>(e, acc, rbase, cbase, c16); break;
    case EPI_STORE_ACT: mid_store<EPI_STORE_ACT, MT, NT>(e, acc, rbase, cbase, c16); break;
    case EPI_PARTIAL: mid_store<EPI_PARTIAL, MT, NT>(e, acc, rbase, cbase, c16); break;
    default: mid_store<EPI_RESID, MT, NT>(e, acc, rbase, cbase, c16);
  }
}

int gemm_mid_cols(int N) { return N / 128 >= 160 ? 128 : 64; }

bool gemm_mid_supports(const GemmArgs& a) {
  const int k = a.e.kind;
  return (k == EPI_STORE_F32 || k == EPI_STORE_ACT || k == EPI_RESID || k == EPI_SWIGLU || k == EPI_PARTIAL ||
          k == EPI_ARGMAX) &&
         a.e.M > 32 && a.e.M <= 512 && (a.e.kind == EPI_PARTIAL || a.ksplit == 1);
}

hipError_t gemm_mid(const GemmArgs& a, hipStream_t s) {
  if (!gemm_mid_supports(a)) return hipErrorInvalidValue;
  const int M = a.e.M, N = a.e.N;
  const int NB = gemm_mid_cols(N);
  const int MB = M <= 128 ? 128 : 256;
  dim3 grid((N + NB - 1) / NB, (M + MB - 1) / MB, a.ksplit);
  if (MB == 128 && NB == 64) RT_LAUNCH((gemm_mid_kernel<128, 64, 4>), grid, dim3(256), 0, s, a);
  else if (MB == 128) RT_LAUNCH((gemm_mid_kernel<128, 128, 4>), grid, dim3(256), 0, s, a);
  else if (NB == 64) RT_LAUNCH((gemm_mid_kernel<256, 64, 3>), grid, dim3(256), 0, s, a);
  else RT_LAUNCH((gemm_mid_kernel<256, 128, 3>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rt
