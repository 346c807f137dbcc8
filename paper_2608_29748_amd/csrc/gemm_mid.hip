// Weight-streaming bf16 MFMA GEMM for 33..512 rows (batched verify / draft blocks and
// prefill chunks): Y = X * W^T with the packed operands of gemm.h.
//
// A workgroup (4, 8 or 16 waves) owns MB rows x NB columns of the output and one k slab.  Per
// 32-wide k tile it copies the MB/16 packed A fragments and NB/16 packed weight tiles
// (1 KiB each, already in MFMA lane order) straight from memory into a ring of LDS
// stages (16-byte direct-to-LDS loads, NSTAGE-1 k tiles in flight), so every weight
// byte is read from HBM once per workgroup and every A byte once per workgroup.  Waves
// split the tile (NW/2) x 2: wave (wm, wn) accumulates MB/(NW/2) rows x NB/2 columns,
// reading its fragments from LDS at consecutive 16-byte lane offsets (conflict free); with
// DB the fragments of k tile kt+1 are read while the MFMAs of tile kt run (a register
// double buffer, one k tile of the ring less in flight).  The epilogue runs on the
// accumulators in registers.
//
// An fp32 A operand (AF32) is copied as 2 KiB fragments and split in registers into a
// bf16 high part and a bf16 remainder, each multiplied by the weight tile (two MFMAs),
// as in the other GEMM kernels.  When the output tiles alone would leave the chip
// underfilled, or the epilogue is one the register epilogue does not cover, the k range
// is split over grid z into fp32 slabs that a second kernel sums in slab order before
// running the epilogue.
#include "gemm.h"

#include <type_traits>

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

// Wait until at most min(N, r) k tiles of LPW copies each are still in flight.
template <int N, int LPW>
__device__ __forceinline__ void wait_tiles(int r) {
  if constexpr (N <= 0) {
    wait_vm<0>();
  } else {
    if (r >= N) wait_vm<N * LPW>();
    else wait_tiles<N - 1, LPW>(r);
  }
}

template <int MB, int NB, int NSTAGE, bool AF32, int NW, bool DB = false, bool NTB = false>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(1, 2))) void gemm_mid_kernel(GemmArgs a) {
  constexpr int WM = NW / 2;            // wave rows (two wave columns)
  constexpr int MT = MB / (16 * WM);    // 16-row tiles per wave
  constexpr int NT = NB / 32;           // 16-column tiles per wave
  constexpr int AG = MB / 16;           // packed A groups per k tile
  constexpr int AB = AF32 ? 2048 : 1024;   // bytes of one A group's k tile
  constexpr int AI = AG * AB / 1024;    // A copy items (1 KiB) per k tile
  constexpr int BT = NB / 16;           // packed weight tiles per k tile (1 KiB each)
  constexpr int IT = AI + BT;           // copy items per k tile
  constexpr int LPW = (IT + NW - 1) / NW;   // direct-to-LDS copies per wave per k tile
  constexpr int STG = IT * 1024;
  static_assert(NW % 2 == 0 && MT >= 1 && MB % (16 * WM) == 0, "wave grid");
  __shared__ __attribute__((aligned(1024))) char smem[NSTAGE * STG];

  const int lane = threadIdx.x & 63, g4 = lane >> 4, c16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int m0 = blockIdx.y * MB, n0 = blockIdx.x * NB;
  const int KT = a.Kp / kTileK;
  const int kb = (int)((long)KT * blockIdx.z / gridDim.z), ke = (int)((long)KT * (blockIdx.z + 1) / gridDim.z);
  const int max_group = (a.a_rows - 1) >> 4;
  const int n_tiles_valid = a.e.N / kTileN;

  // copy j of this wave per k tile: item it = w + NW j (A items first, then weight
  // tiles; items past the last repeat item 0, the same bytes to the same slot, so that
  // every wave issues LPW copies); sources and destinations are uniform per wave
  constexpr size_t AE = AF32 ? 4 : 2;   // bytes per A element
  auto item_of = [&](int j) { const int it = w + NW * j; return it < IT ? it : 0; };
  auto item_src = [&](int j, int kt) -> const char* {
    const int it = item_of(j);
    if (it < AI) {
      int grp = (m0 >> 4) + it * 1024 / AB;
      if (grp > max_group) grp = max_group;
      return (const char*)a.A + (size_t)grp * a.lda * AE + (size_t)kt * AB + (it * 1024) % AB;
    }
    int nt = (n0 >> 4) + (it - AI);
    if (nt >= n_tiles_valid) nt = n_tiles_valid - 1;
    return (const char*)a.B + ((size_t)nt * KT + kt) * 1024;
  };
  // With one row tile every weight tile is read by one workgroup: non-temporal copies.
  // The A fragments, which every workgroup reads, and weights that several row tiles
  // read stay cached.
  const bool stream_b = gridDim.y == 1;
  auto issue = [&](int kt, int stg) {
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const void* src = item_src(j, kt) + lane * 16;
      lds_void_t* dst = (lds_void_t*)(smem + stg * STG + item_of(j) * 1024);
      if (item_of(j) >= AI && stream_b) __builtin_amdgcn_global_load_lds(src, dst, 16, 0, RT_NT_AUX);
      else __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
    }
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < NSTAGE - 1; ++i)
    if (kb + i < ke) issue(kb + i, i);
  if constexpr (DB) {
    static_assert(!AF32 && NSTAGE >= 3, "fragment double buffer: bf16 operands");
    // The fragments of tile kt+1 are read from LDS while the MFMAs of tile kt run.  Step
    // kt: wait for this wave's copies of tile kt+1 (the later tiles' stay in flight) and
    // for its own LDS reads, barrier (all copies of kt+1 visible, every wave done reading
    // tile kt-1, whose stage the step's copies then refill), read tile kt+1's fragments,
    // multiply tile kt's.  The last step reads a stale stage into registers nobody uses, so
    // that every step has one shape and the compiler's wait before the MFMAs covers only
    // the previous step's reads.
    //
    // Per step the scalar work is kept small: every copy's source advances by one 1 KiB k
    // tile per step from a pointer set up once, and the stages to fill and to read are
    // byte offsets that advance by one stage with a wrap (no products or divisions).
    auto read = [&](int off, Frag<bf16_t>(&af)[MT], Frag<bf16_t>(&bf)[NT]) {
      const char* st = smem + off;
#pragma unroll
      for (int m = 0; m < MT; ++m) af[m].v = *reinterpret_cast<const bf16x8*>(st + (wm * MT + m) * 1024 + lane * 16);
#pragma unroll
      for (int n = 0; n < NT; ++n) bf[n].v = *reinterpret_cast<const bf16x8*>(st + (AI + wn * NT + n) * 1024 + lane * 16);
    };
    // (NTB: the weight copies are non-temporal, chosen by the launch: one row tile)
    const char* csrc[LPW];   // this wave's copy j of the next tile to issue (kb + NSTAGE - 1)
    int cdst[LPW];
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      csrc[j] = item_src(j, kb) + (size_t)(NSTAGE - 1) * 1024 + lane * 16;
      cdst[j] = item_of(j) * 1024;
    }
    // copies j < AI / NW of every wave are A items, the later ones weight tiles, except
    // past the last item, where a wave repeats A item 0 (kept cached)
    static_assert(!NTB || AI % NW == 0, "non-temporal copies: A items fill whole rounds of the waves");
    const bool last_is_b = w + NW * (LPW - 1) < IT;
    constexpr int RING = NSTAGE * STG;
    int off_is = (NSTAGE - 1) * STG, off_rd = STG;   // step 0 fills stage NSTAGE-1 and reads stage 1
    // STEADY: the step and the next both issue a tile, so NSTAGE - 3 later tiles are in
    // flight whatever the slab's length
    auto step = [&](int kt, auto steady, Frag<bf16_t>(&ca)[MT], Frag<bf16_t>(&cb)[NT], Frag<bf16_t>(&na)[MT],
                    Frag<bf16_t>(&nb)[NT]) {
      if constexpr (decltype(steady)::value) wait_vm<(NSTAGE - 3) * LPW>();
      else wait_tiles<NSTAGE - 3, LPW>(ke - 2 - kt);
      wait_lds();
      lds_barrier();
      if (decltype(steady)::value || kt + NSTAGE - 1 < ke) {
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
          lds_void_t* dst = (lds_void_t*)(smem + off_is + cdst[j]);
          if (NTB && j >= AI / NW && (j < LPW - 1 || IT % NW == 0 || last_is_b))
            __builtin_amdgcn_global_load_lds((const void*)csrc[j], dst, 16, 0, RT_NT_AUX);
          else __builtin_amdgcn_global_load_lds((const void*)csrc[j], dst, 16, 0, 0);
          csrc[j] += 1024;
        }
      }
      read(off_rd, na, nb);
      off_is = off_is + STG == RING ? 0 : off_is + STG;
      off_rd = off_rd + STG == RING ? 0 : off_rd + STG;
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int n = 0; n < NT; ++n) mma(acc[m][n], ca[m], cb[n]);
    };
    Frag<bf16_t> a0[MT], b0[NT], a1[MT], b1[NT];
    if (kb < ke) {
      wait_tiles<NSTAGE - 2, LPW>(ke - 1 - kb);
      lds_barrier();
      read(0, a0, b0);   // stage 0
    }
    int kt = kb;
    for (; kt + NSTAGE < ke; kt += 2) {
      step(kt, std::true_type{}, a0, b0, a1, b1);
      step(kt + 1, std::true_type{}, a1, b1, a0, b0);
    }
    for (; kt + 1 < ke; kt += 2) {
      step(kt, std::false_type{}, a0, b0, a1, b1);
      step(kt + 1, std::false_type{}, a1, b1, a0, b0);
    }
    if (kt < ke) step(kt, std::false_type{}, a0, b0, a1, b1);
  } else {
    // As in the double-buffered loop, little scalar work per k tile: every copy's source
    // advances by one k tile (2 KiB for fp32 A fragments, 1 KiB otherwise) from a pointer
    // set up once, stage offsets are counters, and one constant wait serves every step
    // that still issues a tile.
    const char* csrc[LPW];
    int cdst[LPW], cstep[LPW];
    bool cnt[LPW];
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int it = item_of(j);
      cstep[j] = it < AI ? AB : 1024;
      csrc[j] = item_src(j, kb) + (size_t)(NSTAGE - 1) * cstep[j] + lane * 16;
      cdst[j] = it * 1024;
      cnt[j] = it >= AI && stream_b;
    }
    constexpr int RING = NSTAGE * STG;
    int off_is = (NSTAGE - 1) * STG, off_rd = 0;   // tile kb + NSTAGE - 1 fills the last stage
    // STEADY: tile kt + NSTAGE - 1 exists, so NSTAGE - 2 later tiles are in flight
    auto step1 = [&](int kt, auto steady) {
      // this wave's copies of k tile kt have landed once at most the later tiles' remain
      if constexpr (decltype(steady)::value) wait_vm<(NSTAGE - 2) * LPW>();
      else wait_tiles<NSTAGE - 2, LPW>(ke - 1 - kt);
      wait_lds();      // this wave's LDS reads of tile kt-1 are done
      lds_barrier();   // every wave's copies of tile kt are visible; tile kt-1's stage is free
      if (decltype(steady)::value || kt + NSTAGE - 1 < ke) {
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
          lds_void_t* dst = (lds_void_t*)(smem + off_is + cdst[j]);
          if (cnt[j]) __builtin_amdgcn_global_load_lds((const void*)csrc[j], dst, 16, 0, RT_NT_AUX);
          else __builtin_amdgcn_global_load_lds((const void*)csrc[j], dst, 16, 0, 0);
          csrc[j] += cstep[j];
        }
      }
      const char* st = smem + off_rd;
      off_is = off_is + STG == RING ? 0 : off_is + STG;
      off_rd = off_rd + STG == RING ? 0 : off_rd + STG;
      Frag<bf16_t> bf[NT];
#pragma unroll
      for (int n = 0; n < NT; ++n)
        bf[n].v = *reinterpret_cast<const bf16x8*>(st + (AI + wn * NT + n) * 1024 + lane * 16);
      if constexpr (AF32) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const float4* pa = reinterpret_cast<const float4*>(st + (wm * MT + m) * 2048 + lane * 32);
          const float4 x0 = pa[0], x1 = pa[1];
          const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
          Frag<bf16_t> hi, lo;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const bf16_t h = f32_to_bf16(xs[e]);
            hi.v[e] = (short)h;
            lo.v[e] = (short)f32_to_bf16(xs[e] - bf16_to_f32(h));
          }
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            mma(acc[m][n], hi, bf[n]);
            mma(acc[m][n], lo, bf[n]);
          }
        }
      } else {
        Frag<bf16_t> af[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) af[m].v = *reinterpret_cast<const bf16x8*>(st + (wm * MT + m) * 1024 + lane * 16);
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int n = 0; n < NT; ++n) mma(acc[m][n], af[m], bf[n]);
      }
    };
    int kt = kb;
    for (; kt + NSTAGE - 1 < ke; ++kt) step1(kt, std::true_type{});
    for (; kt < ke; ++kt) step1(kt, std::false_type{});
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

// Columns per workgroup of the argmax (LM head) launch: 256 at 129..512 rows over a
// large vocabulary (16 waves, 8% faster than 128 columns at the 14B shape), else 128 or 64
int gemm_mid_cols(int N, int M) {
  if (M > 128 && N / 256 >= 160) return 256;
  return N / 128 >= 160 ? 128 : 64;
}

bool gemm_mid_supports(const GemmArgs& a) {
  const int k = a.e.kind;
  if (a.e.M <= 32 || a.e.M > 512) return false;
  if (k == EPI_PARTIAL) return a.ksplit >= 1;
  return a.ksplit == 1;
}

// The register epilogue covers these kinds; the others always take the slab path.
static bool mid_direct_kind(int k) {
  return k == EPI_STORE_F32 || k == EPI_STORE_ACT || k == EPI_RESID || k == EPI_SWIGLU || k == EPI_PARTIAL ||
         k == EPI_ARGMAX;
}

template <bool AF32>
static void mid_launch(const GemmArgs& a, int MB, int NB, dim3 grid, hipStream_t s) {
  // 8 waves (4 x 2, two per SIMD) for 256-row tiles and 128 x 128 tiles: 8-13% faster at
  // the 14B layer shapes and 3-6% at the 8B gate|up and q|k|v than 4 waves (2 x 2); the
  // narrower and wider 128-row tiles stay at 4 waves.  The 256 x 160 and 256 x 192
  // (gate|up) and 256 x 256 (LM head) tiles take 16 waves (8 x 2), another 11% / 8% at
  // the 14B shape.  256 x 160 makes 218 workgroups of the 14B gate|up where 256 x 192
  // makes 182 on 256 CUs: 3-5% faster there and 6% at a 512-row 4B-shape gate|up;
  // deeper LDS rings (5, 6 stages) measured no faster at any of these shapes.  Likewise
  // 128 x 96 makes 256 workgroups of the 8B gate|up at 128 rows (192 of 128 x 128):
  // 50.6 -> 49.0 us.  The bf16 256-row tiles below the LM head's read each k tile's
  // fragments during the previous tile's MFMAs (five LDS stages): 14B gate|up 112.6 ->
  // 107.7 us, down 58.6 -> 54.4, q|k|v 29.3 -> 28.2 (round 21.10 -> 20.90 ms); at 128 rows
  // (8B shape) the same change measured no faster, and staging the tiles through
  // registers (16-byte loads two to four tiles ahead, written to LDS by the waves) instead
  // of direct-to-LDS copies was slower (gate|up 119 us).
  // The output tile is split spatially, so every element is accumulated over k in the
  // same order either way.
  if (MB == 128) {
    if (NB == 64) RT_LAUNCH((gemm_mid_kernel<128, 64, 4, AF32, 4>), grid, dim3(256), 0, s, a);
    else if (NB == 96) { if constexpr (!AF32) RT_LAUNCH((gemm_mid_kernel<128, 96, 4, false, 8>), grid, dim3(512), 0, s, a); }
    else if (NB == 128) RT_LAUNCH((gemm_mid_kernel<128, 128, 4, AF32, 8>), grid, dim3(512), 0, s, a);
    else if constexpr (!AF32) RT_LAUNCH((gemm_mid_kernel<128, 192, 4, false, 4>), grid, dim3(256), 0, s, a);
  } else {
    if constexpr (AF32) {
      if (NB == 64) RT_LAUNCH((gemm_mid_kernel<256, 64, 3, true, 8>), grid, dim3(512), 0, s, a);
      else if (NB == 128) RT_LAUNCH((gemm_mid_kernel<256, 128, 3, true, 8>), grid, dim3(512), 0, s, a);
    } else {
      // one row tile: every weight tile is read by one workgroup (non-temporal copies)
      const bool one = grid.y == 1;
      if (NB == 64 && one) RT_LAUNCH((gemm_mid_kernel<256, 64, 5, false, 8, true, true>), grid, dim3(512), 0, s, a);
      else if (NB == 64) RT_LAUNCH((gemm_mid_kernel<256, 64, 5, false, 8, true>), grid, dim3(512), 0, s, a);
      else if (NB == 128 && one) RT_LAUNCH((gemm_mid_kernel<256, 128, 5, false, 8, true, true>), grid, dim3(512), 0, s, a);
      else if (NB == 128) RT_LAUNCH((gemm_mid_kernel<256, 128, 5, false, 8, true>), grid, dim3(512), 0, s, a);
      else if (NB == 160 && one) RT_LAUNCH((gemm_mid_kernel<256, 160, 5, false, 16, true, true>), grid, dim3(1024), 0, s, a);
      else if (NB == 160) RT_LAUNCH((gemm_mid_kernel<256, 160, 5, false, 16, true>), grid, dim3(1024), 0, s, a);
      else if (NB == 192 && one) RT_LAUNCH((gemm_mid_kernel<256, 192, 5, false, 16, true, true>), grid, dim3(1024), 0, s, a);
      else if (NB == 192) RT_LAUNCH((gemm_mid_kernel<256, 192, 5, false, 16, true>), grid, dim3(1024), 0, s, a);
      else RT_LAUNCH((gemm_mid_kernel<256, 256, 3, false, 16>), grid, dim3(1024), 0, s, a);
    }
  }
}

// Tile width and k slabs.  A workgroup streams (MB + NB) / 16 KiB through LDS per k
// tile, about one workgroup per compute unit is resident for the wide tiles, and the
// grid runs in rounds of 256 workgroups, so the estimated time of a choice is
// rounds x (MB + NB) / 16 x k tiles per slab (slabs cost an extra pass over the
// output).  Outputs of fewer than 128 tiles take k slabs to fill the chip.  The choices
// reproduce the fastest measured configuration at the Qwen3-8B and 14B layer shapes.
struct MidPlan { int NB, ks; };
static MidPlan mid_plan(const GemmArgs& a, int MB, bool a_f32) {
  const int M = a.e.M, N = a.e.N, KT = a.Kp / kTileK;
  const int ai = (MB / 16) * (a_f32 ? 2 : 1);
  const size_t slab = (size_t)M * N;
  MidPlan best{64, 1};
  double best_cost = 1e30;
  for (int NB : {64, 96, 128, 160, 192}) {
    if ((NB >= 160 || NB == 96) && a_f32) continue;
    if (NB == 160 && (MB != 256 || a.e.kind == EPI_PARTIAL)) continue;
    if (NB == 96 && (MB != 128 || a.e.kind == EPI_PARTIAL)) continue;
    const long tiles = (long)((N + NB - 1) / NB) * ((M + MB - 1) / MB);
    int ks = 1;
    if (a.e.kind == EPI_PARTIAL) {
      ks = a.ksplit;
    } else if (tiles < 128) {
      ks = (int)(256 / tiles);
      if (ks > KT / 8) ks = KT / 8;
      if (ks > 8) ks = 8;
      if ((size_t)ks > a.partial_floats / slab) ks = (int)(a.partial_floats / slab);
      if (ks < 1) ks = 1;
    }
    if ((NB >= 160 || NB == 96) && ks > 1) continue;   // tiles for large outputs only
    const double rounds = (double)((tiles * ks + 255) / 256);
    double cost = rounds * (ai + NB / 16) * ((KT + ks - 1) / ks);
    // slabs are written and read back once (mostly from cache): a quarter of their
    // bytes relative to the weights'
    if (ks > 1 && a.e.kind != EPI_PARTIAL) cost *= 1.0 + (double)ks * M / (KT * kTileK);
    if (cost < best_cost) { best_cost = cost; best = MidPlan{NB, ks}; }
  }
  return best;
}

int gemm_mid_store_slabs(const GemmArgs& a, bool a_f32) {
  GemmArgs g = a;
  if (g.e.kind == EPI_PARTIAL) g.e.kind = EPI_STORE_F32;
  if (g.e.M <= 32 || g.e.M > 512) return 1;
  return mid_plan(g, g.e.M <= 128 ? 128 : 256, a_f32).ks;
}

int gemm_mid_partial_slabs(const GemmArgs& a, bool a_f32, int max_slabs) {
  if (a.e.M <= 32 || a.e.M > 512) return 1;
  const int MB = a.e.M <= 128 ? 128 : 256;
  GemmArgs g = a;
  g.e.kind = EPI_PARTIAL;
  int best = 1;
  double best_cost = 1e30;
  for (int ks = 1; ks <= max_slabs; ++ks) {
    if ((size_t)ks * g.e.M * g.e.N > a.partial_floats) break;
    g.ksplit = ks;
    const MidPlan pl = mid_plan(g, MB, a_f32);
    const int KT = a.Kp / kTileK;
    const long tiles = (long)((g.e.N + pl.NB - 1) / pl.NB) * ((g.e.M + MB - 1) / MB);
    const double cost = (double)((tiles * ks + 255) / 256) * ((MB / 16) * (a_f32 ? 2 : 1) + pl.NB / 16) *
                        ((KT + ks - 1) / ks);
    if (cost < best_cost) { best_cost = cost; best = ks; }
  }
  return best;
}

hipError_t gemm_mid(const GemmArgs& a, bool a_f32, hipStream_t s) {
  if (!gemm_mid_supports(a)) return hipErrorInvalidValue;
  const int M = a.e.M, N = a.e.N;
  const int MB = M <= 128 ? 128 : 256;
  if (a.e.kind == EPI_ARGMAX) {   // the caller sizes its key parts by gemm_mid_cols
    const int NB = gemm_mid_cols(N, M);
    const dim3 grid((N + NB - 1) / NB, (M + MB - 1) / MB, 1);
    if (a_f32) mid_launch<true>(a, MB, NB, grid, s);
    else mid_launch<false>(a, MB, NB, grid, s);
    return hipGetLastError();
  }
  const MidPlan pl = mid_plan(a, MB, a_f32);
  const int NB = pl.NB, ks = pl.ks;
  const dim3 grid((N + NB - 1) / NB, (M + MB - 1) / MB, ks);
  if (a.e.kind == EPI_PARTIAL || (ks == 1 && mid_direct_kind(a.e.kind))) {
    if (a_f32) mid_launch<true>(a, MB, NB, grid, s);
    else mid_launch<false>(a, MB, NB, grid, s);
    return hipGetLastError();
  }
  const size_t slab = (size_t)M * N;
  if (!a.partial || a.partial_floats < slab * ks) return hipErrorInvalidValue;
  GemmArgs g = a;
  g.ksplit = ks;
  g.e.kind = EPI_PARTIAL; g.e.out_f32 = a.partial; g.e.ldo = N; g.e.part_stride = slab;
  if (a_f32) mid_launch<true>(g, MB, NB, grid, s);
  else mid_launch<false>(g, MB, NB, grid, s);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return gemm_split_epilogue<bf16_t>(a.e, a.partial, ks, s);
}

}  // namespace rt
