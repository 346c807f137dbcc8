// Device-side helpers shared by the ReTrace round kernels (gfx950, wave64).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rt {

// Profiling hook of the host launchers: when a pair of HIP events is armed for the next
// launch on this thread, that launch goes through hipExtLaunchKernel, which records the
// events at the kernel's own start and end, so their elapsed time is the kernel's
// execution time without queueing gaps.
// A launch marked `skip` is not issued (kernel replay records only one launch class).
struct LaunchEvents {
  hipEvent_t b = nullptr, e = nullptr;
  bool used = false;
  bool skip = false;
};
LaunchEvents& launch_events();   // thread-local
#define RT_LAUNCH(kernel, grid, block, shmem, stream, ...)                                        \
  do {                                                                                            \
    ::rt::LaunchEvents& ev_ = ::rt::launch_events();                                              \
    if (ev_.skip) {                                                                               \
    } else if (ev_.b && !ev_.used) {                                                              \
      ev_.used = true;                                                                            \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev_.b, ev_.e, 0, __VA_ARGS__);    \
    } else {                                                                                      \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                        \
    }                                                                                             \
  } while (0)

typedef uint16_t bf16_t;                                   // bfloat16 bit pattern
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kWave = 64;
constexpr int kTileK = 32;        // k extent of one packed weight tile
constexpr int kTileN = 16;        // n extent of one packed weight tile
constexpr int kPage = 16;         // tokens per KV page

__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
// Round to nearest even (gfx950 converts in hardware; NaN stays NaN, quieted).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  _Float16 v; __builtin_memcpy(&v, &h, 2); return (float)v;
}
__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  _Float16 v = (_Float16)f; uint16_t h; __builtin_memcpy(&h, &v, 2); return h;
}

// Storage-type traits: T is the weight / activation element type (bf16 bit pattern or float).
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  __device__ static __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v); }
  __device__ static __forceinline__ bf16_t from_f32(float v) { return f32_to_bf16(v); }
};
template <> struct Elem<float> {
  static constexpr int kBytes = 4;
  __device__ static __forceinline__ float to_f32(float v) { return v; }
  __device__ static __forceinline__ float from_f32(float v) { return v; }
};

// Eight consecutive k-values of one operand row, as held by one lane for one
// 16x16 MFMA tile step over 32 k (the lane's k-group is (lane/16)*8..+8).
template <typename T> struct Frag;
// Weight and K / V streams are read once per pass: load_stream marks the load
// non-temporal, which on this chip streams HBM at 6.9-7.2 TB/s against 6.0-6.2 TB/s for
// plain loads of the same data (a 1 GiB read, one kernel).
#ifndef RT_NO_NT
#define RT_NT_AUX 2   // cache-policy bits of a direct-to-LDS copy: non-temporal
#else
#define RT_NT_AUX 0
#endif
template <typename V>
__device__ __forceinline__ V ld_stream(const V* p) {
#ifndef RT_NO_NT
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}
template <> struct Frag<bf16_t> {
  bf16x8 v;
  __device__ __forceinline__ void load(const bf16_t* p) { v = *reinterpret_cast<const bf16x8*>(p); }
  __device__ __forceinline__ void load_stream(const bf16_t* p) { v = ld_stream(reinterpret_cast<const bf16x8*>(p)); }
  __device__ __forceinline__ void store(bf16_t* p) const { *reinterpret_cast<bf16x8*>(p) = v; }
  __device__ __forceinline__ void zero() { for (int i = 0; i < 8; ++i) v[i] = 0; }
  __device__ __forceinline__ float get(int i) const { return bf16_to_f32((bf16_t)v[i]); }
  __device__ __forceinline__ void set(int i, float f) { v[i] = (short)f32_to_bf16(f); }
  // elements 0..3 from p0[0..3] and 4..7 from p1[0..3] (8-byte aligned)
  __device__ __forceinline__ void load_halves(const bf16_t* p0, const bf16_t* p1) {
    const uint2 a = *reinterpret_cast<const uint2*>(p0), b = *reinterpret_cast<const uint2*>(p1);
    v[0] = (short)(a.x & 0xffff); v[1] = (short)(a.x >> 16); v[2] = (short)(a.y & 0xffff); v[3] = (short)(a.y >> 16);
    v[4] = (short)(b.x & 0xffff); v[5] = (short)(b.x >> 16); v[6] = (short)(b.y & 0xffff); v[7] = (short)(b.y >> 16);
  }
};
template <> struct Frag<float> {
  float4 lo, hi;
  __device__ __forceinline__ void load(const float* p) {
    lo = *reinterpret_cast<const float4*>(p); hi = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ void load_stream(const float* p) {
    const f32x4 a = ld_stream(reinterpret_cast<const f32x4*>(p));
    const f32x4 b = ld_stream(reinterpret_cast<const f32x4*>(p + 4));
    lo = make_float4(a[0], a[1], a[2], a[3]); hi = make_float4(b[0], b[1], b[2], b[3]);
  }
  __device__ __forceinline__ void store(float* p) const {
    *reinterpret_cast<float4*>(p) = lo; *reinterpret_cast<float4*>(p + 4) = hi;
  }
  __device__ __forceinline__ void zero() { lo = make_float4(0, 0, 0, 0); hi = lo; }
  __device__ __forceinline__ float get(int i) const {
    switch (i) { case 0: return lo.x; case 1: return lo.y; case 2: return lo.z; case 3: return lo.w;
                 case 4: return hi.x; case 5: return hi.y; case 6: return hi.z; default: return hi.w; }
  }
  __device__ __forceinline__ void set(int i, float f) {
    switch (i) { case 0: lo.x = f; break; case 1: lo.y = f; break; case 2: lo.z = f; break;
                 case 3: lo.w = f; break; case 4: hi.x = f; break; case 5: hi.y = f; break;
                 case 6: hi.z = f; break; default: hi.w = f; }
  }
  __device__ __forceinline__ void load_halves(const float* p0, const float* p1) {
    lo = *reinterpret_cast<const float4*>(p0);
    hi = *reinterpret_cast<const float4*>(p1);
  }
};

// acc[16x16] += A[16 x 32] * B[32 x 16]; lane l holds A row l%16 / B column l%16,
// k-values (l/16)*8..+8 (any k permutation shared by A and B is valid).
// Output: lane l, register i -> row 4*(l/16)+i, column l%16.
__device__ __forceinline__ void mma(f32x4& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4& acc, const Frag<float>& a, const Frag<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, acc, 0, 0, 0);
}

__device__ __forceinline__ float warp_sum(float v, int width = 64) {
  for (int o = width / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float warp_max(float v, int width = 64) {
  for (int o = width / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Reductions over the four lanes l, l^16, l^32, l^48 (the same MFMA column in each
// 16-lane group) with the gfx950 lane-swap instructions: each returns the pair
// {v[l], v[l ^ 16]} resp. {v[l], v[l ^ 32]}, no LDS round trip.
__device__ __forceinline__ float group4_max(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group4_sum(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// q / k per-head RMSNorm and rotate-half RoPE of one element pair (x_i, x_{i + hd/2}),
// written out operation by operation with contraction into fused multiply-adds off, so
// that every kernel that applies them -- the q|k|v post-processing and the attention
// kernel that takes it over in the rounds -- rounds identically.  qk_sq is a pair's
// share of the head's sum of squares; the shares are summed over i in the butterfly
// order of xor offsets hd/4, hd/8, .., 1.
__device__ __forceinline__ float qk_sq(float x0, float x1) {
#pragma clang fp contract(off)
  return x0 * x0 + x1 * x1;
}
__device__ __forceinline__ float qk_inv(float ss, int hd, float eps) {
#pragma clang fp contract(off)
  return 1.0f / sqrtf(ss / (float)hd + eps);
}
__device__ __forceinline__ void qk_norm_rope(float& x0, float& x1, float inv, float w0, float w1, float cs, float sn) {
#pragma clang fp contract(off)
  const float a = x0 * inv * w0, b = x1 * inv * w1;
  x0 = a * cs - b * sn;
  x1 = b * cs + a * sn;
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Workgroup barrier that orders LDS accesses for the compiler but does not wait for
// outstanding vector-memory operations (direct-to-LDS copies are waited for explicitly
// with wait_vm, so that later pipeline stages stay in flight).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// s_waitcnt lgkmcnt(0) leaving the other counters alone: this wave's LDS accesses are done.
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xc07f); }
// s_waitcnt vmcnt(N) leaving the other counters alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Fragment-ordered ("packed") layout of GEMM A operands: element (m, k) of an [M][Kp]
// operand lives at (m/16)*ldg + (k/32)*512 + ((m%16) + 16*((k%32)/8))*8 + k%8 with
// ldg = 16*Kp, so the fragment one wave needs for a 16-row group and a 32-wide k tile is
// 512 contiguous elements (lane l reads elements l*8 .. l*8+7).
__host__ __device__ __forceinline__ size_t pa_index(int m, int k, size_t ldg) {
  return (size_t)(m >> 4) * ldg + (size_t)(k >> 5) * 512 + (size_t)((((m & 15) + 16 * ((k & 31) >> 3)) << 3) + (k & 7));
}

// Reductions over the 16 lanes of a DPP row (lanes 16r..16r+15), by row rotations:
// every lane of the row ends with the result.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0x128>(v));   // row_ror:8
  v = fmaxf(v, dpp<0x124>(v));   // row_ror:4
  v = fmaxf(v, dpp<0x122>(v));   // row_ror:2
  v = fmaxf(v, dpp<0x121>(v));   // row_ror:1
  return v;
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0x128>(v);
  v += dpp<0x124>(v);
  v += dpp<0x122>(v);
  v += dpp<0x121>(v);
  return v;
}

// Monotone map float -> uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t orderable(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// 64-bit argmax key: value in the high word, (0xffffffff - index) in the low word, so
// an unsigned max picks the larger value and, among equal values, the lower index.
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t idx) {
  return ((uint64_t)orderable(v) << 32) | (uint64_t)(0xffffffffu - idx);
}
__device__ __forceinline__ int32_t key_index(uint64_t key) {
  return (int32_t)(0xffffffffu - (uint32_t)(key & 0xffffffffu));
}

}  // namespace rt
