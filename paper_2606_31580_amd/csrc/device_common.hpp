// Device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

namespace laser {

// Calls f(integral_constant<int, i>) for i = 0 .. N-1 (compile-time ring-buffer indices, so
// register arrays are never indexed dynamically).
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4;

struct bf16_t {
  uint16_t bits;
};
// OCP FP8 E4M3 (the "fn" variant: bias 7, no infinities, 0x7f/0xff NaN, largest finite 448).
struct fp8_t {
  uint8_t bits;
};

// fp32 -> E4M3 bits: round to nearest even on the E4M3 grid (spacing 2^(e-3) in binade
// [2^e, 2^(e+1)) for e >= -6, 2^-9 below), magnitudes that round past 448 saturate to 448,
// NaN stays NaN.
__device__ __forceinline__ uint8_t f2fp8(float v) {
  const uint32_t sign = (__float_as_uint(v) >> 24) & 0x80u;
  const float a = fabsf(v);
  if (!(a == a)) return (uint8_t)(sign | 0x7fu);
  const int e = a >= 0x1p-6f ? (int)((__float_as_uint(a) >> 23) & 0xffu) - 127 : -6;
  const float ulp = __builtin_amdgcn_ldexpf(1.0f, (e > 8 ? 8 : e) - 3);
  float r = rintf(a / ulp) * ulp;  // exact scaling by a power of two; rint rounds half to even
  if (r > 448.0f) r = 448.0f;
  if (r < 0x1p-6f) return (uint8_t)(sign | (uint32_t)(r * 512.0f));  // zero or subnormal: r = m * 2^-9
  const int re = (int)((__float_as_uint(r) >> 23) & 0xffu) - 127;   // r may have moved up a binade
  const uint32_t m = (__float_as_uint(r) >> 20) & 7u;
  return (uint8_t)(sign | ((uint32_t)(re + 7) << 3) | m);
}

// Four E4M3 bytes of w -> their values as bf16 bit pairs (exact: E4M3 has 3 fraction bits):
// lo = bytes 0, 1, hi = bytes 2, 3 (element 0 in the low half of each word).
__device__ __forceinline__ void fp8x4_to_bf16x4(uint32_t w, uint32_t& lo, uint32_t& hi) {
  const auto a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const auto b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  lo = __builtin_amdgcn_perm(__float_as_uint(a[1]), __float_as_uint(a[0]), 0x07060302u);
  hi = __builtin_amdgcn_perm(__float_as_uint(b[1]), __float_as_uint(b[0]), 0x07060302u);
}

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Split x into bf16 hi + bf16 lo (x - hi, rounded), so hi + lo carries ~16 significand bits.
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
  hi = f2bf(x);
  lo = f2bf(x - bf2f(hi));
}

// Two floats as packed bf16 pairs hi = trunc(x), lo = trunc(x - hi) (element 0 in the low
// half): hi + lo keeps 16 significand bits (relative error below 2^-14), for a third of the
// instructions of the rounded split.
__device__ __forceinline__ void split_trunc2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const uint32_t b0 = __float_as_uint(x0) & 0xffff0000u, b1 = __float_as_uint(x1) & 0xffff0000u;
  const uint32_t r0 = __float_as_uint(x0 - __uint_as_float(b0)), r1 = __float_as_uint(x1 - __uint_as_float(b1));
  hi = __builtin_amdgcn_perm(b1, b0, 0x07060302u);
  lo = __builtin_amdgcn_perm(r1, r0, 0x07060302u);
}

// Loads through the global address space.  A pointer built by arithmetic, or picked among
// several tensors, is otherwise read with flat instructions, which count against the LDS and
// scalar-load counter as well: every later wait on that counter then covers them too.
template <class T>
using global_ptr = const __attribute__((address_space(1))) T*;
template <class T>
__device__ __forceinline__ T ld_global(const void* p) {
  return *(global_ptr<T>)p;
}
__device__ __forceinline__ u32x4 ld_nt16(const void* p) { return __builtin_nontemporal_load((global_ptr<u32x4>)p); }
__device__ __forceinline__ u32x2 ld_nt8(const void* p) { return __builtin_nontemporal_load((global_ptr<u32x2>)p); }

// Cross-lane primitives of gfx950 (no LDS traffic): DPP inside 16-lane rows, and the
// permlane swaps across rows.  permlane16_swap(a, b) leaves (a.r0, b.r0, a.r2, b.r2) and
// (a.r1, b.r1, a.r3, b.r3) (rows of 16 lanes); permlane32_swap(a, b) leaves (a.lo, b.lo) and
// (a.hi, b.hi).  Summing the two results pairs every lane with its partner 16 or 32 lanes
// away, in an order that does not depend on the lane.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppQuad1032 = 0xB1;    // lane ^ 1
constexpr int kDppQuad2301 = 0x4E;    // lane ^ 2
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within 8 lanes
constexpr int kDppRowRor8 = 0x128;    // lane ^ 8 within 16 lanes

__device__ __forceinline__ void swap16(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap32(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
// x combined with the value of the lane 16 (32) away: sum or max.
__device__ __forceinline__ float sum_x16(float x) {
  float a = x, b = x;
  swap16(a, b);
  return a + b;
}
__device__ __forceinline__ float sum_x32(float x) {
  float a = x, b = x;
  swap32(a, b);
  return a + b;
}
__device__ __forceinline__ float max_x16(float x) {
  float a = x, b = x;
  swap16(a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float max_x32(float x) {
  float a = x, b = x;
  swap32(a, b);
  return fmaxf(a, b);
}
// Sum over the 16 lanes of a row, in every lane of it.
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp_f<kDppQuad1032>(x);
  x += dpp_f<kDppQuad2301>(x);
  x += dpp_f<kDppHalfMirror>(x);
  x += dpp_f<kDppRowRor8>(x);
  return x;
}

__device__ __forceinline__ float wave_sum(float x) { return sum_x32(sum_x16(row_sum16(x))); }

// Maximum / minimum over the 16 lanes of a row, then over the wave, in every lane.
__device__ __forceinline__ float row_max16(float x) {
  x = fmaxf(x, dpp_f<kDppQuad1032>(x));
  x = fmaxf(x, dpp_f<kDppQuad2301>(x));
  x = fmaxf(x, dpp_f<kDppHalfMirror>(x));
  x = fmaxf(x, dpp_f<kDppRowRor8>(x));
  return x;
}
__device__ __forceinline__ float wave_max(float x) { return max_x32(max_x16(row_max16(x))); }
__device__ __forceinline__ float wave_min(float x) { return -wave_max(-x); }

// Cross-workgroup hand-off without cache write-back fences.  Each XCD has its own L2, and a
// plain store can sit there unseen by the other XCDs until the kernel ends; an agent-scope
// release fence writes back the whole L2, and many workgroups fencing at once serialise on it
// (about 12 us more for 448 workgroups, measured).  Buffer accesses with the device-scope bit
// (sc1) instead write through to, and read from, the level all XCDs share.  So a workgroup
// that stores its result this way, waits for the stores to complete, then bumps a counter
// with a device-scope atomic, has made the result visible to whichever workgroup sees the
// counter's final value and reads the result with device-scope loads (checked on the device:
// no stale value over 400 launches of 448 and 768 workgroups on different XCDs).
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
constexpr int kDevScope = 16;  // buffer cache-policy operand: sc1 (device scope)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dev_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void st_dev16(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), r, (int)off, 0, kDevScope);
}
__device__ __forceinline__ void st_dev8(__amdgpu_buffer_rsrc_t r, uint32_t off, float a, float b) {
  __builtin_amdgcn_raw_buffer_store_b64(i32x2{(int)__float_as_uint(a), (int)__float_as_uint(b)}, r, (int)off, 0,
                                        kDevScope);
}
__device__ __forceinline__ f32x4 ld_dev16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kDevScope));
}
__device__ __forceinline__ i32x2 ld_dev8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kDevScope);
}
// Waits until every memory access this wave issued has completed (stores acknowledged), and
// keeps the compiler from moving accesses across the wait.
__device__ __forceinline__ void wait_mem() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Value of element e of a stored tensor (fp32 or bf16 bits).
template <class WT>
__device__ __forceinline__ float ldw(const void* base, size_t e);
template <>
__device__ __forceinline__ float ldw<float>(const void* base, size_t e) {
  return ((const float*)base)[e];
}
template <>
__device__ __forceinline__ float ldw<bf16_t>(const void* base, size_t e) {
  return bf2f(((const uint16_t*)base)[e]);
}

// Store a value in the storage type (bf16: round to nearest even; fp8: f2fp8).
template <class WT>
__device__ __forceinline__ void stw(void* base, size_t e, float v);
template <>
__device__ __forceinline__ void stw<fp8_t>(void* base, size_t e, float v) {
  ((uint8_t*)base)[e] = f2fp8(v);
}
template <>
__device__ __forceinline__ void stw<float>(void* base, size_t e, float v) {
  ((float*)base)[e] = v;
}
template <>
__device__ __forceinline__ void stw<bf16_t>(void* base, size_t e, float v) {
  ((uint16_t*)base)[e] = f2bf(v);
}

// Offsets of element (t, d) inside a KV page block (16 positions x hd), chosen so that the
// attention kernel's matrix-core operand loads are contiguous per wave instruction.
__device__ __forceinline__ int k_block_off(int t, int d) { return (((d >> 5) * 4 + ((d & 31) >> 3)) * 16 + t) * 8 + (d & 7); }
__device__ __forceinline__ int v_block_off(int t, int d) { return (((d >> 4) * 4 + (t >> 2)) * 16 + (d & 15)) * 4 + (t & 3); }

}  // namespace laser
