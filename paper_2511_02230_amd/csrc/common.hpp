// Device-side helpers shared by the ckv kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ckv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

// ---------------------------------------------------------------- loads
template <typename T>
__device__ __forceinline__ T ld(const void *p) {
  return *reinterpret_cast<const T *>(p);
}
template <typename T>
__device__ __forceinline__ void st(void *p, T v) {
  *reinterpret_cast<T *>(p) = v;
}

// ------------------------------------------------------------ conversions
// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Four OCP E4M3FN codes (one dword) -> four bf16 (two dwords).  Every E4M3
// value, subnormals included, is exactly representable in bf16, so the
// detour through fp32 is exact.
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t codes) {
  f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)codes, false);
  f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)codes, true);
  u32x2 r;
  r.x = pack_bf16x2(lo.x, lo.y);
  r.y = pack_bf16x2(hi.x, hi.y);
  return r;
}

// Select 16-bit halves: result = {lo16(a), lo16(b)} or {hi16(a), hi16(b)}.
__device__ __forceinline__ uint32_t pack_lo16(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t pack_hi16(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// ------------------------------------------------------------------ MFMA
// D(32x32, f32) += A(32x16, bf16) * B(16x32, bf16).
// Lane l supplies row l%32 of A and column l%32 of B, k-slots 8*(l/32)+0..7;
// it receives column l%32 of D, rows 8*i + 4*(l/32) + j in element 4*i + j.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// D(16x16, f32) += A(16x32, bf16) * B(32x16, bf16).
// Lane l supplies row l%16 of A and column l%16 of B, k-slots 8*(l/16)+0..7;
// it receives column l%16 of D, rows 4*(l/16) + j in element j.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// --------------------------------------------------------------- shuffles
__device__ __forceinline__ float shfl_xor(float v, int mask) {
  int lane = __lane_id();
  return __int_as_float(__builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, __float_as_int(v)));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace ckv
