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

// Four OCP E4M3FN codes (one dword) -> four bf16 (two dwords), byte i to
// element i.  Every E4M3 value, subnormals included, is exactly
// representable in bf16; the packed scaled conversion with a unit scale
// gives exactly those values (checked against the fp32 route on every code
// pair), one instruction per two codes.
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t codes) {
  u32x2 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, false));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes, 1.0f, true));
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

// ------------------------------------------------------------------- LDS
// LDS is addressed through address-space-3 pointers throughout, so no
// generic <-> LDS conversion happens at run time.
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_t;

// View of a __shared__ array as an LDS pointer (folds to a constant).
template <typename T>
__device__ __forceinline__ lds_u8 *as_lds(T *shared_array) {
  return (lds_u8 *)(shared_array);
}

__device__ __forceinline__ u32x2 ds_read_tr16(const lds_u8 *p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(p));
  return __builtin_bit_cast(u32x2, v);
}
// Transposed 8-bit read: within each 16-lane group, lane i = 2m + h of the
// group names an 8-byte run; lane 8h + k of the group receives byte k of the
// runs of lanes h, 2 + h, ..., 14 + h (byte m from lane 2m + h).  With lane
// 2m + h pointing at row m, columns 8h .. 8h + 7 of a row-major byte matrix,
// group lane o gets column o of rows 0..7 (layout checked on the GPU).
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2_t;
__device__ __forceinline__ u32x2 ds_read_tr8(const lds_u8 *p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2_t *)(p)));
}
__device__ __forceinline__ u32x4 lds_ld16(const lds_u8 *p) { return *(const lds_u32x4_t *)(p); }
typedef __attribute__((address_space(3))) u32x2 lds_u32x2_t;
__device__ __forceinline__ u32x2 lds_ld8(const lds_u8 *p) { return *(const lds_u32x2_t *)(p); }

// Eight E4M3FN codes (8 bytes of LDS) -> one 16-byte chunk of bf16 values.
__device__ __forceinline__ u32x4 fp8x8_to_bf16x8(u32x2 codes) {
  const u32x2 a = fp8x4_to_bf16x4(codes.x), b = fp8x4_to_bf16x4(codes.y);
  return u32x4{a.x, a.y, b.x, b.y};
}
__device__ __forceinline__ void lds_st16(lds_u8 *p, u32x4 v) { *(lds_u32x4_t *)(p) = v; }

// Read-only tables (block table, fp8 scales) are read through the constant
// address space so that wave-uniform lookups become scalar loads.
template <typename T>
__device__ __forceinline__ T ldc(const T *p, int i) {
  return ((const __attribute__((address_space(4))) T *)(p))[i];
}

// Wave-wide 16-byte-per-lane loads from global memory straight into LDS:
// lane l's 16 bytes land at dst + 16 l (dst wave-uniform, passed in M0).
// Issued as inline assembly so that the compiler does not track them; the
// kernels order them explicitly (s_waitcnt vmcnt, then a barrier when other
// waves read the data; a stage is overwritten only after its readers have
// passed a barrier or, for a single-wave ring, after the wave has consumed
// it).
__device__ __forceinline__ uint32_t lds_offset(const lds_u8 *p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}

// The compiler's hazard recognizer cannot see that these asm statements are
// vector memory instructions, so they carry their own wait states: the base
// registers are often written by v_readfirstlane right before the load (a
// VALU write of an SGPR needs 5 wait states before a VMEM instruction reads
// it), and M0 by an s_mov (an SALU write of M0 needs 1 before an LDS-DMA
// load).  Without them the load can use a stale base address.
#define CKV_DMA_WAIT "s_nop 4\n\t"

// Per-lane 64-bit source address.
__device__ __forceinline__ void dma16(const void *g, lds_u8 *dst) {
  asm volatile(CKV_DMA_WAIT "global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds_offset(dst))
               : "memory");
}

// Wave-uniform 64-bit base (scalar registers) plus a per-lane 32-bit byte
// offset: no per-lane 64-bit address arithmetic.  NT marks the load
// non-temporal, for data that is read once (decode's V stream); data that
// other workgroups re-read from L2 (prefill's K/V) keeps the default policy.
template <bool NT = false>
__device__ __forceinline__ void dma16_sv(const void *sbase, uint32_t voff, lds_u8 *dst) {
  // readfirstlane returns a signed int: widen each half as unsigned so the
  // low word is not sign-extended into the high word
  const uint64_t base = (uint64_t)(uintptr_t)sbase;
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)base);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
  const uint64_t sb = ((uint64_t)hi << 32) | (uint64_t)lo;
  if constexpr (NT)
    asm volatile(CKV_DMA_WAIT "global_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(sb), "{m0}"(lds_offset(dst))
                 : "memory");
  else
    asm volatile(CKV_DMA_WAIT "global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sb), "{m0}"(lds_offset(dst))
                 : "memory");
}

// Sum of two bf16 values packed in a dword, accumulated in fp32.
__device__ __forceinline__ float add_bf16x2(uint32_t w, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w),
                                         __builtin_bit_cast(bf16x2, 0x3f803f80u), acc, false);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

}  // namespace ckv
