// Device-side helpers shared by the ASP kernels (gfx950).
//
// The 4-bit group quantizer of Eq. 2 (Sec. 3) as the kernels apply it:
//   scale = fl32(absmax / 7)            (0 when absmax < 7 * 2^-126)
//   inv   = fl32(1 / scale)             (0 when scale == 0)
//   code  = clamp(rint(fl32(v * inv)), -8, 7)   rint = round half to even
// Division is IEEE correctly rounded (hipcc's default for float '/'); no
// contraction is allowed anywhere in this file.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace qwam {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef short v8s __attribute__((ext_vector_type(8)));

constexpr int kGroup = 64;

__device__ __forceinline__ float q4_scale(float amax) {
  // 7 * 2^-126 = 1.75 * 2^-124
  return (amax < 0x1.cp-124f) ? 0.0f : amax / 7.0f;
}

__device__ __forceinline__ float q4_inv(float scale) {
  return (scale == 0.0f) ? 0.0f : 1.0f / scale;
}

// Returns the 4-bit two's-complement nibble (0..15) of the code of v.
__device__ __forceinline__ uint32_t q4_nibble(float v, float inv) {
  float p = v * inv;
  p = __builtin_rintf(p);
  p = __builtin_fminf(__builtin_fmaxf(p, -8.0f), 7.0f);
  return static_cast<uint32_t>(static_cast<int>(p)) & 0xFu;
}

// bf16 bits -> float (exact).
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// float -> bf16 bits, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// double -> bf16 bits, round to nearest, ties to even, in one rounding (finite
// inputs): the double is first rounded to float by round-to-odd (truncate, and
// set the last bit when inexact), which keeps enough bits for the second
// rounding to bf16 to be the correctly rounded result.
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double d) {
  const float f = static_cast<float>(d);
  uint32_t u = __float_as_uint(f);
  const double back = static_cast<double>(f);
  if (back != d) {
    if (__builtin_fabs(back) > __builtin_fabs(d)) u -= 1u;   // rounded away from zero: step back
    u |= 1u;
  }
  return f32_to_bf16_rne(__uint_as_float(u));
}

// Two floats -> packed bf16x2 (lo in bits 0..15), RNE.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

// Packed code word, the storage format of every 4-bit code (qwam.h): the codes
// c[k0..k0+7] of 8 consecutive channels share one little-endian 32-bit word,
// byte j holding |c[k0+2j]| in bits 0-2 and its sign in bit 7, |c[k0+2j+1]| in
// bits 4-6, and in bit 3 the sign of the odd code of byte j-1 (of byte 3 for
// j = 0).  The quantizer never yields -8 (|v * inv| <= 7 (1 + 3u) < 7.5), so
// three magnitude bits suffice; a zero code has sign 0.  Masking a word with
// 0x87878787, and the word rotated right by 4 with the same mask, gives the
// even and the odd codes as FP8 e4m3 bytes of value code * 2^-9.
//
// Conversion from 8 two's-complement nibbles t (nibble i = code of k0+i): the
// negative nibbles are negated (one's complement + 1: carry-free, as the
// result lies in 1..7) and every sign bit moves 4 places up, circularly.
__device__ __forceinline__ uint32_t twos_nibbles_to_code_word(uint32_t t) {
  const uint32_t neg = (t >> 3) & 0x11111111u;   // 1 in the low bit of each negative nibble
  const uint32_t mag = ((t ^ (neg * 15u)) + neg) & 0x77777777u;
  return mag | (__builtin_amdgcn_alignbit(t, t, 28) & 0x88888888u);
}

}  // namespace qwam

namespace qwam {

// Raw buffer resource over [base, base + bytes): loads whose byte offset falls
// outside the range return zero (no fault), so ragged tiles and prefetches past
// the last group need no branches.  Offsets are 32-bit.
typedef __amdgpu_buffer_rsrc_t buf_rsrc;

__device__ __forceinline__ buf_rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                           0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(buf_rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ uint2 buf_load8(buf_rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

__device__ __forceinline__ float buf_load4f(buf_rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

}  // namespace qwam

namespace qwam {

typedef __attribute__((address_space(3))) void lds_void;

// Direct global -> LDS copy of 16 bytes per lane (buffer_load_dwordx4 ... lds):
// lane i's bytes land at lds_base + 16 * i.  lds_base must be wave-uniform.
// Out-of-range offsets deposit zeros.  Completion is tracked by vmcnt.
__device__ __forceinline__ void buf_load16_lds(buf_rsrc r, uint32_t off, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_base, 16, off, 0, 0, 0);
}

// Same with 4 bytes per lane (lane i -> lds_base + 4 * i).
__device__ __forceinline__ void buf_load4_lds(buf_rsrc r, uint32_t off, void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds_base, 4, off, 0, 0, 0);
}

// Workgroup barrier without the implicit full memory fence of __syncthreads()
// (which would drain every outstanding copy of the LDS ring).  Callers make
// their own data visible first: wait_vmcnt for their LDS copies, and LDS
// stores / loads are ordered by the barrier itself.  The "memory" clobber keeps
// the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt with only the vector-memory counter constrained (vmcnt <= n).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

}  // namespace qwam

namespace qwam {

typedef unsigned int v2u_t __attribute__((ext_vector_type(2)));

// Buffer stores: bytes whose offset falls outside the resource are dropped.
__device__ __forceinline__ void buf_store8(uint2 v, buf_rsrc r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u_t, v), r, off, 0, 0);
}

__device__ __forceinline__ void buf_store4f(float v, buf_rsrc r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), r, off, 0, 0);
}

}  // namespace qwam
