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

// Code blocks, the storage format of every 4-bit code (qwam.h).  The codes
// c[k0 .. k0+15] of 16 consecutive channels (k0 a multiple of 16) are written
// as 6-bit fields F_i = s << 5 | |c[k0+i]| (the FP6 e2m3 pattern of c / 8; s
// is the sign of the scaled value x = v * inv, so a zero code may carry
// either sign), field i at bits 6i .. 6i+5 of a 96-bit stream
// D0 | D1 << 32 | D2 << 64.  Bits 3-4 of every field are zero; in D0 and D1
// those positions (kFp6Z0, kFp6Z1) together are exactly the data bits of D2,
// which is stored there: word 0 = D0 | (D2 & kFp6Z0), word 1 = D1 | (D2 &
// kFp6Z1).  A reader gets the MFMA operand back with four ANDs (qwam_mfma.h).
// The quantizer never yields -8 (|x| <= 7 (1 + 3u) < 7.5).
constexpr uint32_t kFp6Z0 = 0x18618618u;   // bits 3-4 of the fields in D0
constexpr uint32_t kFp6Z1 = 0x86186186u;   // bits 3-4 of the fields in D1

typedef unsigned v6u __attribute__((ext_vector_type(6)));
typedef float v16f __attribute__((ext_vector_type(16)));

// The codes of 32 scaled values x[0..31] (Eq. 2: rint, ties to even, of x;
// |x| < 7.5) as the FP6 e2m3 stream, field i = x[i], in one instruction:
// v_cvt_scalef32_2xpk16_fp6_f32 writes a[i] to field 2i and b[i] to field
// 2i + 1 of x / scale, rounded to nearest even, with the sign of x.  On
// gfx950 this equals (signbit(x) << 5) | |rint(x)| for every float (checked
// against rint, halfway cases, signed zeros and denormals included).
__device__ __forceinline__ v6u codes_fp6_32(const float (&x)[32]) {
  v16f a, b;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    a[i] = x[2 * i];
    b[i] = x[2 * i + 1];
  }
  return __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(a, b, 8.0f);
}

// The same for 16 values (stream words D0, D1, D2).
__device__ __forceinline__ void codes_fp6_16(const float (&x)[16], uint32_t& d0, uint32_t& d1, uint32_t& d2) {
  v16f a = {}, b = {};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = x[2 * i];
    b[i] = x[2 * i + 1];
  }
  const v6u r = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(a, b, 8.0f);
  d0 = r[0];
  d1 = r[1];
  d2 = r[2];
}

// stream words -> the two stored words of a code block
__device__ __forceinline__ uint2 fp6_code_block(uint32_t d0, uint32_t d1, uint32_t d2) {
  return make_uint2(d0 | (d2 & kFp6Z0), d1 | (d2 & kFp6Z1));
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

namespace qwam {

// max(v, v of lane l ^ 16) and max(v, v of lane l ^ 32) for every lane l, by
// gfx950's row / half swaps (each lane gets its own and its partner's value
// back, in one order or the other) instead of a ds_bpermute
__device__ __forceinline__ float max_xor16(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

}  // namespace qwam
