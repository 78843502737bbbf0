// Matrix-core helpers shared by the ASP GEMM kernels (gfx950): the FP6 view
// of packed code blocks, the exact integer partial of one group on
// v_mfma_scale_f32_32x32x64_f8f6f4, and the per-group float32 scaling of a
// 32 x 32 result block with the row scales broadcast by DPP.
#pragma once
#include <utility>

#include "qwam_device.h"

namespace qwam {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v32f __attribute__((ext_vector_type(32)));
typedef int v8i __attribute__((ext_vector_type(8)));

// 32 packed codes (16 bytes of one row: two code blocks, qwam_device.h) ->
// one FP6 e2m3 MFMA operand: field i of the 192-bit operand (dwords 0-5) is
// the code of channel i of the 32, value code / 8.  Four ANDs per block.
__device__ __forceinline__ v8i codes_to_fp6(const uint4& p) {
  const v4i lo = {static_cast<int>(p.x & ~kFp6Z0), static_cast<int>(p.y & ~kFp6Z1),
                  static_cast<int>((p.x & kFp6Z0) | (p.y & kFp6Z1)), 0};
  const v4i hi = {static_cast<int>(p.z & ~kFp6Z0), static_cast<int>(p.w & ~kFp6Z1),
                  static_cast<int>((p.z & kFp6Z0) | (p.w & kFp6Z1)), 0};
  // words 6-7 are not read with FP6 operands (left undefined)
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 4, 5, 6, -1, -1);
}

// operand format of v_mfma_scale_f32_32x32x64_f8f6f4 (cbsz / blgp): FP6 e2m3
constexpr int kFmtFp6 = 2;
// E8M0 scale 2^3 (127 + 3) for both operands: (code / 8 * 2^3) products are
// the integer products; each lane's scale governs its own 32 values
constexpr int kE8M0Code = 127 + 3;

// exact integer partial of a 32 x 32 block over 32 + 32 channels: lane l holds
// row / column l % 32 and channels 32 * (l / 32) .. +31 of the span; sa and sb
// are the lane's E8M0 scales (kE8M0Code, or 0 to mask its channels: with 2^-127
// on both operands the products underflow to zero)
__device__ __forceinline__ v16f fp6_partial(const v8i& a, const v8i& b, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, v16f{}, kFmtFp6, kFmtFp6, 0, sa, 0, sb);
}

// x of lane 16 * (lane / 16) + V (lane V of this lane's row of 16, DPP
// row_newbcast) times y, in one instruction.  The DPP source x must not be
// written by a VALU instruction in the two instructions before (the callers'
// x always comes straight from a memory load).
template <int V>
__device__ __forceinline__ float row_bcast_mul(float x, float y) {
  float r;
  asm("v_mul_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf bound_ctrl:1"
      : "=v"(r)
      : "v"(x), "v"(y), "i"(V));
  return r;
}

// acc[v] += p[v] * (sx of result row v of this lane) * sw, v = 0..15, where
// lane 16 * rho + v holds the activation scale that result register v of the
// lanes in row rho of 16 needs.  All 16 products first, then the 16 updates, so
// that no update directly follows the product it reads.
template <int... V>
__device__ __forceinline__ void scale_accumulate(std::integer_sequence<int, V...>, v16f& acc, const v16f& p,
                                                 float sx_lane, float sw) {
  float s[sizeof...(V)];
  ((s[V] = row_bcast_mul<V>(sx_lane, sw)), ...);
  ((acc[V] = __builtin_fmaf(p[V], s[V], acc[V])), ...);
}

}  // namespace qwam
