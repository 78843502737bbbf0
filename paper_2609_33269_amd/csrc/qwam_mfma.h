// Matrix-core helpers shared by the ASP GEMM kernels (gfx950): the FP8 view
// of packed code words, the exact integer partial of one group on
// v_mfma_scale_f32_32x32x64_f8f6f4, and the per-group float32 scaling of a
// 32 x 32 result block with the row scales broadcast by DPP.
#pragma once
#include <utility>

#include "qwam_device.h"

namespace qwam {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v32f __attribute__((ext_vector_type(32)));
typedef int v8i __attribute__((ext_vector_type(8)));

// 32 packed codes (16 bytes of one row) -> one FP8 MFMA operand of 32 e4m3
// bytes, ordered [even k of w0, odd k of w0, even k of w1, ...] (the same
// permutation for A and B, so the dot product is unchanged).
__device__ __forceinline__ v8i codes_to_e4m3(const uint4& p) {
  const uint32_t w[4] = {p.x, p.y, p.z, p.w};
  v8i r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    r[2 * d] = static_cast<int>(w[d] & 0x87878787u);
    r[2 * d + 1] = static_cast<int>(__builtin_amdgcn_alignbit(w[d], w[d], 4) & 0x87878787u);
  }
  return r;
}

// E8M0 scale 2^9 (127 + 9) for both operands: (code * 2^-9 * 2^9) products
constexpr int kE8M0Code = 127 + 9;

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
