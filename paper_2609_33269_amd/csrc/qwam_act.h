// Per-group steps of the activation kernels (plain, deflated, rotated), in
// one lane layout: a wave holds one group of 64 channels of 16 tokens, lane l
// holding token l % 16 and the 16 consecutive channels 16*(l/16) .. +15, so
// the four lanes l, l^16, l^32, l^48 hold one token's group.  That is the
// A-operand layout of v_mfma_f32_16x16x32_bf16 (row = token, k slots of lane
// l shared with lane l of the B operand) and, with one k slot per lane group,
// of v_mfma_f64_16x16x4_f64.
#pragma once
#include "qwam_device.h"

namespace qwam {

typedef double v4d __attribute__((ext_vector_type(4)));
typedef float v16f_t __attribute__((ext_vector_type(16)));

typedef unsigned int v4u_act __attribute__((ext_vector_type(4)));

// 16-byte buffer store (bytes outside the resource are dropped)
__device__ __forceinline__ void buf_store16(uint4 v, buf_rsrc r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u_act, v), r, off, 0, 0);
}

template <int RANK>
struct ActFetch {
  uint4 xa, xb;                 // 16 bf16 of x
  v8s l1[RANK / 16][2];         // L1t fragments: 16 channels of 16 columns of t
};

// Waves per workgroup: 16 (4 per SIMD) up to rank 32, 8 above (more registers
// for the larger L1t prefetch).
template <int RANK>
constexpr int act_waves() { return RANK <= 32 ? 16 : 8; }

// x~ = fl32(x * fl32(1/lambda)) for the lane's 16 channels (xa, xb: 16 bf16 of
// x; ip: the matching 16 entries of 1/lambda).
__device__ __forceinline__ void smooth16(const uint4& xa, const uint4& xb, const float4* ip, float (&v)[16]) {
  const uint32_t xw[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
  const float4 i0 = ip[0], i1 = ip[1], i2 = ip[2], i3 = ip[3];
  const float iv[16] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w,
                        i2.x, i2.y, i2.z, i2.w, i3.x, i3.y, i3.z, i3.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[2 * j] = __uint_as_float(xw[j] << 16) * iv[2 * j];
    v[2 * j + 1] = __uint_as_float(xw[j] & 0xFFFF0000u) * iv[2 * j + 1];
  }
}

// The same with the 16 entries of 1/lambda already in registers.
__device__ __forceinline__ void smooth16_regs(const uint4& xa, const uint4& xb, const float4 (&iv4)[4], float (&v)[16]) {
  const uint32_t xw[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
  const float iv[16] = {iv4[0].x, iv4[0].y, iv4[0].z, iv4[0].w, iv4[1].x, iv4[1].y, iv4[1].z, iv4[1].w,
                        iv4[2].x, iv4[2].y, iv4[2].z, iv4[2].w, iv4[3].x, iv4[3].y, iv4[3].z, iv4[3].w};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[2 * j] = __uint_as_float(xw[j] << 16) * iv[2 * j];
    v[2 * j + 1] = __uint_as_float(xw[j] & 0xFFFF0000u) * iv[2 * j + 1];
  }
}

// Quantizes the lane's token over one 64-channel span (Eq. 2): with group 64
// the four lanes l, l^16, l^32, l^48 (16 consecutive channels each) share one
// scale; with group 32 (g32) the lanes l, l^16 share the scale of channels
// 0-31 or 32-63 of the span.  Returns the lane's code block (8 bytes) and its
// group scale.
__device__ __forceinline__ uint2 quantize_block(const float (&v)[16], bool g32, float& scale) {
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[j]));
  amax = max_xor16(amax);
  if (!g32) amax = max_xor32(amax);
  const float s = q4_scale(amax);
  const float inv = q4_inv(s);
  // codes rint(v * inv) of the lane's 16 channels: one code block
  float x[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) x[j] = v[j] * inv;
  uint32_t d0, d1, d2;
  codes_fp6_16(x, d0, d1, d2);
  scale = s;
  return fp6_code_block(d0, d1, d2);
}

// The same, storing the lane's code block (8 bytes) at byte q_off of q_rsrc
// and, if xs_dst is not null, the lane's group scale.
__device__ __forceinline__ void quantize_pack_store(const float (&v)[16], buf_rsrc q_rsrc, uint32_t q_off,
                                                    float* xs_dst, bool g32 = false) {
  float s;
  buf_store8(quantize_block(v, g32, s), q_rsrc, q_off);
  if (xs_dst != nullptr) *xs_dst = s;
}

// Where the lane of token `row` (chunk = lane / 16) stores the scale of the
// 64-channel span g: xs is [K / group][M]; null for tokens past M.
__device__ __forceinline__ float* xs_slot(float* xs, int g, int M, int m0, int row, int rows, int chunk, bool g32) {
  if (row >= rows) return nullptr;
  const int gi = g32 ? 2 * g + (chunk >> 1) : g;
  return xs + static_cast<int64_t>(gi) * M + m0 + row;
}

template <int RANK>
struct DeflFetch {
  uint4 xa, xb;                 // 16 bf16 of x
  uint32_t l1[RANK / 2];        // L1[a_ch][j], two bf16 per word (j even in the low half)
};

// L1 fragments of the lane's 16 channels of 64-channel span g for the RB
// blocks of 16 columns of t: L1[64 g + 16 (l/16) + 8 h + e][16 rb + l%16],
// e = 0..7, h = 0, 1.  L1f holds them in exactly this order
// ([K/64][RB][2][64 lanes][8]), so each of the wave's 2 RB loads reads one
// contiguous kilobyte.
template <int RB>
__device__ __forceinline__ void load_l1_fragments(const uint16_t* __restrict__ L1f, int g, int lane,
                                                  v8s (&l1)[RB][2]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      l1[rb][h] = *reinterpret_cast<const v8s*>(L1f + (static_cast<int64_t>((g * RB + rb) * 2 + h) * 64 + lane) * 8);
}

// t partial on the bf16 matrix cores: A = bf16(x~) of the lane's token and
// channels, B = the matching L1t fragments; two k-steps of 32 per group.
template <int RB>
__device__ __forceinline__ void t_step_bf16(const float (&v)[16], const v8s (&l1)[RB][2], v4f (&acc)[RB]) {
  typedef __bf16 v8b __attribute__((ext_vector_type(8)));
  v8b a_lo, a_hi;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a_lo[j] = static_cast<__bf16>(v[j]);
    a_hi[j] = static_cast<__bf16>(v[8 + j]);
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_lo, __builtin_bit_cast(v8bf, l1[rb][0]), acc[rb], 0, 0, 0);
    acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_hi, __builtin_bit_cast(v8bf, l1[rb][1]), acc[rb], 0, 0, 0);
  }
}

// t partial in double on the FP64 matrix cores: A lane l = token l%16, k-slot
// l/16 -> channel 16*(l/16) + s at step s; B lane l = column l%16 of block rb,
// same k-slot.  Products of two bf16 values are exact in double.
template <int RB>
__device__ __forceinline__ void t_step_f64(const float (&v)[16], const v8s (&l1)[RB][2], v4d (&acc)[RB]) {
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    const double a = static_cast<double>(static_cast<float>(static_cast<__bf16>(v[s])));
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const uint32_t lb = static_cast<uint16_t>(l1[rb][s >> 3][s & 7]);
      acc[rb] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, static_cast<double>(bf16_to_f32(lb)), acc[rb], 0, 0, 0);
    }
  }
}

// Deflation column of L1 for A-operand lane l of v_mfma_f32_16x16x1_4b_f32:
// lane 16B + 4Q + I supplies channel 16Q + 4B + I of the group, which lands in
// result register 4B + I of the lanes with l/16 = Q (token l%16), i.e. the
// layout above.  Two bf16 per word, j even in the low half.
__device__ __forceinline__ int deflate_channel(int lane) {
  return 16 * ((lane >> 2) & 3) + 4 * (lane >> 4) + (lane & 3);
}

// The lane's row L1[ch][0 .. RANK-1] of L1 ([K][RANK] bf16, 16-byte aligned):
// RANK/8 loads of 16 contiguous bytes; word j/2 holds columns j (low half)
// and j+1.
template <int RANK>
__device__ __forceinline__ void load_l1_row(const uint16_t* __restrict__ L1, int ch, uint32_t (&l1w)[RANK / 2]) {
  const uint4* lp = reinterpret_cast<const uint4*>(L1 + static_cast<int64_t>(ch) * RANK);
#pragma unroll
  for (int i = 0; i < RANK / 8; ++i) {
    const uint4 w = lp[i];
    l1w[4 * i] = w.x;
    l1w[4 * i + 1] = w.y;
    l1w[4 * i + 2] = w.z;
    l1w[4 * i + 3] = w.w;
  }
}

// x~_perp = x~ - L1 t: r rank-1 updates on the FP32 matrix cores, K = 1 each,
// j ascending; each step adds L1[:, j] * (-t_j), an exact product, with one
// rounding.  tn_row: -t of the lane's token (float, RANK entries, LDS).
template <int RANK>
__device__ __forceinline__ void deflate_step(float (&v)[16], const uint32_t (&l1w)[RANK / 2], const float* tn_row) {
  v16f_t c;
#pragma unroll
  for (int i = 0; i < 16; ++i) c[i] = v[i];
#pragma unroll
  for (int j = 0; j < RANK; j += 4) {
    const float4 tv = *reinterpret_cast<const float4*>(tn_row + j);
    c = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(l1w[j / 2] << 16), tv.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(l1w[j / 2] & 0xFFFF0000u), tv.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(l1w[j / 2 + 1] << 16), tv.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(l1w[j / 2 + 1] & 0xFFFF0000u), tv.w, c, 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = c[i];
}

// Partial t tiles -> LDS [wave][16][RANK].  bf16 MFMA: register i of lane l is
// token 4*(l/16) + i; f64 MFMA: token l/16 + 4 i; column l%16 of block rb.
template <int RB>
__device__ __forceinline__ void store_t_partials(float* red, int wave, int lane, const v4f (&acc)[RB]) {
  constexpr int RANK = RB * 16;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      red[(wave * 16 + 4 * (lane >> 4) + i) * RANK + rb * 16 + (lane & 15)] = acc[rb][i];
}

template <int RB>
__device__ __forceinline__ void store_t_partials(double* red, int wave, int lane, const v4d (&acc)[RB]) {
  constexpr int RANK = RB * 16;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      red[(wave * 16 + (lane >> 4) + 4 * i) * RANK + rb * 16 + (lane & 15)] = acc[rb][i];
}

// Sums the partial tiles in wave order and writes bf16 t (tokens < rows);
// with tneg != nullptr also -t as float into LDS [16][RANK].  Float partials
// are summed in float and rounded once; double partials in double, then
// rounded once to bf16 (f64_to_bf16_rne).  Call between two barriers.
template <int RANK, typename T>
__device__ __forceinline__ void reduce_t(const T* red, int nwaves, int rows, uint16_t* __restrict__ t_rows,
                                         float* tneg) {
  for (int e = threadIdx.x; e < 16 * RANK; e += blockDim.x) {
    const int i = e / RANK, j = e % RANK;
    T sum = 0;
    for (int w = 0; w < nwaves; ++w) sum += red[(w * 16 + i) * RANK + j];
    uint32_t b;
    if constexpr (sizeof(T) == 8) b = f64_to_bf16_rne(sum);
    else b = f32_to_bf16_rne(sum);
    if (i < rows) t_rows[static_cast<int64_t>(i) * RANK + j] = static_cast<uint16_t>(b);
    if (tneg != nullptr) tneg[i * RANK + j] = -bf16_to_f32(b);
  }
}

}  // namespace qwam
