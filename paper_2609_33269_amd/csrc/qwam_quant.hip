// Weight pack (offline) and the fused activation kernel of the ASP layer.
//
//  pack:  R [N][K] f32 -> wq [N][K/2] packed codes, ws [G][N] scales (Eq. 2, App. B.1)
//  act:   x [M][K] bf16 -> x~ = x * (1/lambda) (Eq. 3), per-token group-64
//         codes xq [M][K/2] and scales xs [G][M] (Eq. 2), and the rank-r
//         down-projection t = bf16(x~) . L1 on bf16 matrix cores (V^T x~ of
//         Eq. 9), all in one pass over x.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

// ---------------------------------------------------------------------------
// Weight pack: 16 lanes per (row, group); each lane owns 4 consecutive floats.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_weights_kernel(const float* __restrict__ R,
                                                           uint8_t* __restrict__ wq,
                                                           float* __restrict__ ws, int N, int K) {
  const int G = K / kGroup;
  const int64_t team = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 4;
  const int sub = threadIdx.x & 15;
  const bool active = team < static_cast<int64_t>(N) * G;
  const int n = active ? static_cast<int>(team / G) : 0;
  const int g = active ? static_cast<int>(team % G) : 0;

  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (active) v = *reinterpret_cast<const float4*>(R + static_cast<int64_t>(n) * K + g * kGroup + sub * 4);
  float amax = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(v.x), __builtin_fabsf(v.y)),
                               __builtin_fmaxf(__builtin_fabsf(v.z), __builtin_fabsf(v.w)));
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, o));
  const float s = q4_scale(amax);
  const float inv = q4_inv(s);
  const uint32_t c = q4_nibble(v.x, inv) | (q4_nibble(v.y, inv) << 4) | (q4_nibble(v.z, inv) << 8) |
                     (q4_nibble(v.w, inv) << 12);
  if (active) {
    *reinterpret_cast<uint16_t*>(wq + static_cast<int64_t>(n) * (K / 2) + g * (kGroup / 2) + sub * 2) =
        static_cast<uint16_t>(c);
    if (sub == 0) ws[static_cast<int64_t>(g) * N + n] = s;
  }
}

__global__ __launch_bounds__(256) void inverse_smoothing_kernel(const float* __restrict__ smooth,
                                                                float* __restrict__ inv, int K) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < K) inv[k] = 1.0f / smooth[k];
}

// ---------------------------------------------------------------------------
// Fused activation kernel.
//
// A workgroup owns 16 tokens and all of K; its waves split the K groups into
// contiguous ranges.  In a wave, lane l handles token (l % 16) and the 16
// consecutive channels 16*(l/16) .. +15 of the current group, so the 4 lanes
// l, l^16, l^32, l^48 together hold one token's group of 64.  That is also the
// A-operand layout of v_mfma_f32_16x16x32_bf16 (row = l % 16, the k slots of
// lane l shared with lane l of the B operand), so the smoothed values feed the
// down-projection directly from registers: two MFMA steps of 32 channels per
// group and 16 columns of t.  The per-wave partial t tiles are summed in LDS
// in wave order (deterministic) and rounded to bf16 once.
// ---------------------------------------------------------------------------
template <int RANK>
__global__ __launch_bounds__(1024) void quantize_act_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth,
    const uint16_t* __restrict__ L1t, uint8_t* __restrict__ xq, float* __restrict__ xs,
    uint16_t* __restrict__ t, int M, int K, int groups_per_wave) {
  constexpr int RB = RANK / 16;
  extern __shared__ float red[];  // [nwaves][16][RANK]

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int row = lane & 15;
  const int chunk = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int m = m0 + row;
  const bool valid = m < M;
  const int G = K / kGroup;
  const int g_begin = wave * groups_per_wave;
  const int g_end = min(G, g_begin + groups_per_wave);

  v4f acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = v4f{0.f, 0.f, 0.f, 0.f};

  const uint16_t* xrow = x + static_cast<int64_t>(valid ? m : 0) * K;

  for (int g = g_begin; g < g_end; ++g) {
    const int k0 = g * kGroup + chunk * 16;
    uint4 xa = make_uint4(0, 0, 0, 0), xb = make_uint4(0, 0, 0, 0);
    if (valid) {
      xa = *reinterpret_cast<const uint4*>(xrow + k0);
      xb = *reinterpret_cast<const uint4*>(xrow + k0 + 8);
    }
    const float4* ip = reinterpret_cast<const float4*>(inv_smooth + k0);
    const float4 i0 = ip[0], i1 = ip[1], i2 = ip[2], i3 = ip[3];
    const uint32_t xw[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
    const float iv[16] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w,
                          i2.x, i2.y, i2.z, i2.w, i3.x, i3.y, i3.z, i3.w};
    float v[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[2 * j] = bf16_to_f32(xw[j] & 0xFFFFu) * iv[2 * j];
      v[2 * j + 1] = bf16_to_f32(xw[j] >> 16) * iv[2 * j + 1];
    }
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[j]));
    amax = __builtin_fmaxf(amax, __shfl_xor(amax, 16));
    amax = __builtin_fmaxf(amax, __shfl_xor(amax, 32));
    const float s = q4_scale(amax);
    const float inv = q4_inv(s);
    uint32_t packed[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t wv = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) wv |= q4_nibble(v[8 * h + j], inv) << (4 * j);
      packed[h] = wv;
    }
    if (valid) {
      *reinterpret_cast<uint2*>(xq + static_cast<int64_t>(m) * (K / 2) + g * (kGroup / 2) + chunk * 8) =
          make_uint2(packed[0], packed[1]);
      if (chunk == 0) xs[static_cast<int64_t>(g) * M + m] = s;
    }

    // down-projection: A = bf16(x~) of this token, B = L1t rows (columns of t)
    v8s a_lo, a_hi;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      a_lo[j] = static_cast<short>(f32_to_bf16_rne(v[j]));
      a_hi[j] = static_cast<short>(f32_to_bf16_rne(v[8 + j]));
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const uint16_t* lp = L1t + static_cast<int64_t>(rb * 16 + row) * K + k0;
      const v8s b_lo = *reinterpret_cast<const v8s*>(lp);
      const v8s b_hi = *reinterpret_cast<const v8s*>(lp + 8);
      acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a_lo),
                                                        __builtin_bit_cast(v8bf, b_lo), acc[rb], 0, 0, 0);
      acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a_hi),
                                                        __builtin_bit_cast(v8bf, b_hi), acc[rb], 0, 0, 0);
    }
  }

  // partial t tiles -> LDS: result row 4*(l/16)+i, column l%16 of block rb
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      red[(wave * 16 + 4 * chunk + i) * RANK + rb * 16 + row] = acc[rb][i];
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * RANK; e += blockDim.x) {
    const int i = e / RANK, j = e % RANK;
    float sum = 0.0f;
    for (int w = 0; w < nwaves; ++w) sum += red[(w * 16 + i) * RANK + j];
    if (m0 + i < M) t[static_cast<int64_t>(m0 + i) * RANK + j] = static_cast<uint16_t>(f32_to_bf16_rne(sum));
  }
}

// ---------------------------------------------------------------------------
hipError_t launch_pack_weights(int K, int N, const float* R, const float* smooth, uint8_t* wq,
                               float* ws, float* inv_smooth, hipStream_t stream) {
  const int64_t teams = static_cast<int64_t>(N) * (K / kGroup);
  const int64_t blocks = (teams * 16 + 255) / 256;
  hipLaunchKernelGGL(pack_weights_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, R,
                     wq, ws, N, K);
  hipLaunchKernelGGL(inverse_smoothing_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, smooth,
                     inv_smooth, K);
  return hipGetLastError();
}

hipError_t launch_quantize_act(int M, int K, int r, const uint16_t* x, const float* inv_smooth,
                               const uint16_t* L1t, uint8_t* xq, float* xs, uint16_t* t,
                               hipStream_t stream) {
  const int G = K / kGroup;
  const int nwaves = G < 16 ? G : 16;
  const int gpw = (G + nwaves - 1) / nwaves;
  const dim3 grid((M + 15) / 16), block(64 * nwaves);
  const size_t lds = static_cast<size_t>(nwaves) * 16 * r * sizeof(float);
  switch (r) {
    case 16:
      hipLaunchKernelGGL(quantize_act_kernel<16>, grid, block, lds, stream, x, inv_smooth, L1t, xq, xs, t, M, K, gpw);
      break;
    case 32:
      hipLaunchKernelGGL(quantize_act_kernel<32>, grid, block, lds, stream, x, inv_smooth, L1t, xq, xs, t, M, K, gpw);
      break;
    case 48:
      hipLaunchKernelGGL(quantize_act_kernel<48>, grid, block, lds, stream, x, inv_smooth, L1t, xq, xs, t, M, K, gpw);
      break;
    case 64:
      hipLaunchKernelGGL(quantize_act_kernel<64>, grid, block, lds, stream, x, inv_smooth, L1t, xq, xs, t, M, K, gpw);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace qwam
