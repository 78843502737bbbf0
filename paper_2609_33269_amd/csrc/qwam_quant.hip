// Weight pack (offline) and the fused activation kernel of the ASP layer.
//
//  pack:  R [N][K] f32 -> wq [N][K/2] packed codes, ws [G][N] scales (Eq. 2, App. B.1),
//         and each scale as two bf16 pieces for the GEMM's scale products
//  act:   x [M][K] bf16 -> x~ = x * (1/lambda) (Eq. 3), per-token group-64
//         codes xq [M][K/2] and scales xs [G][M] (Eq. 2), and the rank-r
//         down-projection t = bf16(x~) . L1 on bf16 matrix cores (V^T x~ of
//         Eq. 9), all in one pass over x.
#include "qwam_act.h"
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

// ---------------------------------------------------------------------------
// Weight pack: 4 lanes per (row, 64-channel span); each lane owns 16
// consecutive floats, i.e. one code block.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_weights_kernel(const float* __restrict__ R,
                                                           uint8_t* __restrict__ wq,
                                                           float* __restrict__ ws, uint32_t* __restrict__ wsp,
                                                           int N, int K, int g32) {
  const int G = K / kGroup;
  const int64_t team = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) >> 2;
  const int sub = threadIdx.x & 3;
  const bool active = team < static_cast<int64_t>(N) * G;
  const int n = active ? static_cast<int>(team / G) : 0;
  const int g = active ? static_cast<int>(team % G) : 0;

  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = 0.0f;
  if (active) {
    const float4* src = reinterpret_cast<const float4*>(R + static_cast<int64_t>(n) * K + g * kGroup + sub * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 a = src[i];
      v[4 * i] = a.x; v[4 * i + 1] = a.y; v[4 * i + 2] = a.z; v[4 * i + 3] = a.w;
    }
  }
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
  // the 4 lanes of a 64-channel span; with group 32 lanes 0-1 and 2-3 separately
  amax = __builtin_fmaxf(amax, __shfl_xor(amax, 1));
  if (!g32) amax = __builtin_fmaxf(amax, __shfl_xor(amax, 2));
  const float s = q4_scale(amax);
  const float inv = q4_inv(s);
  float x[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = v[i] * inv;
  uint32_t d0, d1, d2;
  codes_fp6_16(x, d0, d1, d2);
  if (active) {
    *reinterpret_cast<uint2*>(wq + static_cast<int64_t>(n) * (K / 2) + g * (kGroup / 2) + sub * 8) =
        fp6_code_block(d0, d1, d2);
    if (g32 ? (sub & 1) == 0 : sub == 0) {
      const int64_t at = static_cast<int64_t>(g32 ? 2 * g + (sub >> 1) : g) * N + n;
      ws[at] = s;
      // hi = bf16(s), lo = bf16(s - hi): s - hi is exact in float32
      const uint32_t hi = f32_to_bf16_rne(s);
      wsp[at] = hi | (f32_to_bf16_rne(s - bf16_to_f32(hi)) << 16);
    }
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
// contiguous ranges, in the lane layout of qwam_act.h (lane l: token l % 16,
// channels 16*(l/16) .. +15 of the current group), so the smoothed values feed
// the down-projection on the bf16 matrix cores straight from registers.  Each
// wave prefetches the next group (x, L1 fragments) while it quantizes the current one;
// x is read with buffer loads and the codes / scales are written with buffer
// stores, so rows past M need no branches.  From K = 4096 on, a wave's code
// blocks of four consecutive groups (one 128-byte line of each of its 16 rows)
// are gathered in a 2 KB LDS line buffer of its own and written out as whole
// lines, 16 bytes per lane and 8 lines per instruction, instead of 32-byte
// pieces of 16 lines per group (the wave ranges are then whole line chunks);
// below, the 16 waves keep their ranges and store each group's blocks.  The
// per-wave partial t tiles are summed in LDS in wave order (deterministic) and
// rounded to bf16 once.
// ---------------------------------------------------------------------------
template <int RANK, bool INV_LDS>
__global__ __launch_bounds__(64 * act_waves<RANK>()) void quantize_act_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth,
    const uint16_t* __restrict__ L1f, uint8_t* __restrict__ xq, float* __restrict__ xs,
    uint16_t* __restrict__ t, int M, int K, int groups_per_wave, int g32) {
  constexpr int RB = RANK / 16;
  // dynamic LDS: [nwaves][16][RANK] partial t, then (INV_LDS) [nwaves][groups_per_wave * 64] 1/lambda,
  // then [nwaves][16 rows][128 bytes] code lines
  extern __shared__ float red[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int row = lane & 15;
  const int chunk = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int rows = min(16, M - m0);
  const int G = K / kGroup;
  const int g_begin = wave * groups_per_wave;
  const int g_end = min(G, g_begin + groups_per_wave);

  // the workgroup's 16 rows of x, xq; out-of-range rows read as zero / are dropped
  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<uint32_t>(rows) * K * 2u);
  const buf_rsrc q_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * (K / 2), static_cast<uint32_t>(rows) * (K / 2));
  const uint32_t x_off = static_cast<uint32_t>(row * K + chunk * 16) * 2u;
  const uint32_t q_off = static_cast<uint32_t>(row * (K / 2) + chunk * 8);

  // the wave's slice of 1/lambda goes to LDS once (a per-group float4 load by
  // every lane would move 16x more bytes through the address unit than it uses)
  float* inv_w = red + nwaves * 16 * RANK + wave * groups_per_wave * kGroup;
  if (INV_LDS && g_begin < g_end) {
    const int n4 = (g_end - g_begin) * (kGroup / 4);
    const float4* src = reinterpret_cast<const float4*>(inv_smooth + g_begin * kGroup);
    for (int i = lane; i < n4; i += 64) reinterpret_cast<float4*>(inv_w)[i] = src[i];
  }

  auto fetch = [&](int g, ActFetch<RANK>& f) __attribute__((always_inline)) {
    const uint32_t go = static_cast<uint32_t>(g) * kGroup * 2u;
    f.xa = buf_load16(x_rsrc, x_off + go);
    f.xb = buf_load16(x_rsrc, x_off + go + 16u);
    load_l1_fragments<RB>(L1f, g, lane, f.l1);
  };

  v4f acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = v4f{0.f, 0.f, 0.f, 0.f};

  uint8_t* line = reinterpret_cast<uint8_t*>(red + nwaves * 16 * RANK + (INV_LDS ? nwaves * groups_per_wave * kGroup : 0)) +
                  wave * 2048;
  // the launcher gives whole line chunks per wave from 64 groups on
  const bool lines = groups_per_wave % 4 == 0;
  // writes the staged blocks of groups max(g_begin, g & ~3) .. g (one line
  // chunk): lane l takes row 8h + l/8 and the 16-byte piece l%8 of its line
  auto flush = [&](int g) __attribute__((always_inline)) {
    const int q0 = g & ~3;
    const int p_lo = 2 * (max(g_begin, q0) - q0), p_hi = 2 * (g - q0 + 1);
    const int piece = lane & 7;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = 8 * h + (lane >> 3);
      if (piece >= p_lo && piece < p_hi) {
        const uint4 d = *reinterpret_cast<const uint4*>(line + r * 128 + piece * 16);
        buf_store16(d, q_rsrc, static_cast<uint32_t>(r * (K / 2) + q0 * (kGroup / 2) + piece * 16));
      }
    }
  };

  auto work = [&](int g, const ActFetch<RANK>& f) __attribute__((always_inline)) {
    const float4* ip = INV_LDS ? reinterpret_cast<const float4*>(inv_w + (g - g_begin) * kGroup + chunk * 16)
                               : reinterpret_cast<const float4*>(inv_smooth + g * kGroup + chunk * 16);
    float v[16];
    smooth16(f.xa, f.xb, ip, v);
    float s;
    const uint2 blk = quantize_block(v, g32, s);
    // the block goes to the row's line at its group's 32-byte slot (or, when
    // the wave's range is not made of line chunks, straight out); every lane
    // of a row (of a 32-channel half with group 32) holds the same scale and
    // writes it at the row's slot (letting one lane of each write it instead
    // measured 2-3 us slower at K = 3072)
    if (lines) *reinterpret_cast<uint2*>(line + row * 128 + (g & 3) * 32 + chunk * 8) = blk;
    else buf_store8(blk, q_rsrc, q_off + static_cast<uint32_t>(g) * (kGroup / 2));
    if (float* p = xs_slot(xs, g, M, m0, row, rows, chunk, g32)) *p = s;
    t_step_bf16<RB>(v, f.l1, acc);
    if (lines && ((g & 3) == 3 || g == g_end - 1)) flush(g);
  };

  // software pipeline, two groups per trip so the fetch registers are named statically;
  // the prefetch past the wave's last group re-reads that group (harmless, in bounds)
  if (g_begin < g_end) {
    ActFetch<RANK> fa, fb;
    fetch(g_begin, fa);
    int g = g_begin;
    for (; g + 1 < g_end; g += 2) {
      fetch(g + 1, fb);
      work(g, fa);
      fetch(min(g + 2, g_end - 1), fa);
      work(g + 1, fb);
    }
    if (g < g_end) work(g, fa);
  }

  store_t_partials<RB>(red, wave, lane, acc);
  __syncthreads();
  reduce_t<RANK>(red, nwaves, rows, t + static_cast<int64_t>(m0) * RANK, static_cast<float*>(nullptr));
}

// ---------------------------------------------------------------------------
// Deflated activation kernel: the 4-bit path quantizes x~_perp = x~ - L1 t
// (Eq. 8 / Eq. 9) instead of x~.  Deflation needs t before any token of the
// workgroup is quantized, and it needs t's exact bits (every code depends on
// them), so the workgroup of 16 tokens runs two phases:
//
//  1. t = bf16(sum_k bf16(x~_k) L1[k, :]) on the FP64 matrix cores
//     (t_step_f64): the products are exact in double and the double sum is
//     within ~1e-13 of the exact one, far inside bf16's half ulp, so the
//     single rounding to bf16 gives the bf16 of the exact sum.  The per-wave
//     partial tiles are summed in LDS in wave order.
//  2. every wave walks its groups again: the re-read, re-smoothed x~ goes
//     through r rank-1 updates on the FP32 matrix cores (deflate_step), whose
//     result is in the quantizer's lane layout.
// ---------------------------------------------------------------------------
template <int RANK, bool INV_LDS>
__global__ __launch_bounds__(64 * act_waves<RANK>()) void quantize_act_deflated_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth,
    const uint16_t* __restrict__ L1f, const uint16_t* __restrict__ L1, uint8_t* __restrict__ xq, float* __restrict__ xs,
    uint16_t* __restrict__ t, int M, int K, int groups_per_wave, int g32) {
  constexpr int RB = RANK / 16;
  // dynamic LDS: [nwaves][16][RANK] double partial t | [16][RANK] float -t |
  // (INV_LDS) [nwaves][groups_per_wave * 64] 1/lambda
  extern __shared__ double red64[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int row = lane & 15;
  const int chunk = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int rows = min(16, M - m0);
  const int G = K / kGroup;
  const int g_begin = wave * groups_per_wave;
  const int g_end = min(G, g_begin + groups_per_wave);

  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<uint32_t>(rows) * K * 2u);
  const buf_rsrc q_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * (K / 2), static_cast<uint32_t>(rows) * (K / 2));
  const uint32_t x_off = static_cast<uint32_t>(row * K + chunk * 16) * 2u;
  const uint32_t q_off = static_cast<uint32_t>(row * (K / 2) + chunk * 8);

  float* tneg = reinterpret_cast<float*>(red64 + nwaves * 16 * RANK);
  float* inv_w = tneg + 16 * RANK + wave * groups_per_wave * kGroup;
  if (INV_LDS && g_begin < g_end) {
    const int n4 = (g_end - g_begin) * (kGroup / 4);
    const float4* src = reinterpret_cast<const float4*>(inv_smooth + g_begin * kGroup);
    for (int i = lane; i < n4; i += 64) reinterpret_cast<float4*>(inv_w)[i] = src[i];
  }
  auto inv_ptr = [&](int g) __attribute__((always_inline)) {
    return INV_LDS ? reinterpret_cast<const float4*>(inv_w + (g - g_begin) * kGroup + chunk * 16)
                   : reinterpret_cast<const float4*>(inv_smooth + g * kGroup + chunk * 16);
  };

  // ---- phase 1: t in double ----
  auto fetch1 = [&](int g, ActFetch<RANK>& f) __attribute__((always_inline)) {
    const uint32_t go = static_cast<uint32_t>(g) * kGroup * 2u;
    f.xa = buf_load16(x_rsrc, x_off + go);
    f.xb = buf_load16(x_rsrc, x_off + go + 16u);
    load_l1_fragments<RB>(L1f, g, lane, f.l1);
  };
  v4d acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = v4d{0.0, 0.0, 0.0, 0.0};
  auto work1 = [&](int g, const ActFetch<RANK>& f) __attribute__((always_inline)) {
    float v[16];
    smooth16(f.xa, f.xb, inv_ptr(g), v);
    t_step_f64<RB>(v, f.l1, acc);
  };
  if (g_begin < g_end) {
    ActFetch<RANK> fa, fb;
    fetch1(g_begin, fa);
    int g = g_begin;
    for (; g + 1 < g_end; g += 2) {
      fetch1(g + 1, fb);
      work1(g, fa);
      fetch1(min(g + 2, g_end - 1), fa);
      work1(g + 1, fb);
    }
    if (g < g_end) work1(g, fa);
  }
  store_t_partials<RB>(red64, wave, lane, acc);
  __syncthreads();
  reduce_t<RANK>(red64, nwaves, rows, t + static_cast<int64_t>(m0) * RANK, tneg);
  __syncthreads();

  // ---- phase 2: deflate with r rank-1 updates, then quantize ----
  const int a_ch = deflate_channel(lane);
  auto fetch2 = [&](int g, DeflFetch<RANK>& f) __attribute__((always_inline)) {
    const uint32_t go = static_cast<uint32_t>(g) * kGroup * 2u;
    f.xa = buf_load16(x_rsrc, x_off + go);
    f.xb = buf_load16(x_rsrc, x_off + go + 16u);
    load_l1_row<RANK>(L1, g * kGroup + a_ch, f.l1);
  };
  const float* tn_row = tneg + row * RANK;
  auto work2 = [&](int g, const DeflFetch<RANK>& f) __attribute__((always_inline)) {
    float v[16];
    smooth16(f.xa, f.xb, inv_ptr(g), v);
    deflate_step<RANK>(v, f.l1, tn_row);
    quantize_pack_store(v, q_rsrc, q_off + static_cast<uint32_t>(g) * (kGroup / 2),
                        xs_slot(xs, g, M, m0, row, rows, chunk, g32), g32);
  };
  if (g_begin < g_end) {
    DeflFetch<RANK> fa, fb;
    fetch2(g_begin, fa);
    int g = g_begin;
    for (; g + 1 < g_end; g += 2) {
      fetch2(g + 1, fb);
      work2(g, fa);
      fetch2(min(g + 2, g_end - 1), fa);
      work2(g + 1, fb);
    }
    if (g < g_end) work2(g, fa);
  }
}

// ---------------------------------------------------------------------------
hipError_t launch_pack_weights(int K, int N, int group, const float* R, const float* smooth, uint8_t* wq,
                               float* ws, uint32_t* wsp, float* inv_smooth, hipStream_t stream) {
  const int64_t teams = static_cast<int64_t>(N) * (K / kGroup);
  const int64_t blocks = (teams * 4 + 255) / 256;
  hipLaunchKernelGGL(pack_weights_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, R,
                     wq, ws, wsp, N, K, group == 32 ? 1 : 0);
  hipLaunchKernelGGL(inverse_smoothing_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, smooth,
                     inv_smooth, K);
  return hipGetLastError();
}

hipError_t launch_quantize_act(int M, int K, int r, int group, const uint16_t* x, const float* inv_smooth,
                               const uint16_t* L1f, uint8_t* xq, float* xs, uint16_t* t,
                               hipStream_t stream) {
  const int g32 = group == 32 ? 1 : 0;
  const int G = K / kGroup;
  // 1/lambda is staged in LDS when the slice fits (K <= 16384); larger K reads it from global memory
  const bool inv_lds = K <= 16384;
  auto go = [&](auto kernel_lds, auto kernel_global, int max_waves) {
    int nwaves = G < max_waves ? G : max_waves;
    int gpw = (G + nwaves - 1) / nwaves;
    if (G >= 64) {   // wave ranges of whole 4-group line chunks (below, the waves keep one group or more each)
      gpw = (gpw + 3) & ~3;
      nwaves = (G + gpw - 1) / gpw;
    }
    // the code-line buffers (2 KB per wave) only where the kernel uses them
    const size_t lds = static_cast<size_t>(nwaves) * (16 * r + (inv_lds ? gpw * kGroup : 0)) * sizeof(float) +
                       (gpw % 4 == 0 ? static_cast<size_t>(nwaves) * 2048 : 0);
    if (lds > 64 * 1024) {   // opt in to more than 64 KB of dynamic LDS
      const void* fn = inv_lds ? reinterpret_cast<const void*>(kernel_lds) : reinterpret_cast<const void*>(kernel_global);
      const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      if (e != hipSuccess) return e;
    }
    if (inv_lds)
      hipLaunchKernelGGL(kernel_lds, dim3((M + 15) / 16), dim3(64 * nwaves), lds, stream, x, inv_smooth, L1f,
                         xq, xs, t, M, K, gpw, g32);
    else
      hipLaunchKernelGGL(kernel_global, dim3((M + 15) / 16), dim3(64 * nwaves), lds, stream, x, inv_smooth, L1f,
                         xq, xs, t, M, K, gpw, g32);
    return hipGetLastError();
  };
  switch (r) {
    case 16: return go(quantize_act_kernel<16, true>, quantize_act_kernel<16, false>, act_waves<16>());
    case 32: return go(quantize_act_kernel<32, true>, quantize_act_kernel<32, false>, act_waves<32>());
    case 48: return go(quantize_act_kernel<48, true>, quantize_act_kernel<48, false>, act_waves<48>());
    case 64: return go(quantize_act_kernel<64, true>, quantize_act_kernel<64, false>, act_waves<64>());
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_quantize_act_deflated(int M, int K, int r, int group, const uint16_t* x,
                                        const float* inv_smooth, const uint16_t* L1f, const uint16_t* L1,
                                        uint8_t* xq, float* xs, uint16_t* t, hipStream_t stream) {
  const int g32 = group == 32 ? 1 : 0;
  const int G = K / kGroup;
  const bool inv_lds = K <= 16384;
  auto go = [&](auto kernel_lds, auto kernel_global, int max_waves) {
    const int nwaves = G < max_waves ? G : max_waves;
    const int gpw = (G + nwaves - 1) / nwaves;
    const size_t lds = static_cast<size_t>(nwaves) * 16 * r * sizeof(double) + 16 * r * sizeof(float) +
                       (inv_lds ? static_cast<size_t>(nwaves) * gpw * kGroup * sizeof(float) : 0);
    if (lds > 64 * 1024) {
      const void* fn = inv_lds ? reinterpret_cast<const void*>(kernel_lds) : reinterpret_cast<const void*>(kernel_global);
      const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      if (e != hipSuccess) return e;
    }
    if (inv_lds)
      hipLaunchKernelGGL(kernel_lds, dim3((M + 15) / 16), dim3(64 * nwaves), lds, stream, x, inv_smooth, L1f,
                         L1, xq, xs, t, M, K, gpw, g32);
    else
      hipLaunchKernelGGL(kernel_global, dim3((M + 15) / 16), dim3(64 * nwaves), lds, stream, x, inv_smooth, L1f,
                         L1, xq, xs, t, M, K, gpw, g32);
    return hipGetLastError();
  };
  switch (r) {
    case 16: return go(quantize_act_deflated_kernel<16, true>, quantize_act_deflated_kernel<16, false>, act_waves<16>());
    case 32: return go(quantize_act_deflated_kernel<32, true>, quantize_act_deflated_kernel<32, false>, act_waves<32>());
    case 48: return go(quantize_act_deflated_kernel<48, true>, quantize_act_deflated_kernel<48, false>, act_waves<48>());
    case 64: return go(quantize_act_deflated_kernel<64, true>, quantize_act_deflated_kernel<64, false>, act_waves<64>());
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qwam
