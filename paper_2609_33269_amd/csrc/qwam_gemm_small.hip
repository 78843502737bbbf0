// The ASP GEMM for few tokens (M <= 64: the action-expert layers).  Same
// arithmetic as the large-tile kernel (exact integer group partials on
// v_mfma_scale_f32_32x32x64_f8f6f4, float32 scaling per group, the bf16 branch
// and the bias in the epilogue), organised for latency instead of reuse:
//
//   * one 8-wave workgroup per 32 x 32 block of y (rows = tokens, columns =
//     output channels), the K groups split into eight contiguous ranges, one
//     per wave: with so few tokens the layer is a stream over the packed
//     weights, and the split spreads that stream and the per-group work over
//     eight waves.  The eight partial blocks are summed in LDS in wave order
//     (deterministic); wave w finishes result registers 2w and 2w+1 (the
//     branch t . L2 on the bf16 matrix cores, the bias, the store).  The
//     fused few-token layer uses the same split and the same order, so both
//     paths give the same y from the same codes, scales and t;
//   * every operand goes straight from HBM/L2 into the MFMA register layout
//     (lane l: row / column l % 32, half l / 32 of a group, 16 bytes = 32
//     codes), four groups per chunk, two chunks in flight: with eight waves a
//     K of 4096 is one memory round trip;
//   * the activation scales are broadcast across each row of 16 lanes by DPP
//     inside the scale multiply, as in the large-tile kernel;
//   * group 32 (GS = 32): as in the large-tile kernel, lane half h holds group
//     h of the 64-channel span and each block runs once per group with the
//     other lane half's scales at 2^-127.
#include <type_traits>

#include "qwam_device.h"
#include "qwam_internal.h"
#include "qwam_mfma.h"

namespace qwam {

namespace {

constexpr int SB = 32;             // block edge (rows and columns)
constexpr int CH = 4;              // groups per chunk
constexpr int KW = 8;              // waves per block, each a contiguous range of groups

template <int NS>
struct Chunk {
  uint4 a[CH], b[CH];              // packed codes of this lane's row / column and half
  float sx[CH][NS], sw[CH][NS];    // the lane's activation scale (DPP source) and weight scale
};

}  // namespace

template <int RANK, bool PARTIALS, int GS>
__global__ __launch_bounds__(64 * KW) void asp_gemm_small_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint16_t* __restrict__ t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ P, int M,
    int N, int K) {
  __shared__ float red[KW][16][64];       // partial blocks of the waves

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles_n = (N + SB - 1) / SB;
  const int m0 = (blockIdx.x / tiles_n) * SB;
  const int n0 = (blockIdx.x % tiles_n) * SB;
  constexpr int NS = kGroup / GS;  // scale groups per 64-channel span
  const int G = K / kGroup;
  const int GSC = K / GS;
  const int KB = K / 2;
  // this wave's groups: [g_lo, g_hi)
  const int gpw = (G + KW - 1) / KW;
  const int g_lo = min(G, wave * gpw), g_hi = min(G, g_lo + gpw);
  const int NC = (g_hi - g_lo + CH - 1) / CH;

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int rsub = fhalf * 4;
  // activation-scale row of this lane inside the block: lane 16*rho + v holds
  // the scale of result register v of lanes in rows rho (v = lane % 16):
  // row 8*(v/4) + 4*(lane/32) + v%4
  const int sx_row = 8 * ((lane & 15) >> 2) + 4 * (lane >> 5) + (lane & 3);

  // rows / columns past M / N read as zero
  const buf_rsrc a_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * KB, static_cast<uint32_t>(min(SB, M - m0)) * KB);
  const buf_rsrc b_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB, static_cast<uint32_t>(min(SB, N - n0)) * KB);
  const buf_rsrc xs_rsrc = make_rsrc(xs, static_cast<uint32_t>(GSC) * M * 4u);
  const buf_rsrc ws_rsrc = make_rsrc(ws, static_cast<uint32_t>(GSC) * N * 4u);
  // the lane's 16-byte half of the span (with group 32: one group)
  const uint32_t ab_off = static_cast<uint32_t>(frow * KB + fhalf * 16);
  const uint32_t sx_off = static_cast<uint32_t>(m0 + sx_row) * 4u;
  const uint32_t sw_off = static_cast<uint32_t>(n0 + frow) * 4u;

  // chunk c holds groups g_lo + CH*c .. + CH-1; in the last chunk, groups
  // past g_hi are never loaded (a row's next bytes belong to the next row) and
  // never multiplied.  FULL chunks need no per-group check.
  auto load_frag = [&](buf_rsrc r, uint32_t off) __attribute__((always_inline)) { return buf_load16(r, off); };
  auto load = [&](int c, Chunk<NS>& ch, auto full) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int g = g_lo + c * CH + q;
      if (decltype(full)::value || g < g_hi) {
        ch.a[q] = load_frag(a_rsrc, ab_off + static_cast<uint32_t>(g) * 32u);
        ch.b[q] = load_frag(b_rsrc, ab_off + static_cast<uint32_t>(g) * 32u);
        if (!PARTIALS) {
#pragma unroll
          for (int h = 0; h < NS; ++h) {
            ch.sx[q][h] = buf_load4f(xs_rsrc, sx_off + static_cast<uint32_t>(NS * g + h) * M * 4u);
            ch.sw[q][h] = buf_load4f(ws_rsrc, sw_off + static_cast<uint32_t>(NS * g + h) * N * 4u);
          }
        }
      }
    }
  };

  v16f acc = v16f{};
  auto process = [&](int c, const Chunk<NS>& ch, auto full) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const int g = g_lo + c * CH + q;
      if (decltype(full)::value || g < g_hi) {
        const v8i af = codes_to_fp6(ch.a[q]), bf = codes_to_fp6(ch.b[q]);
#pragma unroll
        for (int h = 0; h < NS; ++h) {
          int sc = kE8M0Code;
          if constexpr (GS == 32) sc = ((lane >> 5) == h) ? kE8M0Code : 0;
          const v16f p = fp6_partial(af, bf, sc, sc);
          if (PARTIALS) {
            // result layout: lane l holds column l%32 and rows 8*(v/4) + 4*(l/32) + v%4
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int m = m0 + 8 * (v >> 2) + rsub + (v & 3);
              const int n = n0 + frow;
              if (m < M && n < N) P[(static_cast<int64_t>(m) * N + n) * GSC + NS * g + h] = static_cast<int32_t>(p[v]);
            }
          } else {
            scale_accumulate(std::make_integer_sequence<int, 16>{}, acc, p, ch.sx[q][h], ch.sw[q][h]);
          }
        }
      }
    }
  };
  using Full = std::true_type;
  using Tail = std::false_type;
  auto load_any = [&](int c, Chunk<NS>& ch) __attribute__((always_inline)) {
    if (g_lo + (c + 1) * CH <= g_hi) load(c, ch, Full{});
    else load(c, ch, Tail{});
  };
  auto process_any = [&](int c, const Chunk<NS>& ch) __attribute__((always_inline)) {
    if (g_lo + (c + 1) * CH <= g_hi) process(c, ch, Full{});
    else process(c, ch, Tail{});
  };

  // the epilogue's operands (t rows, L2t rows, bias) are requested with the
  // first chunk, so that they do not cost a round trip of their own
  constexpr int KSTEPS = RANK / 16;
  const int kk = fhalf * 8;
  const int mt = m0 + frow, nt = n0 + frow;
  v8s tv[KSTEPS], lv[KSTEPS];
  uint32_t bbits = 0;              // bias bits, converted only in the epilogue (no early wait)
  if constexpr (!PARTIALS) {
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      tv[s] = v8s{0, 0, 0, 0, 0, 0, 0, 0};
      lv[s] = v8s{0, 0, 0, 0, 0, 0, 0, 0};
      if (mt < M) tv[s] = *reinterpret_cast<const v8s*>(t + static_cast<int64_t>(mt) * RANK + s * 16 + kk);
      if (nt < N) lv[s] = *reinterpret_cast<const v8s*>(L2t + static_cast<int64_t>(nt) * RANK + s * 16 + kk);
    }
    const buf_rsrc b_rsrc = make_rsrc(bias, bias != nullptr ? static_cast<uint32_t>(N) * 2u : 0u);
    bbits = __builtin_amdgcn_raw_buffer_load_b16(b_rsrc, static_cast<uint32_t>(nt) * 2u, 0, 0);
  }

  // two chunks in flight: chunk c+1 is requested before chunk c is multiplied
  Chunk<NS> c0, c1;
  if (NC > 0) load_any(0, c0);
  for (int c = 0; c < NC; c += 2) {
    if (c + 1 < NC) load_any(c + 1, c1);
    process_any(c, c0);
    if (c + 2 < NC) load_any(c + 2, c0);
    if (c + 1 < NC) process_any(c + 1, c1);
  }
  if (PARTIALS) return;

  // partial blocks -> LDS, summed in wave order: wave w finishes result
  // registers v0 = 2w and v0 + 1 (token 8(v/4) + 4(l/32) + v%4, column l%32)
#pragma unroll
  for (int v = 0; v < 16; ++v) red[wave][v][lane] = acc[v];
  __syncthreads();
  const int v0 = 2 * wave;
  float c2[2] = {0.0f, 0.0f};
#pragma unroll
  for (int w = 0; w < KW; ++w)
#pragma unroll
    for (int e = 0; e < 2; ++e) c2[e] += red[w][v0 + e][lane];

  // ---- epilogue: acc + t . L2 (bf16 MFMA, float32 accumulate) + bias; the
  // other result registers start at zero and are not used ----
  v16f c;
#pragma unroll
  for (int v = 0; v < 16; ++v) c[v] = v == v0 ? c2[0] : (v == v0 + 1 ? c2[1] : 0.0f);
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s)
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, tv[s]), __builtin_bit_cast(v8bf, lv[s]), c,
                                                0, 0, 0);
  const float bv = bf16_to_f32(bbits);
  float yv[2] = {0.0f, 0.0f};
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    if (v == v0) yv[0] = c[v];
    if (v == v0 + 1) yv[1] = c[v];
  }
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int v = v0 + e;
    const int m = m0 + 8 * (v >> 2) + rsub + (v & 3);
    if (m < M && nt < N) y[static_cast<int64_t>(m) * N + nt] = static_cast<uint16_t>(f32_to_bf16_rne(yv[e] + bv));
  }
}

static unsigned small_blocks(int M, int N) {
  return static_cast<unsigned>(((M + SB - 1) / SB) * ((N + SB - 1) / SB));
}

template <int GS>
static hipError_t launch_small_gs(int M, int N, int K, int r, const uint8_t* xq, const float* xs, const uint16_t* t,
                                  const uint8_t* wq, const float* ws, const uint16_t* L2t, const uint16_t* bias,
                                  uint16_t* y, hipStream_t stream) {
  const dim3 grid(small_blocks(M, N)), block(64 * KW);
  switch (r) {
    case 16:
      hipLaunchKernelGGL((asp_gemm_small_kernel<16, false, GS>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 32:
      hipLaunchKernelGGL((asp_gemm_small_kernel<32, false, GS>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 48:
      hipLaunchKernelGGL((asp_gemm_small_kernel<48, false, GS>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 64:
      hipLaunchKernelGGL((asp_gemm_small_kernel<64, false, GS>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_asp_gemm_small(int M, int N, int K, int r, int group, const uint8_t* xq, const float* xs,
                                 const uint16_t* t, const uint8_t* wq, const float* ws,
                                 const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                                 hipStream_t stream) {
  return group == 32 ? launch_small_gs<32>(M, N, K, r, xq, xs, t, wq, ws, L2t, bias, y, stream)
                     : launch_small_gs<64>(M, N, K, r, xq, xs, t, wq, ws, L2t, bias, y, stream);
}

hipError_t launch_group_partials_small(int M, int N, int K, int group, const uint8_t* xq, const uint8_t* wq,
                                       int32_t* P, hipStream_t stream) {
  if (group == 32)
    hipLaunchKernelGGL((asp_gemm_small_kernel<32, true, 32>), dim3(small_blocks(M, N)), dim3(64 * KW), 0, stream, xq,
                       nullptr, nullptr, wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  else
    hipLaunchKernelGGL((asp_gemm_small_kernel<32, true, 64>), dim3(small_blocks(M, N)), dim3(64 * KW), 0, stream, xq,
                       nullptr, nullptr, wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  return hipGetLastError();
}

}  // namespace qwam
