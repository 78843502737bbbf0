// The ASP GEMM: W4A4 integer group partial sums on INT8 matrix cores, float32
// per-group scaling in registers, and the bf16 low-rank branch + bias fused in
// the epilogue (the second kernel of App. B.1; Eq. 2 and Eq. 9).
//
//   y[m, n] = bf16( 2^-8 * sum_g xs[g][m] ws[g][n] * (256 * P[m, n, g])
//                   + sum_j t[m, j] L2t[n, j] + bias[n] )
//
// Tiling: a 256-thread workgroup computes a 128 x 128 tile of y, four waves
// in a 2 x 2 arrangement, each wave 64 x 64 = 4 x 4 blocks of
// v_mfma_i32_16x16x64_i8 (one MFMA per block and group: K = 64 is one group).
// Per group, every thread loads 16 bytes of packed A and 16 of packed B from
// HBM/L2, unpacks them to int8 (16*code, so each product is 256*qx*qw) into
// LDS, and the waves read their MFMA fragments back from LDS.  The int32 block
// results of a group are converted and scaled right away (three VALU ops per
// output and group) into float32 accumulators.  The epilogue initialises the
// bf16 MFMA of the branch with the scaled 4-bit result, adds the bias, rounds
// to bf16 and stores through LDS so that each lane writes 16 contiguous bytes.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int NT = 256;
constexpr int LDA = 80;            // LDS row stride (bytes) of the int8 tiles: 64 + 16 pad
constexpr int LDY = 64 + 8;        // LDS row stride (bf16 elements) of the output staging

struct TileSmem {
  int8_t a[BM * LDA];
  int8_t b[BN * LDA];
  float sx[BM];
  float sw[BN];
};
constexpr int kEpiBytes = 4 * 64 * LDY * 2;
constexpr int kSmemBytes = sizeof(TileSmem) > kEpiBytes ? sizeof(TileSmem) : kEpiBytes;

__device__ __forceinline__ void store_unpacked(int8_t* dst, uint4 p) {
  uint32_t e0, o0, e1, o1, e2, o2, e3, o3;
  unpack_nibbles_x16(p.x, e0, o0);
  unpack_nibbles_x16(p.y, e1, o1);
  unpack_nibbles_x16(p.z, e2, o2);
  unpack_nibbles_x16(p.w, e3, o3);
  reinterpret_cast<uint4*>(dst)[0] = make_uint4(e0, e1, e2, e3);
  reinterpret_cast<uint4*>(dst)[1] = make_uint4(o0, o1, o2, o3);
}

}  // namespace

template <int RANK, bool PARTIALS>
__global__ __launch_bounds__(NT) void asp_gemm_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint16_t* __restrict__ t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ P, int M,
    int N, int K) {
  __shared__ __attribute__((aligned(16))) char smem_raw[kSmemBytes];
  TileSmem& sm = *reinterpret_cast<TileSmem*>(smem_raw);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int G = K / kGroup;
  const int KB = K / 2;  // bytes per packed row

  const int tiles_m = (M + BM - 1) / BM;
  const int tm = blockIdx.x % tiles_m;
  const int tn = blockIdx.x / tiles_m;
  const int m0 = tm * BM, n0 = tn * BN;

  // global -> LDS mapping: thread owns 16 packed bytes (32 codes) of one row
  const int lrow = tid >> 1, lhalf = tid & 1;
  const bool a_ok = (m0 + lrow) < M;
  const bool b_ok = (n0 + lrow) < N;
  const uint8_t* a_src = xq + static_cast<int64_t>(a_ok ? m0 + lrow : 0) * KB + lhalf * 16;
  const uint8_t* b_src = wq + static_cast<int64_t>(b_ok ? n0 + lrow : 0) * KB + lhalf * 16;
  // scales: threads 0..127 fetch xs of the tile's rows, 128..255 ws of its columns
  const bool s_is_x = tid < BM;
  const int s_idx = s_is_x ? tid : tid - BM;
  const bool s_ok = s_is_x ? (m0 + s_idx < M) : (n0 + s_idx < N);
  const float* s_src = s_is_x ? (xs + m0 + s_idx) : (ws + n0 + s_idx);
  const int64_t s_stride = s_is_x ? M : N;

  float accf[4][4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) accf[i][j][v] = 0.0f;

  uint4 pa = make_uint4(0, 0, 0, 0), pb = make_uint4(0, 0, 0, 0);
  float ps = 0.0f;
  if (a_ok) pa = *reinterpret_cast<const uint4*>(a_src);
  if (b_ok) pb = *reinterpret_cast<const uint4*>(b_src);
  if (!PARTIALS && s_ok) ps = s_src[0];

  const int frow = lane & 15;   // fragment row inside a 16-row block
  const int fk = (lane >> 4) * 16;  // fragment byte offset inside the 64-byte row

  for (int g = 0; g < G; ++g) {
    __syncthreads();
    store_unpacked(sm.a + lrow * LDA + lhalf * 32, pa);
    store_unpacked(sm.b + lrow * LDA + lhalf * 32, pb);
    if (!PARTIALS) {
      if (s_is_x) sm.sx[s_idx] = ps; else sm.sw[s_idx] = ps;
    }
    __syncthreads();
    if (g + 1 < G) {
      pa = make_uint4(0, 0, 0, 0);
      pb = make_uint4(0, 0, 0, 0);
      if (a_ok) pa = *reinterpret_cast<const uint4*>(a_src + (g + 1) * 32);
      if (b_ok) pb = *reinterpret_cast<const uint4*>(b_src + (g + 1) * 32);
      if (!PARTIALS && s_ok) ps = s_src[static_cast<int64_t>(g + 1) * s_stride];
    }

    v4i af[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      af[i] = *reinterpret_cast<const v4i*>(sm.a + (wm * 64 + i * 16 + frow) * LDA + fk);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfr[j] = *reinterpret_cast<const v4i*>(sm.b + (wn * 64 + j * 16 + frow) * LDA + fk);

    v4i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bfr[j], v4i{0, 0, 0, 0}, 0, 0, 0);

    if (PARTIALS) {
      // exact partials: P = (256 * P) >> 8; result row 4*(l/16)+v, column l%16
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + v;
            const int n = n0 + wn * 64 + j * 16 + frow;
            if (m < M && n < N) P[(static_cast<int64_t>(m) * N + n) * G + g] = acc[i][j][v] >> 8;
          }
    } else {
      float sxv[4][4], swv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) sxv[i][v] = sm.sx[wm * 64 + i * 16 + (lane >> 4) * 4 + v];
#pragma unroll
      for (int j = 0; j < 4; ++j) swv[j] = sm.sw[wn * 64 + j * 16 + frow];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float sc = sxv[i][v] * swv[j];
            accf[i][j][v] = __builtin_fmaf(static_cast<float>(acc[i][j][v]), sc, accf[i][j][v]);
          }
    }
  }

  if (PARTIALS) return;

  // ---- epilogue: 2^-8 * acc + t . L2 (bf16 MFMA, float32 accumulate) + bias ----
  constexpr int KSTEPS = (RANK + 31) / 32;
  v8s tf[4][KSTEPS], lf[4][KSTEPS];
  const int kk = (lane >> 4) * 8;  // 8 rank slots of this lane inside a 32-wide step
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + wm * 64 + i * 16 + frow;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const int j0 = s * 32 + kk;
      v8s val = {0, 0, 0, 0, 0, 0, 0, 0};
      if (m < M && j0 < RANK) val = *reinterpret_cast<const v8s*>(t + static_cast<int64_t>(m) * RANK + j0);
      tf[i][s] = val;
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + wn * 64 + j * 16 + frow;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const int j0 = s * 32 + kk;
      v8s val = {0, 0, 0, 0, 0, 0, 0, 0};
      if (n < N && j0 < RANK) val = *reinterpret_cast<const v8s*>(L2t + static_cast<int64_t>(n) * RANK + j0);
      lf[j][s] = val;
    }
  }
  float bv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + wn * 64 + j * 16 + frow;
    bv[j] = (bias != nullptr && n < N) ? bf16_to_f32(bias[n]) : 0.0f;
  }

  __syncthreads();  // the tile buffers are reused for output staging
  uint16_t* ys = reinterpret_cast<uint16_t*>(smem_raw) + wave * 64 * LDY;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v4f c;
#pragma unroll
      for (int v = 0; v < 4; ++v) c[v] = accf[i][j][v] * 0x1p-8f;
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, tf[i][s]),
                                                    __builtin_bit_cast(v8bf, lf[j][s]), c, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = i * 16 + (lane >> 4) * 4 + v;
        const int cidx = j * 16 + frow;
        ys[r * LDY + cidx] = static_cast<uint16_t>(f32_to_bf16_rne(c[v] + bv[j]));
      }
    }
  __syncthreads();
  // each wave writes its 64 x 64 tile: 8 lanes per row, 16 bytes per lane
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int r = it * 8 + (lane >> 3);
    const int c8 = (lane & 7) * 8;
    const int m = m0 + wm * 64 + r;
    const int n = n0 + wn * 64 + c8;
    if (m < M && n < N) {
      const uint4 val = *reinterpret_cast<const uint4*>(ys + r * LDY + c8);
      *reinterpret_cast<uint4*>(y + static_cast<int64_t>(m) * N + n) = val;
    }
  }
}

hipError_t launch_asp_gemm(int M, int N, int K, int r, const uint8_t* xq, const float* xs,
                           const uint16_t* t, const uint8_t* wq, const float* ws,
                           const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                           hipStream_t stream) {
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const dim3 grid(tiles), block(NT);
  switch (r) {
    case 16:
      hipLaunchKernelGGL((asp_gemm_kernel<16, false>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 32:
      hipLaunchKernelGGL((asp_gemm_kernel<32, false>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 48:
      hipLaunchKernelGGL((asp_gemm_kernel<48, false>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    case 64:
      hipLaunchKernelGGL((asp_gemm_kernel<64, false>), grid, block, 0, stream, xq, xs, t, wq, ws, L2t, bias, y, nullptr, M, N, K);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_group_partials(int M, int N, int K, const uint8_t* xq, const uint8_t* wq,
                                 int32_t* P, hipStream_t stream) {
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  hipLaunchKernelGGL((asp_gemm_kernel<32, true>), dim3(tiles), dim3(NT), 0, stream, xq, nullptr, nullptr,
                     wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  return hipGetLastError();
}

}  // namespace qwam
