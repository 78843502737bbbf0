// The ASP GEMM: W4A4 integer group partial sums on INT8 matrix cores, float32
// per-group scaling in registers, and the bf16 low-rank branch + bias fused in
// the epilogue (the second kernel of App. B.1; Eq. 2 and Eq. 9).
//
//   y[m, n] = bf16( 2^-8 * sum_g xs[g][m] ws[g][n] * (256 * P[m, n, g])
//                   + sum_j t[m, j] L2t[n, j] + bias[n] )
//
// Work decomposition (gfx950, 256 CUs in 8 XCDs, 64-wide waves):
//   * a 256-thread workgroup (4 waves) owns a 128 x 128 tile of y and three
//     workgroups share a CU (3 waves per SIMD), so one workgroup's barrier and
//     LDS waits are covered by the others' VALU work;
//   * the packed 4-bit codes stay packed all the way into LDS: every group's
//     A and B tiles (128 rows x 32 bytes each) and scales are copied straight
//     from HBM/L2 into a 4-stage LDS ring by buffer_load ... lds (no VGPR
//     staging, zero past the valid rows and past the last group), three groups
//     ahead of the group being multiplied; one barrier per group;
//   * a tile is stored half-major ([2 halves][128 rows][16 bytes]), so the
//     fragment loads (one ds_read_b128 = 32 codes of one row per lane) read
//     contiguous 512-byte runs and are free of bank conflicts;
//   * wave (wm, wn) owns rows 64*wm.. and columns 64*wn.. as 2 x 2 blocks of
//     v_mfma_i32_32x32x32_i8: lane l holds row l%32 and half l/32 of a group,
//     unpacked in registers to int8 (16 * code: each product is 256 * qx * qw,
//     exact); two MFMA k-steps per block give the exact int32 partial of the
//     group;
//   * the MFMAs of the next block are issued before the convert / scale of the
//     current one (convert, scale product, fused multiply-add into float32
//     accumulators), so the VALU never waits on a just-issued MFMA;
//   * workgroups are mapped XCD-major: the 8 XCDs each take a contiguous range
//     of tiles, ordered in bands of 8 tile-rows so that the concurrently
//     resident tiles of one XCD share their A and B panels in its L2;
//   * epilogue: the bf16 branch (v_mfma_f32_32x32x16_bf16, same result layout
//     as the integer blocks) starts from 2^-8 * acc, the bias is added, the
//     result is rounded to bf16 and stored through LDS so that every lane
//     writes 16 contiguous bytes.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int NWAVES = 4;
constexpr int NT = 64 * NWAVES;
constexpr int WG_PER_CU = 3;
constexpr int LDY = 64 + 8;        // LDS row stride (bf16) of the output staging
constexpr int BAND = 8;            // tile-rows per band of the tile order

struct Stage {
  uint8_t a[2 * BM * 16];          // [half][row][16 bytes]
  uint8_t b[2 * BN * 16];
  float sx[BM];
  float sw[BN];
};
constexpr int kStageBytes = sizeof(Stage);
static_assert(64 * LDY * 2 <= kStageBytes, "a wave's output staging must fit in one ring stage");

// 16 packed codes (two dwords, low nibble = even k) -> one MFMA operand of 16
// int8 values 16*code, ordered [even k of w0, even k of w1, odd k of w0, odd k of w1]
// (the same permutation for A and B, so the dot product is unchanged).
__device__ __forceinline__ v4i unpack16(uint32_t w0, uint32_t w1) {
  uint32_t e0, o0, e1, o1;
  unpack_nibbles_x16(w0, e0, o0);
  unpack_nibbles_x16(w1, e1, o1);
  return v4i{static_cast<int>(e0), static_cast<int>(e1), static_cast<int>(o0), static_cast<int>(o1)};
}

// Tile of workgroup `bid`: XCD-major remap (hardware places workgroup b on XCD
// b % 8), then bands of BAND tile-rows, columns fastest inside a band-column.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  const int per = total / 8, rem = total % 8;
  const int x = bid % 8, i = bid / 8;
  const int logical = (x < rem) ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
  const int band_tiles = BAND * tiles_n;
  const int band = logical / band_tiles;
  const int in_band = logical % band_tiles;
  const int rows_in_band = min(BAND, tiles_m - band * BAND);
  tm = band * BAND + in_band % rows_in_band;
  tn = in_band / rows_in_band;
}

}  // namespace

template <int RANK, bool PARTIALS>
__global__ __launch_bounds__(NT, WG_PER_CU) void asp_gemm_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint16_t* __restrict__ t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ P, int M,
    int N, int K) {
  // four distinct LDS objects (not one indexed array), so that the compiler
  // can tell which ring stage a copy writes and a fragment load reads, and
  // waits only for the copies of the stage being read
  __shared__ __attribute__((aligned(16))) Stage st0, st1, st2, st3;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (SGPR)
  const int wm = wave >> 1, wn = wave & 1;                      // 2 x 2 waves
  const int G = K / kGroup;
  const int KB = K / 2;

  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  // ---- LDS-DMA assignment: wave w fills 16-byte units w*64 .. w*64+63 of the
  // half-major tile, i.e. half w/2, rows (w%2)*64 + lane ----
  const buf_rsrc a_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * KB,
                                    static_cast<uint32_t>(min(BM, M - m0)) * KB);
  const buf_rsrc b_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB,
                                    static_cast<uint32_t>(min(BN, N - n0)) * KB);
  const int d_row = (wave & 1) * 64 + lane;
  const int d_half = wave >> 1;
  const uint32_t d_off = static_cast<uint32_t>(d_row * KB + d_half * 16);
  // scales: waves 0-1 copy xs of the tile's rows, waves 2-3 ws of its columns
  const bool s_is_x = wave < 2;
  const buf_rsrc s_rsrc = s_is_x ? make_rsrc(xs, static_cast<uint32_t>(G) * M * 4u)
                                 : make_rsrc(ws, static_cast<uint32_t>(G) * N * 4u);
  const uint32_t s_off = static_cast<uint32_t>((s_is_x ? m0 : n0) + (wave & 1) * 64 + lane) * 4u;
  const uint32_t s_stride = static_cast<uint32_t>(s_is_x ? M : N) * 4u;

  auto issue = [&](int g, Stage& st) {
    const uint32_t go = static_cast<uint32_t>(g) * 32u;
    buf_load16_lds(a_rsrc, d_off + go, st.a + wave * 1024);
    buf_load16_lds(b_rsrc, d_off + go, st.b + wave * 1024);
    if (!PARTIALS)
      buf_load4_lds(s_rsrc, s_off + static_cast<uint32_t>(g) * s_stride,
                    s_is_x ? static_cast<void*>(st.sx + (wave & 1) * 64)
                           : static_cast<void*>(st.sw + (wave & 1) * 64));
  };
  // vector-memory ops per issue(); the partials dump also stores inside the
  // loop, so it simply waits for everything
  constexpr int kWaitOps = PARTIALS ? 0 : 2 * 3;

  v16f accf[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) accf[i][j] = v16f{};

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int rsub = fhalf * 4;

  issue(0, st0);
  issue(1, st1);
  issue(2, st2);

  // one group: `cur` holds group g, `nxt3` (the stage of group g-1) receives g+3
  auto group_step = [&](int g, const Stage& cur, Stage& nxt3) {
    wait_vmcnt<kWaitOps>();           // this thread's copies of group g have landed
    lds_barrier();                    // ... and every thread's; group g-1 is fully consumed
    issue(g + 3, nxt3);

    // fragments: one ds_read_b128 per 32-row block = 32 codes of row frow, half fhalf
    v4i af[2][2], bf[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint4 pa = *reinterpret_cast<const uint4*>(cur.a + (fhalf * BM + wm * 64 + i * 32 + frow) * 16);
      af[i][0] = unpack16(pa.x, pa.y);
      af[i][1] = unpack16(pa.z, pa.w);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint4 pb = *reinterpret_cast<const uint4*>(cur.b + (fhalf * BN + wn * 64 + j * 32 + frow) * 16);
      bf[j][0] = unpack16(pb.x, pb.y);
      bf[j][1] = unpack16(pb.z, pb.w);
    }

    auto mfma_block = [&](int i, int j) {
      v16i acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i][0], bf[j][0], v16i{}, 0, 0, 0);
      return __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i][1], bf[j][1], acc, 0, 0, 0);
    };
    // result layout of a 32x32 block: lane l holds column l%32 and rows
    // 8*(v/4) + 4*(l/32) + v%4, v = 0..15
    auto consume = [&](int i, int j, const v16i& p) {
      if (PARTIALS) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = m0 + wm * 64 + i * 32 + 8 * (v >> 2) + rsub + (v & 3);
          const int n = n0 + wn * 64 + j * 32 + frow;
          if (m < M && n < N) P[(static_cast<int64_t>(m) * N + n) * G + g] = p[v] >> 8;
        }
      } else {
        const float swv = cur.sw[wn * 64 + j * 32 + frow];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 sx4 = *reinterpret_cast<const float4*>(&cur.sx[wm * 64 + i * 32 + 8 * q + rsub]);
          const float sxv[4] = {sx4.x, sx4.y, sx4.z, sx4.w};
#pragma unroll
          for (int v = 0; v < 4; ++v)
            accf[i][j][4 * q + v] =
                __builtin_fmaf(static_cast<float>(p[4 * q + v]), sxv[v] * swv, accf[i][j][4 * q + v]);
        }
      }
    };
    // software pipeline: MFMAs of the next block before the epilogue of this one
    const v16i p00 = mfma_block(0, 0);
    const v16i p01 = mfma_block(0, 1);
    consume(0, 0, p00);
    const v16i p10 = mfma_block(1, 0);
    consume(0, 1, p01);
    const v16i p11 = mfma_block(1, 1);
    consume(1, 0, p10);
    consume(1, 1, p11);
  };

  // four groups per trip so that every ring stage is named statically
  int g = 0;
  for (; g + 3 < G; g += 4) {
    group_step(g, st0, st3);
    group_step(g + 1, st1, st0);
    group_step(g + 2, st2, st1);
    group_step(g + 3, st3, st2);
  }
  if (g < G) group_step(g, st0, st3);
  if (g + 1 < G) group_step(g + 1, st1, st0);
  if (g + 2 < G) group_step(g + 2, st2, st1);
  wait_vmcnt<0>();     // the copies issued past the last group (zeros) must land
  __syncthreads();     // before the LDS is reused below

  if (PARTIALS) return;

  // ---- epilogue: 2^-8 * acc + t . L2 (bf16 MFMA, float32 accumulate) + bias ----
  // v_mfma_f32_32x32x16_bf16: lane l holds row/column l%32 and the 8 rank slots
  // 8*(l/32) .. +7 of a 16-wide rank step (the same slots for t and L2t).
  constexpr int KSTEPS = RANK / 16;
  const int kk = fhalf * 8;
  v8s tf[2][KSTEPS], lf[2][KSTEPS];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = m0 + wm * 64 + i * 32 + frow;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      v8s val = {0, 0, 0, 0, 0, 0, 0, 0};
      if (m < M) val = *reinterpret_cast<const v8s*>(t + static_cast<int64_t>(m) * RANK + s * 16 + kk);
      tf[i][s] = val;
    }
  }
  float bv[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + wn * 64 + j * 32 + frow;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      v8s val = {0, 0, 0, 0, 0, 0, 0, 0};
      if (n < N) val = *reinterpret_cast<const v8s*>(L2t + static_cast<int64_t>(n) * RANK + s * 16 + kk);
      lf[j][s] = val;
    }
    bv[j] = (bias != nullptr && n < N) ? bf16_to_f32(bias[n]) : 0.0f;
  }
  // each wave stages its 64 x 64 bf16 outputs in one of the (now idle) ring stages
  Stage* mine = (wave == 0) ? &st0 : (wave == 1) ? &st1 : (wave == 2) ? &st2 : &st3;
  uint16_t* ys = reinterpret_cast<uint16_t*>(mine);   // [64][LDY] bf16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      v16f c = accf[i][j] * 0x1p-8f;
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, tf[i][s]),
                                                    __builtin_bit_cast(v8bf, lf[j][s]), c, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 16; ++v)
        ys[(i * 32 + 8 * (v >> 2) + rsub + (v & 3)) * LDY + j * 32 + frow] =
            static_cast<uint16_t>(f32_to_bf16_rne(c[v] + bv[j]));
    }
  __syncthreads();
  // the wave's 64 rows x 64 columns: 8 lanes per row, 16 bytes each
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int r = it * 8 + (lane >> 3);
    const int c8 = (lane & 7) * 8;
    const int m = m0 + wm * 64 + r;
    const int n = n0 + wn * 64 + c8;
    if (m < M && n < N)
      *reinterpret_cast<uint4*>(y + static_cast<int64_t>(m) * N + n) =
          *reinterpret_cast<const uint4*>(ys + r * LDY + c8);
  }
}

static int gemm_tiles(int M, int N) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

hipError_t launch_asp_gemm(int M, int N, int K, int r, const uint8_t* xq, const float* xs,
                           const uint16_t* t, const uint8_t* wq, const float* ws,
                           const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                           hipStream_t stream) {
  const dim3 grid(gemm_tiles(M, N)), block(NT);
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
  hipLaunchKernelGGL((asp_gemm_kernel<32, true>), dim3(gemm_tiles(M, N)), dim3(NT), 0, stream, xq, nullptr,
                     nullptr, wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  return hipGetLastError();
}

}  // namespace qwam
