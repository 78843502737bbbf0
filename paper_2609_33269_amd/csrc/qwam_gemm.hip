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
//   * wave (wm, wn) owns rows 64*wm.. and columns 64*wn.. as 4 x 4 blocks of
//     v_mfma_i32_16x16x64_i8 (K = 64 is exactly one quantization group, so one
//     MFMA per block and group gives the exact int32 partial of that group);
//   * per group, every thread fetches 16 packed bytes of A and 16 of B with
//     buffer loads (zero past the valid rows / the last group, so the loop is
//     branch-free and the fetch ring stays three groups deep), unpacks them to
//     int8 (16 * code: each product is 256 * qx * qw, exact) into one of two LDS
//     stages, and the waves read MFMA fragments back; one barrier per group;
//   * LDS tile rows are 64 bytes with an XOR swizzle of the four 16-byte chunks
//     so that both the unpack stores and the fragment loads are free of bank
//     conflicts;
//   * the int32 block results of a group are converted and scaled at once into
//     float32 accumulators (convert, scale product, fused multiply-add);
//   * workgroups are mapped XCD-major: the 8 XCDs each take a contiguous range
//     of tiles, ordered in bands of 8 tile-rows so that the concurrently
//     resident tiles of one XCD share their A and B panels in its L2;
//   * epilogue: the bf16 branch MFMA starts from 2^-8 * acc, the bias is added,
//     the result is rounded to bf16 and stored through LDS so that every lane
//     writes 16 contiguous bytes.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int NWAVES = 4;
constexpr int NT = 64 * NWAVES;
constexpr int WG_PER_CU = 3;
constexpr int LDY = 64 + 8;        // LDS row stride (bf16) of the output staging
constexpr int YROWS = 32;          // output rows staged per pass and wave
constexpr int BAND = 8;            // tile-rows per band of the tile order

struct Stage {
  int8_t a[BM * 64];
  int8_t b[BN * 64];
  float sx[BM];
  float sw[BN];
};
constexpr int kStageBytes = sizeof(Stage);
constexpr int kEpiBytes = NWAVES * YROWS * LDY * 2;
constexpr int kSmemBytes = (2 * kStageBytes > kEpiBytes) ? 2 * kStageBytes : kEpiBytes;

// Byte offset of 16-byte chunk c (0..3) of tile row r: rows are 64 bytes and
// the chunk index is XORed with a function of the row such that 16 consecutive
// rows at one logical chunk (a fragment load, or a stash store) fall on 16
// distinct 16-byte bank groups, and any 8 consecutive rows on 8.
__device__ __forceinline__ int swz(int r, int c) {
  return r * 64 + ((c ^ (((r >> 1) ^ (r >> 3)) & 3)) << 4);
}

// Unpack 16 packed bytes (32 codes, k = 0..31 of one half of a group row) and
// store the even-k codes to logical chunk 2h and the odd-k codes to chunk 2h+1
// of row r (the same permutation of k for A and B, so the MFMA dot products
// are unchanged).
__device__ __forceinline__ void store_unpacked(int8_t* tile, int r, int h, uint4 p) {
  uint32_t e0, o0, e1, o1, e2, o2, e3, o3;
  unpack_nibbles_x16(p.x, e0, o0);
  unpack_nibbles_x16(p.y, e1, o1);
  unpack_nibbles_x16(p.z, e2, o2);
  unpack_nibbles_x16(p.w, e3, o3);
  *reinterpret_cast<uint4*>(tile + swz(r, 2 * h)) = make_uint4(e0, e1, e2, e3);
  *reinterpret_cast<uint4*>(tile + swz(r, 2 * h + 1)) = make_uint4(o0, o1, o2, o3);
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

// Per-thread global fetch of one group: 16 packed bytes of A (32 codes of one
// row), 16 packed bytes of B and one scale.
struct Fetch {
  uint4 a, b;
  float s;
};

template <int RANK, bool PARTIALS>
__global__ __launch_bounds__(NT, WG_PER_CU) void asp_gemm_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint16_t* __restrict__ t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ P, int M,
    int N, int K) {
  __shared__ __attribute__((aligned(16))) char smem[kSmemBytes];
  Stage* stages = reinterpret_cast<Stage*>(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (SGPR)
  const int wm = wave >> 1, wn = wave & 1;   // 2 x 2 waves
  const int G = K / kGroup;
  const int KB = K / 2;

  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  // ---- global fetch assignment (branch-free: buffer loads return 0 past the
  // valid rows of the tile and past the end of each array) ----
  const buf_rsrc a_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * KB,
                                    static_cast<uint32_t>(min(BM, M - m0)) * KB);
  const buf_rsrc b_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB,
                                    static_cast<uint32_t>(min(BN, N - n0)) * KB);
  // thread -> (row, half): 16 consecutive lanes take 16 consecutive rows, so a
  // stash store instruction hits the same conflict-free pattern as a fragment load
  const int lrow = (tid & 15) + 16 * (tid >> 5);
  const int lhalf = (tid >> 4) & 1;
  const uint32_t l_off = static_cast<uint32_t>(lrow * KB + lhalf * 16);
  // scales: waves 0-1 fetch xs of the tile's rows, waves 2-3 ws of its columns
  const bool s_is_x = wave < 2;
  const int s_idx = tid & (BM - 1);
  buf_rsrc s_rsrc = s_is_x ? make_rsrc(xs, static_cast<uint32_t>(G) * M * 4u)
                           : make_rsrc(ws, static_cast<uint32_t>(G) * N * 4u);
  const uint32_t s_off = static_cast<uint32_t>((s_is_x ? m0 : n0) + s_idx) * 4u;
  const uint32_t s_stride = static_cast<uint32_t>(s_is_x ? M : N) * 4u;

  auto fetch = [&](int g, Fetch& f) {
    f.a = buf_load16(a_rsrc, l_off + static_cast<uint32_t>(g) * 32u);
    f.b = buf_load16(b_rsrc, l_off + static_cast<uint32_t>(g) * 32u);
    if (!PARTIALS) f.s = buf_load4f(s_rsrc, s_off + static_cast<uint32_t>(g) * s_stride);
  };
  auto stash = [&](const Fetch& f, Stage& st) {
    store_unpacked(st.a, lrow, lhalf, f.a);
    store_unpacked(st.b, lrow, lhalf, f.b);
    if (!PARTIALS) {
      if (s_is_x) st.sx[s_idx] = f.s;
      else st.sw[s_idx] = f.s;
    }
  };

  float accf[4][4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) accf[i][j][v] = 0.0f;

  const int frow = lane & 15;
  const int fc = lane >> 4;
  const int rsub = fc * 4;

  // prologue: group 0 into LDS stage 0; groups 1..3 in flight in f1, f2, f0
  Fetch f0, f1, f2;
  fetch(0, f0);
  fetch(1, f1);
  fetch(2, f2);
  stash(f0, stages[0]);
  fetch(3, f0);
  __syncthreads();

  // one group: stage group g+1 (held in `nxt`) into `other` (its last readers
  // passed the barrier that ended the previous group), refill `nxt` with group
  // g+4, then MFMA + scale the current stage.  Stashes and fetches past the
  // last group touch only the unused stage and read zeros.
  auto group_step = [&](int g, Fetch& nxt, const Stage& cur, Stage& other) {
    stash(nxt, other);
    fetch(g + 4, nxt);

    v4i bfr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfr[j] = *reinterpret_cast<const v4i*>(cur.b + swz(wn * 64 + j * 16 + frow, fc));
    float swv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) swv[j] = cur.sw[wn * 64 + j * 16 + frow];

    // software pipeline over the four 16-row blocks: the MFMAs of block i+1 are
    // issued before the convert/scale of block i, so the VALU never waits on a
    // just-issued MFMA
    v4i pc[4], pn[4];
    {
      const v4i af = *reinterpret_cast<const v4i*>(cur.a + swz(wm * 64 + frow, fc));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        pc[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bfr[j], v4i{0, 0, 0, 0}, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i < 3) {
        const v4i af = *reinterpret_cast<const v4i*>(cur.a + swz(wm * 64 + (i + 1) * 16 + frow, fc));
#pragma unroll
        for (int j = 0; j < 4; ++j)
          pn[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bfr[j], v4i{0, 0, 0, 0}, 0, 0, 0);
      }
      if (PARTIALS) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + wm * 64 + i * 16 + rsub + v;
            const int n = n0 + wn * 64 + j * 16 + frow;
            if (m < M && n < N) P[(static_cast<int64_t>(m) * N + n) * G + g] = pc[j][v] >> 8;
          }
      } else {
        const float4 sx4 = *reinterpret_cast<const float4*>(&cur.sx[wm * 64 + i * 16 + rsub]);
        const float sxv[4] = {sx4.x, sx4.y, sx4.z, sx4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            accf[i][j][v] = __builtin_fmaf(static_cast<float>(pc[j][v]), sxv[v] * swv[j], accf[i][j][v]);
      }
      if (i < 3) {
#pragma unroll
        for (int j = 0; j < 4; ++j) pc[j] = pn[j];
      }
    }
    __syncthreads();
  };

  // six groups per trip so that the three fetch registers and two LDS stages
  // are named statically
  int g = 0;
  for (; g + 5 < G; g += 6) {
    group_step(g, f1, stages[0], stages[1]);
    group_step(g + 1, f2, stages[1], stages[0]);
    group_step(g + 2, f0, stages[0], stages[1]);
    group_step(g + 3, f1, stages[1], stages[0]);
    group_step(g + 4, f2, stages[0], stages[1]);
    group_step(g + 5, f0, stages[1], stages[0]);
  }
  if (g < G) group_step(g, f1, stages[0], stages[1]);
  if (g + 1 < G) group_step(g + 1, f2, stages[1], stages[0]);
  if (g + 2 < G) group_step(g + 2, f0, stages[0], stages[1]);
  if (g + 3 < G) group_step(g + 3, f1, stages[1], stages[0]);
  if (g + 4 < G) group_step(g + 4, f2, stages[0], stages[1]);

  if (PARTIALS) return;

  // ---- epilogue: 2^-8 * acc + t . L2 (bf16 MFMA, float32 accumulate) + bias ----
  constexpr int KSTEPS = (RANK + 31) / 32;
  const int kk = (lane >> 4) * 8;
  v8s lf[4][KSTEPS];
  float bv[4];
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
    bv[j] = (bias != nullptr && n < N) ? bf16_to_f32(bias[n]) : 0.0f;
  }
  uint16_t* ys = reinterpret_cast<uint16_t*>(smem) + wave * YROWS * LDY;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    __syncthreads();   // LDS free (previous pass's reads, or the main loop's)
#pragma unroll
    for (int ii = 0; ii < 2; ++ii) {
      const int i = pass * 2 + ii;
      const int m = m0 + wm * 64 + i * 16 + frow;
      v8s tf[KSTEPS];
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const int j0 = s * 32 + kk;
        v8s val = {0, 0, 0, 0, 0, 0, 0, 0};
        if (m < M && j0 < RANK) val = *reinterpret_cast<const v8s*>(t + static_cast<int64_t>(m) * RANK + j0);
        tf[s] = val;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v4f c;
#pragma unroll
        for (int v = 0; v < 4; ++v) c[v] = accf[i][j][v] * 0x1p-8f;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s)
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, tf[s]),
                                                      __builtin_bit_cast(v8bf, lf[j][s]), c, 0, 0, 0);
#pragma unroll
        for (int v = 0; v < 4; ++v)
          ys[(ii * 16 + rsub + v) * LDY + j * 16 + frow] =
              static_cast<uint16_t>(f32_to_bf16_rne(c[v] + bv[j]));
      }
    }
    __syncthreads();
    // the wave's 32 staged rows x 64 columns: 8 lanes per row, 16 bytes each
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int r = it * 8 + (lane >> 3);
      const int c8 = (lane & 7) * 8;
      const int m = m0 + wm * 64 + pass * 32 + r;
      const int n = n0 + wn * 64 + c8;
      if (m < M && n < N)
        *reinterpret_cast<uint4*>(y + static_cast<int64_t>(m) * N + n) =
            *reinterpret_cast<const uint4*>(ys + r * LDY + c8);
    }
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
