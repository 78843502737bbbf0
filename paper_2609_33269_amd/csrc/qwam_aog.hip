// Accumulation of the Action Observability Gramian (AOG) estimate: every
// probe's vector-Jacobian product g = J^T u adds g g^T to a d x d float32
// accumulator (the probe estimator's procedure; G^ = A / (N P), Sec. 4.1).
// A batch of n VJPs stored channel-major, gT [d][n] (row c = channel c of the
// n vectors), makes this a symmetric rank-n update
//
//     A += gT gT^T,      A[i][j] += sum_k gT[i][k] gT[j][k],
//
// an NT matrix product whose two operands are both K-contiguous rows of gT.
//
//   * only the tiles (I, J) with I <= J are computed (128 x 128, four waves of
//     64 x 64 = 2 x 2 blocks of v_mfma_f32_32x32x16_bf16); each is added to
//     A[I][J] and, transposed, to A[J][I].  On a diagonal tile the upper
//     triangle comes from the normal write and the strict lower triangle from
//     the transposed one, so A stays exactly symmetric;
//   * products of two bf16 values are exact in float32; the sums are float32
//     in the matrix cores' order;
//   * a ring stage holds 64 values of n, i.e. one 128-byte line of every row
//     of the two operand tiles, copied straight from HBM/L2 into LDS by
//     buffer_load ... lds (rows past d read as zero), with the chunk swizzle of
//     the ASP GEMM so that the fragment loads are bank-conflict free; two
//     stages, one barrier per stage, two workgroups per CU;
//   * workgroups are mapped XCD-major onto the triangle of tiles taken in
//     8 x 8 super-blocks, so that the tiles resident on one XCD at a time
//     share their row panels of gT in its L2.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int TB = 128;            // tile edge
constexpr int NWAVES_S = 4;
constexpr int NT_S = 64 * NWAVES_S;
constexpr int KS = 64;             // values of n per ring stage (one 128-byte line per row)
constexpr int ROWB_S = KS * 2;

typedef float v16f_s __attribute__((ext_vector_type(16)));

struct SyrkStage {
  uint8_t a[TB * ROWB_S];          // [row][8 chunk slots of 16 bytes], swizzled
  uint8_t b[TB * ROWB_S];
};

__device__ __forceinline__ int swz_s(int r) { return (r & 7) ^ ((r >> 3) & 1); }

constexpr int SBK = 8;             // tiles per edge of a super-block

// Tile (ti, tj), ti <= tj, of workgroup `bid`.  The upper triangle of tiles is
// enumerated super-block by super-block (8 x 8 tiles, the diagonal ones
// triangular; super-blocks in row-major order, tiles row-major inside), and
// the 8 XCDs take contiguous ranges of that order (hardware places workgroup b
// on XCD b % 8).  The ~64 workgroups resident on one XCD then cover about one
// super-block, whose tiles share 16 row panels of gT in that XCD's L2.
__device__ __forceinline__ void triangle_tile(int bid, int T, int& ti, int& tj) {
  const int total = T * (T + 1) / 2;
  const int per = total / 8, rem = total % 8;
  const int x = bid % 8, i = bid / 8;
  int idx = (x < rem) ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
  const int SB = (T + SBK - 1) / SBK;
  for (int I = 0; I < SB; ++I) {
    const int h = min(SBK, T - I * SBK);                 // tile rows of this super-row
    for (int J = I; J < SB; ++J) {
      const int w = min(SBK, T - J * SBK);               // tile columns of this super-column
      const int cnt = (I == J) ? h * (h + 1) / 2 : h * w;
      if (idx < cnt) {
        if (I == J) {                                    // triangle: row a has h - a tiles
          int a = 0;
          while (idx >= h - a) {
            idx -= h - a;
            ++a;
          }
          ti = I * SBK + a;
          tj = I * SBK + a + idx;
        } else {
          ti = I * SBK + idx / w;
          tj = J * SBK + idx % w;
        }
        return;
      }
      idx -= cnt;
    }
  }
  ti = tj = 0;                                           // not reached for bid < total
}

}  // namespace

__global__ __launch_bounds__(NT_S, 2) void aog_syrk_kernel(const uint16_t* __restrict__ gT, float* __restrict__ A,
                                                          int d, int n) {
  __shared__ __attribute__((aligned(16))) SyrkStage st0, st1;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int T = (d + TB - 1) / TB;
  int ti, tj;
  triangle_tile(blockIdx.x, T, ti, tj);
  const int m0 = ti * TB, n0 = tj * TB;
  const uint32_t RB = static_cast<uint32_t>(n) * 2u;   // bytes per row of gT
  const int S = n / KS;

  // LDS-DMA: copy i (0..3) of wave w fills rows 8*(4w+i) .. +7 of a tile, lane
  // l taking row 8*(4w+i) + l/8 and slot l%8, which holds chunk (l%8) ^ swz(row)
  const buf_rsrc a_rsrc = make_rsrc(gT + static_cast<int64_t>(m0) * n, static_cast<uint32_t>(min(TB, d - m0)) * RB);
  const buf_rsrc b_rsrc = make_rsrc(gT + static_cast<int64_t>(n0) * n, static_cast<uint32_t>(min(TB, d - n0)) * RB);
  uint32_t d_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 8 * (4 * wave + i) + (lane >> 3);
    d_off[i] = static_cast<uint32_t>(row) * RB + static_cast<uint32_t>(((lane & 7) ^ swz_s(row)) * 16);
  }
  auto issue = [&](int s, SyrkStage& st) __attribute__((always_inline)) {
    const uint32_t ko = static_cast<uint32_t>(s) * ROWB_S;
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(a_rsrc, d_off[i] + ko, st.a + (4 * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(b_rsrc, d_off[i] + ko, st.b + (4 * wave + i) * 1024);
  };

  v16f_s acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16f_s{};

  // v_mfma_f32_32x32x16_bf16 operands: lane l holds row l%32 and the 8
  // consecutive k of half l/32 of a 16-wide k step, i.e. chunk 2q + l/32 of
  // the row in step q
  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int frow_off = frow * ROWB_S;
  const int fslot = fhalf ^ swz_s(frow);

  auto stage_step = [&](int s, const SyrkStage& cur, SyrkStage& nxt) __attribute__((always_inline)) {
    wait_vmcnt<0>();
    lds_barrier();
    if (s + 1 < S) issue(s + 1, nxt);
#pragma unroll
    for (int q = 0; q < KS / 16; ++q) {
      const int slot_off = ((2 * q) ^ fslot) * 16;
      v8s af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const v8s*>(cur.a + (wm * 64 + i * 32) * ROWB_S + frow_off + slot_off);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = *reinterpret_cast<const v8s*>(cur.b + (wn * 64 + j * 32) * ROWB_S + frow_off + slot_off);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, af[i]),
                                                              __builtin_bit_cast(v8bf, bf[j]), acc[i][j], 0, 0, 0);
    }
  };

  issue(0, st0);
  int s = 0;
  for (; s + 1 < S; s += 2) {
    stage_step(s, st0, st1);
    stage_step(s + 1, st1, st0);
  }
  if (s < S) stage_step(s, st0, st1);

  // ---- epilogue: read-modify-write of A[I][J] and, transposed, A[J][I] ----
  // result layout of a 32x32 block: lane l holds column l%32 and rows
  // 8*(v/4) + 4*(l/32) + v%4, v = 0..15
  const bool diag = ti == tj;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = n0 + wn * 64 + j * 32 + frow;                  // column of A[I][J]
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const int r0 = m0 + wm * 64 + i * 32 + 8 * v4 + 4 * fhalf; // rows r0 .. r0+3
        // normal orientation: A[r][c] += acc, r <= c on the diagonal tile
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = r0 + u;
          if (r < d && c < d && (!diag || r <= c)) A[static_cast<int64_t>(r) * d + c] += acc[i][j][4 * v4 + u];
        }
        // transposed: A[c][r0 .. r0+3] += acc, r < c on the diagonal tile
        if (c < d) {
          float* dst = A + static_cast<int64_t>(c) * d + r0;
          if (!diag && r0 + 3 < d) {
            float4 o = *reinterpret_cast<const float4*>(dst);
            o.x += acc[i][j][4 * v4 + 0];
            o.y += acc[i][j][4 * v4 + 1];
            o.z += acc[i][j][4 * v4 + 2];
            o.w += acc[i][j][4 * v4 + 3];
            *reinterpret_cast<float4*>(dst) = o;
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int r = r0 + u;
              if (r < d && (!diag || r < c)) dst[u] += acc[i][j][4 * v4 + u];
            }
          }
        }
      }
    }
}

hipError_t launch_aog_accumulate(int d, int n, const uint16_t* gT, float* A, hipStream_t stream) {
  const int T = (d + TB - 1) / TB;
  hipLaunchKernelGGL(aog_syrk_kernel, dim3(T * (T + 1) / 2), dim3(NT_S), 0, stream, gT, A, d, n);
  return hipGetLastError();
}

}  // namespace qwam
