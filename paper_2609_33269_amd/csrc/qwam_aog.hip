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
//     the ASP GEMM so that the fragment loads are bank-conflict free; one
//     barrier per stage;
//   * the matrix cores consume a stage (64 x 128 x 128 MACs) far faster than
//     a copy from the infinity cache or HBM returns, so the ring is four
//     stages deep (three in flight while one is multiplied, 96 KB per CU) and
//     a CU runs one workgroup, which owns 128 KB of LDS;
//   * workgroups are mapped XCD-major onto the triangle of tiles taken in
//     8 x 8 super-blocks, so that the tiles resident on one XCD at a time
//     share their row panels of gT in its L2.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int TB = 128;            // tile edge
constexpr int NST = 2;             // ring stages
constexpr int WG_PER_CU = 2;       // workgroups per CU (LDS: NST stages or the epilogue tile each)
constexpr int NWAVES_S = 4;
constexpr int NT_S = 64 * NWAVES_S;
constexpr int KS = 64;             // values of n per ring stage (one 128-byte line per row)
constexpr int ROWB_S = KS * 2;
constexpr int STAGE_B = 2 * TB * ROWB_S;   // bytes of one stage: A tile, then B tile ([row][8 swizzled chunk slots])
constexpr int LDC = TB + 4;        // float row stride of the epilogue tile (16-byte rows, conflict-free reads)
constexpr int SMEM_B = NST * STAGE_B > TB * LDC * 4 ? NST * STAGE_B : TB * LDC * 4;

typedef float v16f_s __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int swz_s(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// LDS byte address of a pointer into a __shared__ variable
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  typedef const __attribute__((address_space(3))) uint8_t lds_u8;
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u8*)(p)));
}

// 16-byte LDS read issued as inline assembly: the compiler's wait insertion
// cannot tell an LDS read of one ring stage from the direct copies into
// another and would make every read wait for all copies in flight.  The
// caller waits for the result with lgkm_wait_for.
__device__ __forceinline__ v4i lds_read16(uint32_t addr) {
  v4i r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

// s_waitcnt lgkmcnt(N), tied to the fragments it makes valid so that no use
// of them is scheduled before it
template <int N>
__device__ __forceinline__ void lgkm_wait_for(v4i (&f)[4]) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]) : "i"(N));
}

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

__global__ __launch_bounds__(NT_S, WG_PER_CU) void aog_syrk_kernel(const uint16_t* __restrict__ gT,
                                                                  float* __restrict__ A, int d, int n) {
  // the ring of NST stages; after the main loop, the epilogue tile
  __shared__ __attribute__((aligned(16))) uint8_t smem[SMEM_B];

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
  auto stage_a = [&](int k) __attribute__((always_inline)) { return smem + k * STAGE_B; };
  auto stage_b = [&](int k) __attribute__((always_inline)) { return smem + k * STAGE_B + TB * ROWB_S; };
  auto issue = [&](int s, int k) __attribute__((always_inline)) {
    const uint32_t ko = static_cast<uint32_t>(s) * ROWB_S;
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(a_rsrc, d_off[i] + ko, stage_a(k) + (4 * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(b_rsrc, d_off[i] + ko, stage_b(k) + (4 * wave + i) * 1024);
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

  // stage s (slot k = s % NST): wait for this wave's copies of stage s (those
  // of the next NST - 2 stages, when issued, may stay in flight: 8 copies per
  // stage and wave), barrier, then refill the slot of stage s-1 (every wave
  // is past it) with stage s + NST - 1
  auto stage_step = [&](int s, int k) __attribute__((always_inline)) {
    static_assert(NST == 2 || NST == 4, "wait counts for 2 or 4 stages");
    if (NST == 4 && s + 2 < S) wait_vmcnt<16>();
    else if (NST == 4 && s + 1 < S) wait_vmcnt<8>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (s + NST - 1 < S) issue(s + NST - 1, (k + NST - 1) % NST);
    // fragments of k-step q + 1 are read while step q multiplies
    const uint32_t a_base = lds_addr(stage_a(k)) + (wm * 64) * ROWB_S + frow_off;
    const uint32_t b_base = lds_addr(stage_b(k)) + (wn * 64) * ROWB_S + frow_off;
    v4i fr[2][4];
    auto read_step = [&](int q, v4i (&f)[4]) __attribute__((always_inline)) {
      const uint32_t so = static_cast<uint32_t>(((2 * q) ^ fslot) * 16);
      f[0] = lds_read16(a_base + so);
      f[1] = lds_read16(a_base + so + 32 * ROWB_S);
      f[2] = lds_read16(b_base + so);
      f[3] = lds_read16(b_base + so + 32 * ROWB_S);
    };
    read_step(0, fr[0]);
#pragma unroll
    for (int q = 0; q < KS / 16; ++q) {
      v4i(&f)[4] = fr[q & 1];
      if (q + 1 < KS / 16) {
        read_step(q + 1, fr[(q + 1) & 1]);
        lgkm_wait_for<4>(f);
      } else {
        lgkm_wait_for<0>(f);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, f[i]),
                                                              __builtin_bit_cast(v8bf, f[2 + j]), acc[i][j], 0, 0, 0);
    }
  };

#pragma unroll
  for (int k = 0; k + 1 < NST; ++k)
    if (k < S) issue(k, k);
  // whole rounds of NST stages (slots static after unrolling), then the rest
  int s = 0;
  for (; s + NST <= S; s += NST) {
#pragma unroll
    for (int k = 0; k < NST; ++k) stage_step(s + k, k);
  }
#pragma unroll
  for (int k = 0; k + 1 < NST; ++k)
    if (s + k < S) stage_step(s + k, k);

  // ---- epilogue: A[I][J] += C and, transposed, A[J][I] += C^T, through LDS ----
  // The tile C goes to LDS ([row][LDC] floats); both read-modify-write passes
  // then touch whole rows of A: the normal one 16 bytes per lane along a row
  // of C, the transposed one 4 bytes per lane down a column of C (64
  // consecutive rows of C = 256 contiguous bytes of a row of A).  On a
  // diagonal tile the normal pass writes r <= c and the transposed one r < c.
  lds_barrier();                                   // every wave is past the ring
  float* C = reinterpret_cast<float*>(smem);
  // result layout of a 32x32 block: lane l holds column l%32 and rows
  // 8*(v/4) + 4*(l/32) + v%4, v = 0..15
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        C[(wm * 64 + i * 32 + 8 * (v >> 2) + 4 * fhalf + (v & 3)) * LDC + wn * 64 + j * 32 + frow] = acc[i][j][v];
  __syncthreads();

  const bool diag = ti == tj;
  const bool full = m0 + TB <= d && n0 + TB <= d;
  // normal pass: thread t takes the float4 of columns 4 (t % 32) .. +3 in rows
  // t / 32 + 8 q, q = 0..15
  {
    const int c4 = tid & 31, rr = tid >> 5;
    float* arow = A + static_cast<int64_t>(m0 + rr) * d + n0 + 4 * c4;
    if (full && !diag) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float4 o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = *reinterpret_cast<const float4*>(arow + static_cast<int64_t>(8 * (8 * h + q)) * d);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float4 cv = *reinterpret_cast<const float4*>(C + (rr + 8 * (8 * h + q)) * LDC + 4 * c4);
          o[q].x += cv.x;
          o[q].y += cv.y;
          o[q].z += cv.z;
          o[q].w += cv.w;
          *reinterpret_cast<float4*>(arow + static_cast<int64_t>(8 * (8 * h + q)) * d) = o[q];
        }
      }
    } else {
      for (int q = 0; q < 16; ++q) {
        const int r = rr + 8 * q;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 4 * c4 + u;
          if (m0 + r < d && n0 + c < d && (!diag || r <= c))
            arow[static_cast<int64_t>(8 * q) * d + u] += C[r * LDC + c];
        }
      }
    }
  }
  // transposed pass: thread t takes row r = t % 128 of C and the columns
  // 4 (t / 128 + 2 q) .. +3, q = 0..15: A[n0 + c][m0 + r] += C[r][c]
  {
    const int r = tid & (TB - 1), cq = tid >> 7;
    float* acol = A + static_cast<int64_t>(n0) * d + m0 + r;
    if (full && !diag) {
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        float o[16];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int u = 0; u < 4; ++u) o[4 * q + u] = acol[static_cast<int64_t>(4 * (cq + 2 * (4 * h + q)) + u) * d];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c4 = cq + 2 * (4 * h + q);
          const float4 cv = *reinterpret_cast<const float4*>(C + r * LDC + 4 * c4);
          acol[static_cast<int64_t>(4 * c4 + 0) * d] = o[4 * q + 0] + cv.x;
          acol[static_cast<int64_t>(4 * c4 + 1) * d] = o[4 * q + 1] + cv.y;
          acol[static_cast<int64_t>(4 * c4 + 2) * d] = o[4 * q + 2] + cv.z;
          acol[static_cast<int64_t>(4 * c4 + 3) * d] = o[4 * q + 3] + cv.w;
        }
      }
    } else {
      for (int q = 0; q < 16; ++q) {
        const int c4 = cq + 2 * q;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 4 * c4 + u;
          if (m0 + r < d && n0 + c < d && (!diag || r < c)) acol[static_cast<int64_t>(c) * d] += C[r * LDC + c];
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
