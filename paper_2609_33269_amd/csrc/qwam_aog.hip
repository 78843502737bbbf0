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
//   * only the tiles (I, J) with I <= J are computed (TB x TB); each is added
//     to A[I][J] and, transposed, to A[J][I].  Eight waves, two per SIMD: wave
//     w owns the TB/2 x TB/2 block (w%4)/2, w%2 of the tile (BW x BW blocks of
//     v_mfma_f32_32x32x16_bf16) for half w/4 of every stage's k-steps, so that
//     one wave's matrix-core work covers the other's LDS reads; the two
//     partial blocks are summed once, after the last stage (the half with the
//     later k-steps added to the other, in that fixed order).  On a diagonal tile the upper
//     triangle comes from the normal write and the strict lower triangle from
//     the transposed one, so A stays exactly symmetric;
//   * products of two bf16 values are exact in float32; the sums are float32
//     in the matrix cores' order;
//   * a ring stage holds 64 values of n, i.e. one 128-byte line of every row
//     of the two operand tiles, copied straight from HBM/L2 into LDS by
//     buffer_load ... lds (rows past d read as zero), with the chunk swizzle of
//     the ASP GEMM so that the fragment loads are bank-conflict free; one
//     barrier per stage, one workgroup per CU;
//   * the tile is as large as one round of workgroups allows (LDS traffic per
//     product falls with the tile edge): TB = 192 when the 192-tile triangle
//     fits on the 256 CUs and the 128-tile one does not (d = 2817 .. 4224, the
//     paper's layer widths up to 4096), TB = 128 otherwise.  Three stages of 48 KB (192) or
//     four of 32 KB (128) keep 96 KB in flight per CU;
//   * the tile goes through LDS (C, then C^T) so that both read-modify-write
//     passes move 16 bytes per lane along rows of A; with TB = 128 the reads
//     of A[I][J] are issued during the last stages;
//   * workgroups are mapped XCD-major onto the triangle of tiles taken in
//     8 x 8 super-blocks, so that the tiles resident on one XCD at a time
//     share their row panels of gT in its L2.
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int NWAVES_S = 8;
constexpr int NT_S = 64 * NWAVES_S;
constexpr int KS = 64;             // values of n per ring stage (one 128-byte line per row)
constexpr int ROWB_S = KS * 2;

typedef float v16f_s __attribute__((ext_vector_type(16)));

template <int TB>
struct SyrkCfg {
  static_assert(TB == 128 || TB == 192, "tile edge 128 or 192");
  static constexpr int BW = TB / 64;                       // 32x32 blocks per wave edge
  static constexpr int NST = TB == 128 ? 4 : 3;            // ring stages
  static constexpr int STAGE_B = 2 * TB * ROWB_S;          // A tile, then B tile ([row][8 swizzled chunk slots])
  static constexpr int CPW = TB / (8 * NWAVES_S);          // 1 KB copies per operand, stage and wave
  static constexpr int IPS = 2 * CPW;                      // copies per stage and wave
  static constexpr int LDC = TB + 4;                       // float row stride of the epilogue tile
  static constexpr int F4 = TB * TB / 4 / NT_S;            // float4 of a tile per thread
  static constexpr int SMEM_B = NST * STAGE_B > TB * LDC * 4 ? NST * STAGE_B : TB * LDC * 4;
  // the early reads of A[I][J] (F4 float4 per thread) fit in the registers
  // beside the accumulators only for TB = 128
  static constexpr bool PREFETCH = TB == 128;
};

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
template <int N, int NF>
__device__ __forceinline__ void lgkm_wait_for(v4i (&f)[NF]) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  if constexpr (NF == 4) {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]) : "i"(N));
  } else {
    static_assert(NF == 6, "four or six fragments");
    asm volatile("s_waitcnt lgkmcnt(%6)"
                 : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5])
                 : "i"(N));
  }
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

template <int TB>
__global__ __launch_bounds__(NT_S, 1) void aog_syrk_kernel(const uint16_t* __restrict__ gT, float* __restrict__ A,
                                                          int d, int n) {
  using Cf = SyrkCfg<TB>;
  constexpr int BW = Cf::BW, NST = Cf::NST, CPW = Cf::CPW, IPS = Cf::IPS, LDC = Cf::LDC, F4 = Cf::F4;
  // the ring of NST stages; after the main loop, the epilogue tile
  __shared__ __attribute__((aligned(16))) uint8_t smem[Cf::SMEM_B];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = (wave >> 1) & 1, wn = wave & 1;       // block of the tile
  const int kh = wave >> 2;                            // half of the k-steps of a stage
  const int T = (d + TB - 1) / TB;
  int ti, tj;
  triangle_tile(blockIdx.x, T, ti, tj);
  const int m0 = ti * TB, n0 = tj * TB;
  const uint32_t RB = static_cast<uint32_t>(n) * 2u;   // bytes per row of gT
  const int S = n / KS;

  // LDS-DMA: copy i (0..CPW-1) of wave w fills rows 8*(CPW*w+i) .. +7 of a
  // tile, lane l taking row 8*(CPW*w+i) + l/8 and slot l%8, which holds chunk
  // (l%8) ^ swz(row)
  const buf_rsrc a_rsrc = make_rsrc(gT + static_cast<int64_t>(m0) * n, static_cast<uint32_t>(min(TB, d - m0)) * RB);
  const buf_rsrc b_rsrc = make_rsrc(gT + static_cast<int64_t>(n0) * n, static_cast<uint32_t>(min(TB, d - n0)) * RB);
  uint32_t d_off[CPW];
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int row = 8 * (CPW * wave + i) + (lane >> 3);
    d_off[i] = static_cast<uint32_t>(row) * RB + static_cast<uint32_t>(((lane & 7) ^ swz_s(row)) * 16);
  }
  auto stage_a = [&](int k) __attribute__((always_inline)) { return smem + k * Cf::STAGE_B; };
  auto stage_b = [&](int k) __attribute__((always_inline)) { return smem + k * Cf::STAGE_B + TB * ROWB_S; };
  auto issue = [&](int s, int k) __attribute__((always_inline)) {
    const uint32_t ko = static_cast<uint32_t>(s) * ROWB_S;
#pragma unroll
    for (int i = 0; i < CPW; ++i) buf_load16_lds(a_rsrc, d_off[i] + ko, stage_a(k) + (CPW * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < CPW; ++i) buf_load16_lds(b_rsrc, d_off[i] + ko, stage_b(k) + (CPW * wave + i) * 1024);
  };

  v16f_s acc[BW][BW];
#pragma unroll
  for (int i = 0; i < BW; ++i)
#pragma unroll
    for (int j = 0; j < BW; ++j) acc[i][j] = v16f_s{};

  // v_mfma_f32_32x32x16_bf16 operands: lane l holds row l%32 and the 8
  // consecutive k of half l/32 of a 16-wide k step, i.e. chunk 2q + l/32 of
  // the row in step q
  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int frow_off = frow * ROWB_S;
  const int fslot = fhalf ^ swz_s(frow);

  // With TB = 128 the epilogue's reads of A[I][J] are issued right after the
  // last stage's copies (step S - NST), so that their latency hides behind the
  // last stages: thread t holds float4 number t + NT_S q (q < F4) of the tile, row
  // (t + NT_S q) / (TB/4), columns 4 ((t + NT_S q) % (TB/4)) .. +3.  Interior
  // off-diagonal tiles only.
  const bool diag = ti == tj;
  const bool fast = m0 + TB <= d && n0 + TB <= d && !diag;
  const bool pref = Cf::PREFETCH && fast && S >= NST;
  const buf_rsrc A_rsrc = make_rsrc(A, 0xFFFFFFFFu);
  auto f4_row = [&](int q) __attribute__((always_inline)) { return (tid + NT_S * q) / (TB / 4); };
  auto f4_col = [&](int q) __attribute__((always_inline)) { return 4 * ((tid + NT_S * q) % (TB / 4)); };
  float4 pn[F4];
  auto load_block = [&](int r0, int c0, float4 (&dst)[F4]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < F4; ++q)
      dst[q] = __builtin_bit_cast(
          float4, buf_load16(A_rsrc, (static_cast<uint32_t>(r0 + f4_row(q)) * d + c0 + f4_col(q)) * 4u));
  };

  // stage s (slot k = s % NST): wait for this wave's copies of stage s (those
  // of the next NST - 2 stages, when issued, may stay in flight, and after
  // step S - NST the F4 reads of A), barrier, then refill the slot of stage
  // s-1 (every wave is past it) with stage s + NST - 1
  auto stage_wait = [&](int s) __attribute__((always_inline)) {
    const bool after = pref && s > S - NST;
    if constexpr (NST == 4) {
      if (s + 2 < S) {
        if (after) wait_vmcnt<2 * IPS + F4>();
        else wait_vmcnt<2 * IPS>();
      } else if (s + 1 < S) {
        if (after) wait_vmcnt<IPS + F4>();
        else wait_vmcnt<IPS>();
      } else {
        if (after) wait_vmcnt<F4>();
        else wait_vmcnt<0>();
      }
    } else {
      if (s + 1 < S) {
        if (after) wait_vmcnt<IPS + F4>();
        else wait_vmcnt<IPS>();
      } else {
        if (after) wait_vmcnt<F4>();
        else wait_vmcnt<0>();
      }
    }
  };
  auto stage_step = [&](int s, int k) __attribute__((always_inline)) {
    stage_wait(s);
    lds_barrier();
    if (s + NST - 1 < S) issue(s + NST - 1, (k + NST - 1) % NST);
    if (pref && s == S - NST) load_block(m0, n0, pn);
    // fragments of the wave's next k-step are read while the current one multiplies
    const uint32_t a_base = lds_addr(stage_a(k)) + (wm * (TB / 2)) * ROWB_S + frow_off;
    const uint32_t b_base = lds_addr(stage_b(k)) + (wn * (TB / 2)) * ROWB_S + frow_off;
    v4i fr[2][2 * BW];
    auto read_step = [&](int q, v4i (&f)[2 * BW]) __attribute__((always_inline)) {
      const uint32_t so = static_cast<uint32_t>(((2 * q) ^ fslot) * 16);
#pragma unroll
      for (int i = 0; i < BW; ++i) f[i] = lds_read16(a_base + so + i * 32 * ROWB_S);
#pragma unroll
      for (int j = 0; j < BW; ++j) f[BW + j] = lds_read16(b_base + so + j * 32 * ROWB_S);
    };
    // this wave's k-steps of the stage: KH consecutive 16-wide steps from kh * KH
    constexpr int KH = KS / 16 / 2;
    read_step(kh * KH, fr[0]);
#pragma unroll
    for (int q = 0; q < KH; ++q) {
      v4i(&f)[2 * BW] = fr[q & 1];
      if (q + 1 < KH) {
        read_step(kh * KH + q + 1, fr[(q + 1) & 1]);
        lgkm_wait_for<2 * BW>(f);
      } else {
        lgkm_wait_for<0>(f);
      }
#pragma unroll
      for (int i = 0; i < BW; ++i)
#pragma unroll
        for (int j = 0; j < BW; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, f[i]),
                                                              __builtin_bit_cast(v8bf, f[BW + j]), acc[i][j], 0, 0, 0);
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

  // ---- epilogue: A[I][J] += C, then A[J][I] += C^T, through LDS ----
  // C is staged in LDS ([row][LDC] floats), then transposed in place, and
  // each pass moves 16 bytes per lane along rows of A.  A diagonal tile
  // (I = J) is one pass over its block: element (r, c) gets C[r][c] for
  // r <= c and C[c][r] below the diagonal.  Blocks past d are skipped float4
  // by float4 (d % 16 == 0, so a float4 is all in or all out).
  float* C = reinterpret_cast<float*>(smem);
  // result layout of a 32x32 block: lane l holds column l%32 and rows
  // 8*(v/4) + 4*(l/32) + v%4, v = 0..15
  // with `add`, the block already in C (the other k-half's, same element
  // positions) is first added to the accumulators
  auto stage_tile = [&](bool add) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < BW; ++i)
#pragma unroll
      for (int j = 0; j < BW; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = wm * (TB / 2) + i * 32 + 8 * (v >> 2) + 4 * fhalf + (v & 3);
          const int c = wn * (TB / 2) + j * 32 + frow;
          float* e = &C[r * LDC + c];
          if (add) acc[i][j][v] += *e;
          *e = acc[i][j][v];
        }
  };
  auto in_range = [&](int r0, int c0, int q) __attribute__((always_inline)) {
    return r0 + f4_row(q) < d && c0 + f4_col(q) < d;
  };
  auto load_ranged = [&](int r0, int c0, float4 (&dst)[F4]) __attribute__((always_inline)) {
    if (fast) {
      load_block(r0, c0, dst);
    } else {
#pragma unroll
      for (int q = 0; q < F4; ++q) {
        dst[q] = float4{0.0f, 0.0f, 0.0f, 0.0f};
        if (in_range(r0, c0, q))
          dst[q] = __builtin_bit_cast(
              float4, buf_load16(A_rsrc, (static_cast<uint32_t>(r0 + f4_row(q)) * d + c0 + f4_col(q)) * 4u));
      }
    }
  };
  auto add_store = [&](int r0, int c0, const float4 (&cur)[F4]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < F4; ++q) {
      const int r = f4_row(q), c = f4_col(q);
      float4 cv = *reinterpret_cast<const float4*>(C + r * LDC + c);
      if (diag) {                                  // below the diagonal: the mirrored element
        if (r > c) cv.x = C[c * LDC + r];
        if (r > c + 1) cv.y = C[(c + 1) * LDC + r];
        if (r > c + 2) cv.z = C[(c + 2) * LDC + r];
        if (r > c + 3) cv.w = C[(c + 3) * LDC + r];
      }
      const float4 o = {cur[q].x + cv.x, cur[q].y + cv.y, cur[q].z + cv.z, cur[q].w + cv.w};
      if (fast || in_range(r0, c0, q))
        *reinterpret_cast<float4*>(A + static_cast<int64_t>(r0 + r) * d + c0 + c) = o;
    }
  };

  lds_barrier();                                   // every wave is past the ring
  // C = first k-half + second k-half: the second half's waves stage their
  // blocks, then each first-half thread adds the elements it owns (the same
  // positions) into its accumulators and stores the sums in their place.
  // Every thread then requests its share of both blocks of A, so that the
  // reads of A[J][I] overlap the first pass.
  if (kh == 1) stage_tile(false);
  __syncthreads();
  if (kh == 0) stage_tile(true);
  asm volatile("" ::: "memory");                 // the reads of A stay after the staging
  float4 pt[F4];
  if (!pref) load_ranged(m0, n0, pn);
  if (!diag) load_ranged(n0, m0, pt);
  __syncthreads();
  add_store(m0, n0, pn);
  if (diag) return;
  // C transposed in place: each thread takes half of the elements of its
  // block positions (the k-half picks the half), all read before any is
  // written back at its transposed position
  float tv[BW][BW][8];
#pragma unroll
  for (int i = 0; i < BW; ++i)
#pragma unroll
    for (int j = 0; j < BW; ++j)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int v = 8 * kh + u;
        const int r = wm * (TB / 2) + i * 32 + 8 * (v >> 2) + 4 * fhalf + (v & 3);
        tv[i][j][u] = C[r * LDC + wn * (TB / 2) + j * 32 + frow];
      }
  __syncthreads();                                 // every thread is done reading C
#pragma unroll
  for (int i = 0; i < BW; ++i)
#pragma unroll
    for (int j = 0; j < BW; ++j)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int v = 8 * kh + u;
        const int r = wm * (TB / 2) + i * 32 + 8 * (v >> 2) + 4 * fhalf + (v & 3);
        C[(wn * (TB / 2) + j * 32 + frow) * LDC + r] = tv[i][j][u];
      }
  __syncthreads();
  add_store(n0, m0, pt);
}

static int syrk_tiles(int d, int tb) {
  const int T = (d + tb - 1) / tb;
  return T * (T + 1) / 2;
}

hipError_t launch_aog_accumulate(int d, int n, const uint16_t* gT, float* A, hipStream_t stream) {
  // 192-row tiles when they fit in one round on the 256 CUs and 128-row ones do not
  if (syrk_tiles(d, 128) > 256 && syrk_tiles(d, 192) <= 256)
    hipLaunchKernelGGL(aog_syrk_kernel<192>, dim3(syrk_tiles(d, 192)), dim3(NT_S), 0, stream, gT, A, d, n);
  else
    hipLaunchKernelGGL(aog_syrk_kernel<128>, dim3(syrk_tiles(d, 128)), dim3(NT_S), 0, stream, gT, A, d, n);
  return hipGetLastError();
}

}  // namespace qwam
