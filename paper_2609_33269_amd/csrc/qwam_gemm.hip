// The ASP GEMM: W4A4 integer group partial sums on FP6 matrix cores (exact),
// float32 per-group scaling in registers, and the bf16 low-rank branch + bias
// fused in the epilogue (the second kernel of App. B.1; Eq. 2 and Eq. 9).
//
//   y[m, n] = bf16( sum_g xs[g][m] ws[g][n] * P[m, n, g]
//                   + sum_j t[m, j] L2t[n, j] + bias[n] )
//
// Work decomposition (gfx950, 256 CUs in 8 XCDs, 64-wide waves):
//   * a 256-thread workgroup (4 waves) owns a 128 x 128 tile of y; two
//     workgroups share a CU (2 waves per SIMD), so one workgroup's barrier and
//     LDS waits are covered by the other's work;
//   * the packed 4-bit codes stay packed all the way into LDS: a ring stage
//     holds four consecutive groups, i.e. one 128-byte line of every packed row
//     of the A and B tiles (128 rows each) plus their scales, copied straight
//     from HBM/L2 into LDS by buffer_load ... lds (no VGPR staging, zero past
//     the valid rows).  Eight lanes cover one line, so a 64-lane copy touches
//     8 cache lines: the vector-memory address path (about one line per clock
//     per CU) is what limits a copy of one 16-byte piece per row and group;
//   * two stages: stage s+1 is copied while stage s is multiplied, one barrier
//     per stage; each tile and scale array of a stage is an LDS variable of
//     its own, so that the compiler can tell a copy into one stage from a read
//     of the other and does not make the read wait for the copy;
//   * inside a stage, row r keeps its eight 16-byte chunks in slot order
//     chunk ^ swz(r), swz(r) = (r & 7) ^ ((r >> 3) & 1), so that the fragment
//     loads (one ds_read_b128 = 32 codes of one row per lane, 32 consecutive
//     rows per half-wave) hit distinct banks;
//   * wave (wm, wn) owns rows 64*wm.. and columns 64*wn.. as 2 x 2 blocks of
//     v_mfma_scale_f32_32x32x64_f8f6f4 (FP6 e2m3 operands, one 64-channel
//     span per instruction, twice the FP8 rate), with the weight rows as the
//     A operand and the activation rows as the B operand, so that a block's
//     result holds y transposed (lane l: token l%32, and four consecutive
//     output columns per result quarter); lane l of an operand holds its row
//     l%32 and half l/32 of the span.  A code block (16 codes in two words, qwam.h)
//     turns into three operand words with four ANDs: each 6-bit field is then
//     sign | |code| in the mantissa field, the e2m3 subnormal code / 8.  The
//     E8M0 scales (2^3 on each side) cancel the 2^-6, so the float32 result is
//     the integer partial P itself, exactly (|P| <= 3136);
//   * the per-output scale products sw[n] * sx[m] of a group are an outer
//     product: one v_mfma_f32_32x32x4_2b_bf16 over two-piece bf16 splits of
//     the scales (scale_outer, within about 2^-15 of the float32 product)
//     gives them for two 32 x 32 blocks at once, in the result layout of the
//     integer blocks, so the VALU is left with one fused multiply-add per
//     output and group;
//   * group 64 runs as a software pipeline across groups: every MFMA is
//     followed by VALU work that does not depend on it (the updates of blocks
//     whose products landed earlier, the unpacking of the next group);
//   * workgroups are mapped XCD-major: the 8 XCDs each take a contiguous range
//     of tiles, ordered in bands of 8 tile-rows so that the concurrently
//     resident tiles of one XCD share their A and B panels in its L2;
//   * the accumulators start from the bias plus the bf16 branch
//     (v_mfma_f32_32x32x16_bf16, same result layout as the integer blocks),
//     computed while the first stage is copied; the epilogue rounds to bf16
//     (v_cvt_pk_bf16_f32), and one v_permlane32_swap per pair of result words
//     gives every lane 8 consecutive columns of its token, so each lane stores
//     16 contiguous bytes straight from registers (no LDS, no barrier).
//
// Group 32 (GS = 32, the paper's setting): the MFMA's K = 64 covers two groups,
// one per lane half, and each lane's E8M0 scale governs its own 32 values.
// Each block runs twice, once per group, with the other lane half's scales set
// to 2^-127 on both operands: its products (2^-254 and below) underflow to
// zero, so each result is one group's integer partial, exactly.  Twice the
// MFMA work and twice the scaling per output.
#include <type_traits>

#include "qwam_device.h"
#include "qwam_internal.h"
#include "qwam_mfma.h"

namespace qwam {

namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int NWAVES = 4;
constexpr int NT = 64 * NWAVES;
constexpr int WG_PER_CU = 2;
constexpr int BAND = 8;            // tile-rows per band of the tile order
constexpr int KC = 4;              // groups per ring stage
constexpr int ROWB = KC * 32;      // bytes of one packed row per stage (one cache line)

// One ring stage: the A and B tiles ([row][8 chunk slots of 16 bytes],
// swizzled) and the scales of its GPS scale groups.  Each array is its own
// LDS variable: the compiler then keeps the copies into one stage apart from
// the reads of the other and does not make those reads wait for the copies.
template <int GPS>
struct StageRef {
  uint8_t* a;
  uint8_t* b;
  float (*sx)[BM];
  uint32_t (*sw)[BN];   // the weight scales as bf16 pieces hi | lo << 16
};
static_assert(BM == BN && BM * 64 * 2 <= BM * ROWB,
              "the tile's rows of t and L2t (up to rank 64) must fit in one tile buffer of a stage");

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// waits for this wave's LDS reads, then a workgroup barrier (outstanding
// global-to-LDS copies stay in flight)
__device__ __forceinline__ void lds_wait_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// chunk slot permutation of a row inside a stage
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// LDS reads that the compiler keeps in program order (volatile)
__device__ __forceinline__ uint4 lds_load16_volatile(const uint8_t* p) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  typedef const volatile __attribute__((address_space(3))) v4u lds_v4u;
  const v4u v = *(lds_v4u*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float lds_load4_volatile(const float* p) {
  typedef const volatile __attribute__((address_space(3))) float lds_f;
  return *(lds_f*)(p);
}
__device__ __forceinline__ uint32_t lds_load4_volatile(const uint32_t* p) {
  typedef const volatile __attribute__((address_space(3))) uint32_t lds_u;
  return *(lds_u*)(p);
}

// bf16 bits of (a, b) rounded to nearest even, a in the low half
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v2f{a, b}, v2bf));
}

// The scale products sw * sx of two 32 x 32 blocks (lane l: sw of the weight
// row l%32 (A side), sx of the token l%32 of B block l/32), in the result
// layout of the integer blocks.  Each scale is split into two bf16 pieces,
// hi = bf16(s) and lo = bf16(s - hi) (the difference is exact in float32), and
// one v_mfma_f32_32x32x4_2b_bf16 sums the four exact products of
// [hi, lo, hi, lo] (sw, the packed pieces hi | lo << 16 the weight pack wrote,
// twice) and [hi, hi, lo, lo] (sx, split here) in float32.  That is the product
// of the two 16-bit splits, each within 2^-16 of its scale, so the result is
// within about 2^-15 of sw * sx.  Unlike the float32 outer-product MFMA, the
// bf16 one lets the SIMD issue VALU work while it runs.
__device__ __forceinline__ v32f scale_outer(uint32_t wpieces, float sx) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  const uint32_t hx = bf16_pair(sx, sx);
  const float lo_x = sx - __builtin_bit_cast(float, hx << 16);
  const uint32_t lx = bf16_pair(lo_x, lo_x);
  const v4s a = __builtin_bit_cast(v4s, static_cast<uint64_t>(wpieces) | (static_cast<uint64_t>(wpieces) << 32));
  const v4s b = __builtin_bit_cast(v4s, static_cast<uint64_t>(hx) | (static_cast<uint64_t>(lx) << 32));
  return __builtin_amdgcn_mfma_f32_32x32x4bf16_1k(a, b, v32f{}, 0, 0, 0);
}

// Tile of workgroup `bid`: XCD-major remap (hardware places workgroup b on XCD
// b % 8), then bands of BAND tile-rows, columns fastest inside a band-column.
// (An XCD owning a range of whole tile-columns instead, so that its weight
// panel stays in its L2, fetched twice the bytes: a 2.7 MB panel plus the
// streaming activation tiles and the output does not stay in a 4 MB L2.)
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

template <int RANK, bool PARTIALS, int GS>
__global__ __launch_bounds__(NT, WG_PER_CU) void asp_gemm_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ xs, const uint16_t* __restrict__ t,
    const uint8_t* __restrict__ wq, const uint32_t* __restrict__ wsp, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ P, int M,
    int N, int K) {
  constexpr int NS = kGroup / GS;                               // scale groups per 64-channel span
  constexpr int GPS = KC * NS;                                  // scale groups per stage
  typedef StageRef<GPS> Stage;
  __shared__ __attribute__((aligned(16))) uint8_t lds_a0[BM * ROWB], lds_b0[BN * ROWB];
  __shared__ __attribute__((aligned(16))) uint8_t lds_a1[BM * ROWB], lds_b1[BN * ROWB];
  __shared__ __attribute__((aligned(16))) float lds_sx0[GPS][BM], lds_sx1[GPS][BM];
  __shared__ __attribute__((aligned(16))) uint32_t lds_sw0[GPS][BN], lds_sw1[GPS][BN];
  const Stage st0{lds_a0, lds_b0, lds_sx0, lds_sw0};
  const Stage st1{lds_a1, lds_b1, lds_sx1, lds_sw1};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (SGPR)
  const int wm = wave >> 1, wn = wave & 1;                      // 2 x 2 waves
  const int G = K / kGroup;                                     // 64-channel spans
  const int GSC = K / GS;                                       // scale groups
  const int KB = K / 2;
  const int S = (G + KC - 1) / KC;                              // ring stages
  const int S_full = G / KC;                                    // stages with KC groups

  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  // ---- LDS-DMA assignment: copy i (0..3) of wave w fills rows 8*(4w+i) .. +7
  // of a tile, lane l taking row 8*(4w+i) + l/8 and LDS slot l%8, which holds
  // the row's chunk (l%8) ^ swz(row) ----
  const buf_rsrc a_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * KB,
                                    static_cast<uint32_t>(min(BM, M - m0)) * KB);
  const buf_rsrc b_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB,
                                    static_cast<uint32_t>(min(BN, N - n0)) * KB);
  uint32_t d_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 8 * (4 * wave + i) + (lane >> 3);
    d_off[i] = static_cast<uint32_t>(row * KB + (((lane & 7) ^ swz(row)) * 16));
  }
  // scales: waves 0-1 copy xs of the tile's rows, waves 2-3 the weight-scale
  // pieces (wsp) of its columns;
  // copy i of such a wave covers scale group (GPS/2 * (w%2) + i/2) of the
  // stage, rows 64*(i%2) .. +63
  const bool s_is_x = wave < 2;
  const buf_rsrc s_rsrc = s_is_x ? make_rsrc(xs, static_cast<uint32_t>(GSC) * M * 4u)
                                 : make_rsrc(wsp, static_cast<uint32_t>(GSC) * N * 4u);
  const uint32_t s_stride = static_cast<uint32_t>(s_is_x ? M : N) * 4u;
  uint32_t s_off[GPS];
#pragma unroll
  for (int i = 0; i < GPS; ++i) {
    const int q = (GPS / 2) * (wave & 1) + (i >> 1);
    s_off[i] = static_cast<uint32_t>(q) * s_stride +
               static_cast<uint32_t>((s_is_x ? m0 : n0) + (i & 1) * 64 + lane) * 4u;
  }

  auto issue = [&](int s, const Stage& st) __attribute__((always_inline)) {
    const uint32_t ko = static_cast<uint32_t>(s) * ROWB;
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(a_rsrc, d_off[i] + ko, st.a + (4 * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load16_lds(b_rsrc, d_off[i] + ko, st.b + (4 * wave + i) * 1024);
    if (!PARTIALS) {
      const uint32_t so = static_cast<uint32_t>(s) * GPS * s_stride;
#pragma unroll
      for (int i = 0; i < GPS; ++i) {
        const int q = (GPS / 2) * (wave & 1) + (i >> 1);
        buf_load4_lds(s_rsrc, s_off[i] + so,
                      s_is_x ? static_cast<void*>(&st.sx[q][(i & 1) * 64])
                             : static_cast<void*>(&st.sw[q][(i & 1) * 64]));
      }
    }
  };

  v16f accf[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) accf[i][j] = v16f{};

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int rsub = fhalf * 4;
  // byte offset of this lane's row inside a 32-row block; slot of chunk
  // 2q + fhalf is (2q) ^ fslot (the block bases are multiples of 16 rows, so
  // swz depends on frow only)
  const int frow_off = frow * ROWB;
  const int fslot = fhalf ^ swz(frow);

  // LDS data of one 64-channel span: packed A / B fragments (16 bytes, the
  // lane's half of the span: A from the weight tile, B from the activation
  // tile) and the lane's scales (NS groups): the weight scale of row l%32 of
  // each A block (A operand of the scale product) and the activation scale of
  // row l%32 of B block l/32 (B operand).
  struct GroupData {
    uint4 a[2], b[2];
    uint32_t sa[2][NS];   // weight-scale pieces of the A blocks
    float sb[NS];         // activation scale of the B-side token
  };
  // Reads group q's data one group ahead of its use.  The loads are volatile
  // and followed by a compiler-only fence, so they are issued here and not
  // sunk next to their first use; the wait for them lands at that use.
  auto load_frag = [&](const uint8_t* rowp, int q) __attribute__((always_inline)) {
    if constexpr (GS == 64) return *reinterpret_cast<const uint4*>(rowp + ((2 * q) ^ fslot) * 16);
    else return lds_load16_volatile(rowp + ((2 * q) ^ fslot) * 16);
  };
  auto load_group = [&](const Stage& cur, int q) __attribute__((always_inline)) {
    GroupData d;
#pragma unroll
    for (int i = 0; i < 2; ++i) d.a[i] = load_frag(cur.b + (wn * 64 + i * 32) * ROWB + frow_off, q);
#pragma unroll
    for (int j = 0; j < 2; ++j) d.b[j] = load_frag(cur.a + (wm * 64 + j * 32) * ROWB + frow_off, q);
    if (!PARTIALS) {
#pragma unroll
      for (int h = 0; h < NS; ++h) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const uint32_t* p = &cur.sw[NS * q + h][wn * 64 + i * 32 + frow];
          d.sa[i][h] = GS == 64 ? *p : lds_load4_volatile(p);
        }
        const float* p = &cur.sx[NS * q + h][wm * 64 + fhalf * 32 + frow];
        d.sb[h] = GS == 64 ? *p : lds_load4_volatile(p);
      }
    }
    asm volatile("" ::: "memory");
    return d;
  };

  // block (i, j) of group g, scale group h of the span: acc += P * sw * sx
  // (the partials themselves with PARTIALS).  Result layout of a 32x32 block
  // (i: weight block, j: activation block): lane l holds token l%32 of block j
  // and output columns 8*(v/4) + 4*(l/32) + v%4 of block i, v = 0..15.
  auto update = [&](int i, int j, int g, int h, const v16f& p, const v32f& sc) __attribute__((always_inline)) {
    if (PARTIALS) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int n = n0 + wn * 64 + i * 32 + 8 * (v >> 2) + rsub + (v & 3);
        const int m = m0 + wm * 64 + j * 32 + frow;
        if (m < M && n < N) P[(static_cast<int64_t>(m) * N + n) * GSC + NS * g + h] = static_cast<int32_t>(p[v]);
      }
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) accf[i][j][v] = __builtin_fmaf(p[v], sc[16 * j + v], accf[i][j][v]);
    }
  };

  // one group g of a stage, from its LDS data (group 32)
  auto group = [&](int g, const GroupData& d) __attribute__((always_inline)) {
    v8i af[2], bf[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) af[i] = codes_to_fp6(d.a[i]);
#pragma unroll
    for (int j = 0; j < 2; ++j) bf[j] = codes_to_fp6(d.b[j]);

    // the exact integer partial of block (i, j) for group h of the span, as
    // float32 (group 64: the whole span; group 32: the other lane half's
    // scales are 2^-127 on both operands, so its products underflow to zero)
    auto mfma_block = [&](int i, int j, int h) __attribute__((always_inline)) {
      int sc = kE8M0Code;
      if constexpr (GS == 32) sc = ((lane >> 5) == h) ? kE8M0Code : 0;
      return fp6_partial(af[i], bf[j], sc, sc);
    };
    // scale products of row block i and both column blocks, group h:
    // registers 0-15 belong to column block 0, 16-31 to column block 1
    auto scale_block = [&](int i, int h) __attribute__((always_inline)) {
      return scale_outer(d.sa[i][h], d.sb[h]);
    };
    // per group h and row block i: the scale products (one MFMA for both
    // column blocks), the two integer blocks, then their updates; each update
    // reads results issued at least one MFMA earlier
    const v32f none = {};
#pragma unroll
    for (int h = 0; h < NS; ++h)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const v32f sc = PARTIALS ? none : scale_block(i, h);
        const v16f p0 = mfma_block(i, 0, h);
        const v16f p1 = mfma_block(i, 1, h);
        update(i, 0, g, h, p0, sc);
        update(i, 1, g, h, p1, sc);
      }
  };

  // one stage: `cur` holds stage s (groups KC*s ..), `nxt` (the stage of s-1)
  // receives s+1; nq groups of the stage are valid
  auto stage_step = [&](int s, const Stage& cur, const Stage& nxt, int nq) __attribute__((always_inline)) {
    wait_vmcnt<0>();                  // this thread's copies of stage s have landed
    lds_barrier();                    // ... and every thread's; stage s-1 is fully consumed
    issue(s + 1, nxt);                // past the last stage: harmless reads, never used
    GroupData d = load_group(cur, 0);
#pragma unroll
    for (int q = 0; q < KC; ++q) {
      if (q < nq) {
        GroupData next = d;
        if (q + 1 < nq) next = load_group(cur, q + 1);
        group(s * KC + q, d);
        d = next;
      }
    }
  };

  issue(0, st0);
  // The accumulators start from the bias and the low-rank branch t . L2
  // (v_mfma_f32_32x32x16_bf16 with L2t as the A operand and t as the B
  // operand, the roles of the integer blocks: lane l holds row / column l%32
  // and the 8 rank slots 8*(l/32) .. +7 of a 16-wide rank step, the same slots
  // for both).  The tile's rows of t and L2t and its bias come into the
  // second stage's buffers (idle until stage 1 is copied) by the same LDS DMA
  // as the codes, alongside stage 0: t rows [128][RANK] over the A tile, L2t
  // rows over the B tile, the 128 bias values over the activation scales.
  // Result register v of block (i, j) is output column
  // n0 + 64 wn + 32 i + 8 (v/4) + 4 (l/32) + v%4, so each lane takes the bias
  // of four consecutive columns per v/4.
  if (!PARTIALS) {
    constexpr int RB2 = RANK * 2;                 // bytes of one row of t / L2t
    const buf_rsrc t_rsrc = make_rsrc(t + static_cast<int64_t>(m0) * RANK,
                                      static_cast<uint32_t>(min(BM, M - m0)) * RB2);
    const buf_rsrc l_rsrc = make_rsrc(L2t + static_cast<int64_t>(n0) * RANK,
                                      static_cast<uint32_t>(min(BN, N - n0)) * RB2);
    // 128 rows of RB2 bytes = RANK / 16 kilobyte pieces per wave and array
#pragma unroll
    for (int c = 0; c < RANK / 16; ++c) {
      const int piece = wave * (RANK / 16) + c;   // kilobyte of the array
      const uint32_t src = static_cast<uint32_t>(piece * 1024 + lane * 16);
      buf_load16_lds(t_rsrc, src, st1.a + piece * 1024);
      buf_load16_lds(l_rsrc, src, st1.b + piece * 1024);
    }
    if (wave == 0) {
      const buf_rsrc b_rsrc = make_rsrc(bias != nullptr ? bias + n0 : nullptr,
                                        bias != nullptr ? static_cast<uint32_t>(min(BN, N - n0)) * 2u : 0u);
      buf_load4_lds(b_rsrc, static_cast<uint32_t>(lane * 4), &st1.sx[0][0]);
    }
    wait_vmcnt<0>();
    lds_wait_barrier();
    constexpr int KSTEPS = RANK / 16;
    const int kk = fhalf * 16;                    // byte offset of the lane's 8 rank slots
    const uint16_t* bias_lds = reinterpret_cast<const uint16_t*>(&st1.sx[0][0]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        v16f c;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const uint2 w = *reinterpret_cast<const uint2*>(bias_lds + wn * 64 + i * 32 + 8 * q4 + rsub);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t word = (e & 2) ? w.y : w.x;
            c[4 * q4 + e] = __builtin_bit_cast(float, (e & 1) ? (word & 0xFFFF0000u) : (word << 16));
          }
        }
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
          const v8s lf = *reinterpret_cast<const v8s*>(st1.b + (wn * 64 + i * 32 + frow) * RB2 + s * 32 + kk);
          const v8s tf = *reinterpret_cast<const v8s*>(st1.a + (wm * 64 + j * 32 + frow) * RB2 + s * 32 + kk);
          c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, lf), __builtin_bit_cast(v8bf, tf), c,
                                                      0, 0, 0);
        }
        accf[i][j] = c;
      }
    // every wave has read the branch operands before stage 1 is copied over them
    lds_wait_barrier();
  }

  if constexpr (GS == 32 && PARTIALS) {
    int s = 0;
    for (; s + 1 < S_full; s += 2) {
      stage_step(s, st0, st1, KC);
      stage_step(s + 1, st1, st0, KC);
    }
    // at most one full stage and one partial stage remain
    if (s < S_full) {
      stage_step(s, st0, st1, KC);
      ++s;
      if (s < S) stage_step(s, st1, st0, G - s * KC);
    } else if (s < S) {
      stage_step(s, st0, st1, G - s * KC);
    }
  } else if constexpr (GS == 32) {
    // every stage runs all KC spans: a span past K reads finite FP6 codes (the
    // next row's, or zeros past the buffer) with scales of zero (its scale
    // groups lie past the scale arrays, where the buffer loads return zero),
    // so it adds exactly zero; the single loop body keeps the registers of a
    // partial-stage tail out of the kernel
    int s = 0;
    for (; s + 1 < S; s += 2) {
      stage_step(s, st0, st1, KC);
      stage_step(s + 1, st1, st0, KC);
    }
    if (s < S) stage_step(s, st0, st1, KC);
  } else {
    // Group 64: a software pipeline across groups.  The matrix core runs one
    // MFMA at a time and a wave that issues an MFMA while the previous one is
    // still running waits for it, so every MFMA gets its own slot, followed by
    // 16-20 VALU instructions that do not depend on it: the updates of blocks
    // whose products landed one slot or more earlier, or the unpacking of
    // fragments (8 instructions each, split in halves to even out the
    // slots).  Per group g (S = scale products, P = integer partials):
    //   slot 1  S0(g)              | update (1,1) of g-1; 1/2 A1(g)
    //   slot 2  P00(g) = A0 x B0   | B1(g); 1/2 A1(g)
    //   slot 3  P01(g) = A0 x B1   | LDS reads of g+1; update (0,0)
    //   slot 4  S1(g)              | update (0,1); 1/2 A0(g+1)
    //   slot 5  P10(g) = A1 x B0   | 1/2 A0(g+1); 1/2 B0(g+1)
    //   slot 6  P11(g) = A1 x B1   | update (1,0); 1/2 B0(g+1)
    // A stage ends inside its last group: before the LDS reads of g+1 the
    // wave waits for its copies of the next stage and for its own LDS reads,
    // then the barrier frees the stage just read for the copy of the stage
    // after next.
    struct Pipe {
      v8i af0, bf0;        // unpacked A0 / B0 fragments of the current group
      uint4 ra1, rb1;      // packed A1 / B1 fragments of the current group
      uint32_t sa0, sa1;   // its weight-scale pieces
      float sb;            // and activation scale
      v32f s1;             // scale products and partial of block (1, 1) of
      v16f p11;            // the previous group, updated in slot 1
    };
    auto span_partial = [&](const v8i& a, const v8i& b) __attribute__((always_inline)) {
      return fp6_partial(a, b, kE8M0Code, kE8M0Code);
    };
    auto scale_products = [&](uint32_t sa, float sb) __attribute__((always_inline)) {
      if constexpr (PARTIALS) return v32f{};
      else return scale_outer(sa, sb);
    };
    auto start = [&](Pipe& pp, const GroupData& d) __attribute__((always_inline)) {
      pp.af0 = codes_to_fp6(d.a[0]);
      pp.bf0 = codes_to_fp6(d.b[0]);
      pp.ra1 = d.a[1];
      pp.rb1 = d.b[1];
      if (!PARTIALS) { pp.sa0 = d.sa[0][0]; pp.sa1 = d.sa[1][0]; pp.sb = d.sb[0]; }
    };
    // group g at position q (0..7) of two consecutive stages: q < 4 reads
    // st0, q >= 4 st1; the last group of a stage (q % 4 == 3) switches the
    // ring, issuing stage s_next into the buffer it has just finished
    // half of an unpack: code block (w0, w1) -> operand words 3h .. 3h+2 of r
    // (words 6-7 are not read with FP6 operands and stay unset)
    auto unpack_half = [&](v8i& r, int h, uint32_t w0, uint32_t w1) __attribute__((always_inline)) {
      r[3 * h] = static_cast<int>(w0 & ~kFp6Z0);
      r[3 * h + 1] = static_cast<int>(w1 & ~kFp6Z1);
      r[3 * h + 2] = static_cast<int>((w0 & kFp6Z0) | (w1 & kFp6Z1));
    };
    auto step = [&](auto qc, int g, Pipe& pp, int s_next) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      // slot 1: S0 | update (1,1) of g-1, half of A1
      const v32f s0 = scale_products(pp.sa0, pp.sb);
      __builtin_amdgcn_sched_barrier(0);
      if (!PARTIALS || g > 0) update(1, 1, g - 1, 0, pp.p11, pp.s1);
      v8i af1, bf1, af0n, bf0n;
      unpack_half(af1, 0, pp.ra1.x, pp.ra1.y);
      __builtin_amdgcn_sched_barrier(0);
      // slot 2: P00 | B1, other half of A1
      const v16f p00 = span_partial(pp.af0, pp.bf0);
      __builtin_amdgcn_sched_barrier(0);
      unpack_half(bf1, 0, pp.rb1.x, pp.rb1.y);
      unpack_half(bf1, 1, pp.rb1.z, pp.rb1.w);
      unpack_half(af1, 1, pp.ra1.z, pp.ra1.w);
      __builtin_amdgcn_sched_barrier(0);
      // slot 3: P01 | LDS reads of g+1, update (0,0)
      const v16f p01 = span_partial(pp.af0, bf1);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (q % 4 == 3) {
        wait_vmcnt<0>();
        lds_wait_barrier();
      }
      // the reads come before the copy into the other buffer, so that the
      // compiler does not make them wait for it
      const GroupData nd = load_group(q < 3 || q == 7 ? st0 : st1, (q + 1) % 4);
      if constexpr (q % 4 == 3) issue(s_next, q == 3 ? st0 : st1);
      update(0, 0, g, 0, p00, s0);
      __builtin_amdgcn_sched_barrier(0);
      // slot 4: S1 | update (0,1), half of A0 of g+1
      const v32f s1 = scale_products(pp.sa1, pp.sb);
      __builtin_amdgcn_sched_barrier(0);
      update(0, 1, g, 0, p01, s0);
      unpack_half(af0n, 0, nd.a[0].x, nd.a[0].y);
      __builtin_amdgcn_sched_barrier(0);
      // slot 5: P10 | other half of A0 of g+1, half of B0 of g+1
      const v16f p10 = span_partial(af1, pp.bf0);
      __builtin_amdgcn_sched_barrier(0);
      unpack_half(af0n, 1, nd.a[0].z, nd.a[0].w);
      unpack_half(bf0n, 0, nd.b[0].x, nd.b[0].y);
      __builtin_amdgcn_sched_barrier(0);
      // slot 6: P11 | update (1,0), other half of B0 of g+1
      const v16f p11 = span_partial(af1, bf1);
      __builtin_amdgcn_sched_barrier(0);
      update(1, 0, g, 0, p10, s1);
      unpack_half(bf0n, 1, nd.b[0].z, nd.b[0].w);
      __builtin_amdgcn_sched_barrier(0);
      pp.af0 = af0n;
      pp.bf0 = bf0n;
      pp.ra1 = nd.a[1];
      pp.rb1 = nd.b[1];
      if (!PARTIALS) { pp.sa0 = nd.sa[0][0]; pp.sa1 = nd.sa[1][0]; pp.sb = nd.sb[0]; }
      pp.s1 = s1;
      pp.p11 = p11;
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using I4 = std::integral_constant<int, 4>;
    using I5 = std::integral_constant<int, 5>;
    using I6 = std::integral_constant<int, 6>;
    using I7 = std::integral_constant<int, 7>;

    wait_vmcnt<0>();
    lds_wait_barrier();
    issue(1, st1);
    Pipe pp;
    start(pp, load_group(st0, 0));
    pp.s1 = v32f{};
    pp.p11 = v16f{};
    // two stages (8 groups) per iteration; stage s is in st0, s + 1 in st1
    int g = 0;
    for (; g + 2 * KC <= G; g += 2 * KC) {
      const int s = g / KC;
      step(I0{}, g, pp, 0);
      step(I1{}, g + 1, pp, 0);
      step(I2{}, g + 2, pp, 0);
      step(I3{}, g + 3, pp, s + 2);
      step(I4{}, g + 4, pp, 0);
      step(I5{}, g + 5, pp, 0);
      step(I6{}, g + 6, pp, 0);
      step(I7{}, g + 7, pp, s + 3);
    }
    // fewer than 8 groups remain, in the same ring positions
    const int rest = G - g;
    const int s = g / KC;
    if (rest > 0) step(I0{}, g, pp, 0);
    if (rest > 1) step(I1{}, g + 1, pp, 0);
    if (rest > 2) step(I2{}, g + 2, pp, 0);
    if (rest > 3) step(I3{}, g + 3, pp, s + 2);
    if (rest > 4) step(I4{}, g + 4, pp, 0);
    if (rest > 5) step(I5{}, g + 5, pp, 0);
    if (rest > 6) step(I6{}, g + 6, pp, 0);
    update(1, 1, G - 1, 0, pp.p11, pp.s1);
  }
  // the copies issued past the last stage (a stage earlier) must land before
  // the workgroup's LDS can go to another workgroup
  wait_vmcnt<0>();
  if (PARTIALS) return;

  // ---- epilogue: round to bf16 and store straight from registers.  Lane l
  // holds, per block (i, j), output row m = m0 + 64 wm + 32 j + l%32 and
  // columns 8 q + 4 (l/32) .. +3 (q = v/4) of the block: two bf16 pairs per
  // q.  One v_permlane32_swap per pair of words gives the lower half-wave
  // columns 16 p .. +7 and the upper half-wave columns 16 p + 8 .. +15 of the
  // block (p = 0, 1), so every lane stores 16 contiguous bytes and no LDS or
  // barrier is involved. ----
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int m = m0 + wm * 64 + j * 32 + frow;
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        // words (q, e): columns 8 q + 4 (l/32) + 2 e, +1 of the block
        uint32_t w[2][2];
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const int v = 4 * (2 * p + qq) + 2 * e;
            w[qq][e] = bf16_pair(accf[i][j][v], accf[i][j][v + 1]);
          }
        // the upper half-wave's words of q = 2p trade places with the lower
        // half-wave's words of q = 2p + 1
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const auto r = __builtin_amdgcn_permlane32_swap(w[0][e], w[1][e], false, false);
          w[0][e] = r[0];
          w[1][e] = r[1];
        }
        const int n = n0 + wn * 64 + i * 32 + 16 * p + 8 * fhalf;
        if (m < M && n < N)
          *reinterpret_cast<uint4*>(y + static_cast<int64_t>(m) * N + n) = make_uint4(w[0][0], w[0][1], w[1][0], w[1][1]);
      }
    }
}

static int gemm_tiles(int M, int N) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

template <int GS>
static hipError_t launch_asp_gemm_gs(int M, int N, int K, int r, const uint8_t* xq, const float* xs,
                                     const uint16_t* t, const uint8_t* wq, const uint32_t* wsp,
                                     const uint16_t* L2t, const uint16_t* bias, uint16_t* y, hipStream_t stream) {
  const dim3 grid(gemm_tiles(M, N)), block(NT);
  switch (r) {
    case 16:
      hipLaunchKernelGGL((asp_gemm_kernel<16, false, GS>), grid, block, 0, stream, xq, xs, t, wq, wsp, L2t, bias, y, nullptr, M, N, K);
      break;
    case 32:
      hipLaunchKernelGGL((asp_gemm_kernel<32, false, GS>), grid, block, 0, stream, xq, xs, t, wq, wsp, L2t, bias, y, nullptr, M, N, K);
      break;
    case 48:
      hipLaunchKernelGGL((asp_gemm_kernel<48, false, GS>), grid, block, 0, stream, xq, xs, t, wq, wsp, L2t, bias, y, nullptr, M, N, K);
      break;
    case 64:
      hipLaunchKernelGGL((asp_gemm_kernel<64, false, GS>), grid, block, 0, stream, xq, xs, t, wq, wsp, L2t, bias, y, nullptr, M, N, K);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// few tokens: the float32 scales (asp_gemm_small_kernel); otherwise the
// weight-scale pieces
hipError_t launch_asp_gemm(int M, int N, int K, int r, int group, const uint8_t* xq, const float* xs,
                           const uint16_t* t, const uint8_t* wq, const float* ws, const uint32_t* wsp,
                           const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                           hipStream_t stream) {
  if (M <= kSmallM) return launch_asp_gemm_small(M, N, K, r, group, xq, xs, t, wq, ws, L2t, bias, y, stream);
  return group == 32 ? launch_asp_gemm_gs<32>(M, N, K, r, xq, xs, t, wq, wsp, L2t, bias, y, stream)
                     : launch_asp_gemm_gs<64>(M, N, K, r, xq, xs, t, wq, wsp, L2t, bias, y, stream);
}

hipError_t launch_group_partials(int M, int N, int K, int group, const uint8_t* xq, const uint8_t* wq,
                                 int32_t* P, hipStream_t stream) {
  if (M <= kSmallM) return launch_group_partials_small(M, N, K, group, xq, wq, P, stream);
  if (group == 32)
    hipLaunchKernelGGL((asp_gemm_kernel<32, true, 32>), dim3(gemm_tiles(M, N)), dim3(NT), 0, stream, xq, nullptr,
                       nullptr, wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  else
    hipLaunchKernelGGL((asp_gemm_kernel<32, true, 64>), dim3(gemm_tiles(M, N)), dim3(NT), 0, stream, xq, nullptr,
                       nullptr, wq, nullptr, nullptr, nullptr, nullptr, P, M, N, K);
  return hipGetLastError();
}

}  // namespace qwam
