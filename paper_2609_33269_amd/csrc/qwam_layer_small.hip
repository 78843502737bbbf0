// The whole ASP layer for few tokens (M <= 64, the action-expert layers) in
// one launch: the activation step of qwam_quantize_act and the GEMM of
// qwam_asp_linear, fused.  With so few tokens both steps are latency-bound
// (a launch floor of ~1.5 us each and a dependent memory round trip in
// between), so every workgroup quantizes the tokens it needs itself.  That
// quantization is the bulk of a workgroup's vector work and is repeated by
// every workgroup of a token block, so a CU is best given one workgroup:
// the 16-token form (the second kernel below, 16 x 16 NB outputs) runs when
// at most 256 workgroups cover y, the 32-token form otherwise:
//
//   * a workgroup owns a 32 x 32 block of y (32 tokens x 32 output channels)
//     and all of K; its 8 waves split the 64-channel spans into contiguous
//     ranges, one per wave (the split of the few-token GEMM, so that both
//     paths sum the partial blocks in the same order);
//   * lane l of a wave holds token l % 32 and channels 32*(l/32) .. +31 of the
//     current span: the A-operand rows of v_mfma_scale_f32_32x32x64_f8f6f4.
//     It smooths them (x * 1/lambda; each wave copies its slice of 1/lambda
//     into LDS once, where both lane halves read it by broadcast), takes the
//     span's absmax with its partner lane l ^ 32, quantizes (Eq. 2, the same
//     arithmetic as the activation kernel, so the codes are identical) and
//     writes them as FP6 fields in the order codes_to_fp6 gives the weights'
//     fields: both operands then carry the same channel order, and the MFMA
//     returns the span's exact integer partial;
//   * the same registers feed the down-projection t = bf16(x~) . L1 on
//     v_mfma_f32_32x32x16_bf16 (rank columns, four 16-deep steps per span);
//   * per span: acc += P * xs * ws as in the GEMMs (the token scale of each
//     result row reaches its lanes through one cross-lane read);
//   * the waves' partial blocks (acc and t) are summed in LDS in wave order;
//     wave w finishes result registers 2w and 2w+1 (four rows of the block):
//     it rounds those rows of t to bf16, adds their t . L2 (bf16 MFMA; the
//     rows it does not own are ignored, since each result row depends only on
//     its own row of t) and the bias, and stores them.  The epilogue is spread
//     over all waves, so no wave sums every partial alone.
//   * optionally (xq / xs / t not null) the workgroups of the first column
//     block also store the codes, scales and t, as qwam_quantize_act would.
#include "qwam_device.h"
#include "qwam_internal.h"
#include "qwam_mfma.h"

namespace qwam {

namespace {

constexpr int LW = 8;              // waves per workgroup (two per SIMD)
constexpr int LB = 32;             // block edge (tokens and output channels)

}  // namespace

template <int RANK>
__global__ __launch_bounds__(64 * LW) void asp_layer_small_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth, const uint16_t* __restrict__ L1t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, uint8_t* __restrict__ xq_out,
    float* __restrict__ xs_out, uint16_t* __restrict__ t_out, int M, int N, int K) {
  static_assert(RANK == 16 || RANK == 32, "one 32-column block of t");
  // dynamic LDS: partial acc [LW][16][64] | partial t [LW][16][64] | t bf16 [32][RANK] | 1/lambda [K]
  extern __shared__ __attribute__((aligned(16))) float lds[];
  float* red_acc = lds;
  float* red_t = red_acc + LW * 16 * 64;
  uint16_t* t_l = reinterpret_cast<uint16_t*>(red_t + LW * 16 * 64);
  float* inv_l = red_t + LW * 16 * 64 + LB * RANK / 2;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tiles_n = (N + LB - 1) / LB;
  const int m0 = (blockIdx.x / tiles_n) * LB;
  const int n0 = (blockIdx.x % tiles_n) * LB;
  const bool write_act = xq_out != nullptr && blockIdx.x % tiles_n == 0;
  const int G = K / kGroup;
  const int KB = K / 2;
  const int gpw = (G + LW - 1) / LW;
  const int g_lo = min(G, wave * gpw), g_hi = min(G, g_lo + gpw);
  const int rows = min(LB, M - m0);

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  const int rsub = fhalf * 4;
  const int sx_row = 8 * ((lane & 15) >> 2) + 4 * (lane >> 5) + (lane & 3);

  // the workgroup's tokens (rows past M read as zero) and output channels
  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<uint32_t>(rows) * K * 2u);
  const buf_rsrc w_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB, static_cast<uint32_t>(min(LB, N - n0)) * KB);
  const buf_rsrc ws_rsrc = make_rsrc(ws, static_cast<uint32_t>(G) * N * 4u);
  const uint32_t x_off = static_cast<uint32_t>(frow * K + fhalf * 32) * 2u;
  const uint32_t w_off = static_cast<uint32_t>(frow * KB + fhalf * 16);
  const uint32_t sw_off = static_cast<uint32_t>(n0 + frow) * 4u;
  // t columns j = lane % 32 (rows of L1t past RANK read as zero), channels
  // 32*half + 8 s of a span
  const buf_rsrc l1_rsrc = make_rsrc(L1t, static_cast<uint32_t>(RANK) * K * 2u);
  const uint32_t l1_off = static_cast<uint32_t>(frow * K + fhalf * 32) * 2u;

  struct Fetch {
    uint4 x[4];                    // 32 bf16 of x: channels 32*half .. +31 of the span
    uint4 w;                       // 32 packed weight codes of column n0 + lane%32
    float sw;
    v8s l1[4];                     // L1t[j][span + 32*half + 8 s .. +7], s = 0..3
  };
  auto fetch = [&](int g, Fetch& f) __attribute__((always_inline)) {
    const uint32_t go = static_cast<uint32_t>(g) * kGroup * 2u;
#pragma unroll
    for (int q = 0; q < 4; ++q) f.x[q] = buf_load16(x_rsrc, x_off + go + 16u * q);
    f.w = buf_load16(w_rsrc, w_off + static_cast<uint32_t>(g) * 32u);
    f.sw = buf_load4f(ws_rsrc, sw_off + static_cast<uint32_t>(g) * N * 4u);
#pragma unroll
    for (int s = 0; s < 4; ++s) f.l1[s] = __builtin_bit_cast(v8s, buf_load16(l1_rsrc, l1_off + go + 16u * s));
  };

  v16f acc = v16f{};
  v16f tacc = v16f{};
  auto work = [&](int g, const Fetch& f) __attribute__((always_inline)) {
    // x~ = x * (1/lambda) for the lane's 32 channels (1/lambda from LDS, one
    // address per lane half)
    const float4* ip = reinterpret_cast<const float4*>(inv_l + g * kGroup + fhalf * 32);
    float v[32];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t xw[4] = {f.x[q].x, f.x[q].y, f.x[q].z, f.x[q].w};
      const float4 i0 = ip[2 * q];
      const float4 i1 = ip[2 * q + 1];
      const float iv[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[8 * q + 2 * j] = __uint_as_float(xw[j] << 16) * iv[2 * j];
        v[8 * q + 2 * j + 1] = __uint_as_float(xw[j] & 0xFFFF0000u) * iv[2 * j + 1];
      }
    }
    // the span's scale (Eq. 2): absmax of the token's 64 channels (lanes l, l^32)
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
    amax = max_xor32(amax);
    const float s = q4_scale(amax);
    const float inv = q4_inv(s);
    // codes -> FP6 fields (one conversion for the lane's 32 channels): the
    // MFMA operand itself, and the two code blocks (the storage format) for
    // the optional copy of the codes
    float xs32[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) xs32[i] = v[i] * inv;
    const v6u d = codes_fp6_32(xs32);
    v8i af;          // words 6-7 are not read with FP6 operands and stay unset
    uint32_t cw[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      af[3 * h] = static_cast<int>(d[3 * h]);
      af[3 * h + 1] = static_cast<int>(d[3 * h + 1]);
      af[3 * h + 2] = static_cast<int>(d[3 * h + 2]);
      const uint2 blk = fp6_code_block(d[3 * h], d[3 * h + 1], d[3 * h + 2]);
      cw[2 * h] = blk.x;
      cw[2 * h + 1] = blk.y;
    }
    if (write_act && m0 + frow < M) {
      *reinterpret_cast<uint4*>(xq_out + static_cast<int64_t>(m0 + frow) * KB + g * 32 + fhalf * 16) =
          make_uint4(cw[0], cw[1], cw[2], cw[3]);
      if (fhalf == 0) xs_out[static_cast<int64_t>(g) * M + m0 + frow] = s;
    }
    // exact integer partial of the span, then acc += P * xs * ws
    const v16f p = fp6_partial(af, codes_to_fp6(f.w), kE8M0Code, kE8M0Code);
    const float sx_lane = __shfl(s, sx_row);            // scale of the token of result register v
    scale_accumulate(std::make_integer_sequence<int, 16>{}, acc, p, sx_lane, f.sw);
    // t partial: A = bf16(x~) of 8 channels per step, B = the matching L1t slice
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      v8bf a;
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = static_cast<__bf16>(v[8 * st + i]);
      tacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(v8bf, f.l1[st]), tacc, 0, 0, 0);
    }
  };

  // epilogue operands: L2t rows of the block's columns, bias
  constexpr int KSTEPS = RANK / 16;
  const int nt = n0 + frow;
  v8s lv[KSTEPS];
#pragma unroll
  for (int k = 0; k < KSTEPS; ++k) {
    lv[k] = v8s{0, 0, 0, 0, 0, 0, 0, 0};
    if (nt < N) lv[k] = *reinterpret_cast<const v8s*>(L2t + static_cast<int64_t>(nt) * RANK + k * 16 + fhalf * 8);
  }
  // the bias bits (zero without a bias or past N) are converted only at the end,
  // so that no wait for this load lands before the spans
  const buf_rsrc b_rsrc = make_rsrc(bias, bias != nullptr ? static_cast<uint32_t>(N) * 2u : 0u);
  const uint32_t bbits = __builtin_amdgcn_raw_buffer_load_b16(b_rsrc, static_cast<uint32_t>(nt) * 2u, 0, 0);

  // the wave's slice of 1/lambda goes to LDS (direct copies, 256 floats per
  // instruction; lanes past the slice copy nothing), then the first spans are
  // requested; all of it is waited for before the first span is used
  if (g_lo < g_hi) {
    const buf_rsrc i_rsrc = make_rsrc(inv_smooth, static_cast<uint32_t>(K) * 4u);
    const int nfl = (g_hi - g_lo) * kGroup;
    for (int c = 0; c < nfl; c += 256)
      if (c + 4 * lane < nfl)
        buf_load16_lds(i_rsrc, static_cast<uint32_t>(g_lo * kGroup + c + 4 * lane) * 4u, inv_l + g_lo * kGroup + c);
  }

  // the wave's spans, one fetched ahead
  if (g_lo < g_hi) {
    // a fetch is 4 requests of x, then 6 (weights, scale, L1t); the 1/lambda
    // copies were issued before both fetches and requests complete in issue
    // order, so waiting until only the later requests are outstanding lets
    // the first span's quantization overlap the weights' arrival
    Fetch fa, fb;
    fetch(g_lo, fa);
    int g = g_lo;
    if (g + 1 < g_hi) {
      fetch(g + 1, fb);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(6 + 10) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(6) : "memory");
    }
    for (; g + 1 < g_hi; g += 2) {
      work(g, fa);
      if (g + 2 < g_hi) fetch(g + 2, fa);
      work(g + 1, fb);
      if (g + 3 < g_hi) fetch(g + 3, fb);
    }
    if (g < g_hi) work(g, fa);
  }

  // partial blocks -> LDS, summed in wave order below
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    red_acc[(wave * 16 + v) * 64 + lane] = acc[v];
    red_t[(wave * 16 + v) * 64 + lane] = tacc[v];
  }
  __syncthreads();
  // this wave's result registers v0, v0 + 1: token 8(v/4) + 4(l/32) + v%4, column l%32
  const int v0 = 2 * wave;
  float c2[2] = {0.0f, 0.0f}, t2[2] = {0.0f, 0.0f};
#pragma unroll
  for (int w = 0; w < LW; ++w)
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      c2[e] += red_acc[(w * 16 + v0 + e) * 64 + lane];
      t2[e] += red_t[(w * 16 + v0 + e) * 64 + lane];
    }
  // t = bf16(sum) of those rows, to LDS (and out)
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int v = v0 + e;
    const int row = 8 * (v >> 2) + rsub + (v & 3);
    if (frow < RANK) {
      const uint16_t b = static_cast<uint16_t>(f32_to_bf16_rne(t2[e]));
      t_l[row * RANK + frow] = b;
      if (write_act && m0 + row < M) t_out[static_cast<int64_t>(m0 + row) * RANK + frow] = b;
    }
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's t stores are in LDS
  // y = acc + t . L2 + bias; A operand: token l%32, rank slots 16 k + 8(l/32) .. +7.  Only
  // the rows of this wave's registers are used; the other rows of t_l may still be written
  // by other waves, and they reach only result rows this wave discards.
  v16f c;
#pragma unroll
  for (int v = 0; v < 16; ++v) c[v] = v == v0 ? c2[0] : (v == v0 + 1 ? c2[1] : 0.0f);
#pragma unroll
  for (int k = 0; k < KSTEPS; ++k) {
    const v8s tv = *reinterpret_cast<const v8s*>(t_l + frow * RANK + k * 16 + fhalf * 8);
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, tv), __builtin_bit_cast(v8bf, lv[k]), c, 0,
                                                0, 0);
  }
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

// ---------------------------------------------------------------------------
// The same layer in 16-token blocks.  The workgroup owns 16 tokens x 16 NB
// output channels (NB = 1, 2 or 4 blocks of 16) and runs the integer
// partials on v_mfma_scale_f32_16x16x128_f8f6f4: lane l holds token (or
// output channel) l % 16 and channels 32*(l/16) .. +31 of a 128-channel
// step, i.e. two 64-channel spans, lane groups 0-1 the first and 2-3 the
// second.  Each span's partial is its own instruction, with the other span's
// lane scales at 2^-127 on both operands (their products underflow to zero).
// Per lane and step this quantizes 32 real channels (the 32-token form
// quantizes 32 channels for two tokens), and the NB weight blocks reuse the
// quantized operand.  Every workgroup quantizes its 16 tokens itself, so the
// quantization is repeated once per workgroup of a token block; the launcher
// takes this form when it fits one workgroup per CU (at most 256 workgroups
// with NB <= 4), the 32-token form above otherwise.  With NB = 4 (only for
// K <= 1024, one step per wave) there is no prefetch buffer.
//
// The K split (eight waves, contiguous ranges of spans), the order of the
// per-span scaling and of the sum over the waves, and the epilogue's
// v_mfma_f32_32x32x16_bf16 (rows 16-31 zero) are those of the few-token
// GEMM, so the two paths give the same y from the same codes, scales and t.
// ---------------------------------------------------------------------------
template <int RANK, int NB>
__global__ __launch_bounds__(64 * LW) void asp_layer_tiny_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth, const uint16_t* __restrict__ L1t,
    const uint8_t* __restrict__ wq, const float* __restrict__ ws, const uint16_t* __restrict__ L2t,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, uint8_t* __restrict__ xq_out,
    float* __restrict__ xs_out, uint16_t* __restrict__ t_out, int M, int N, int K) {
  static_assert(RANK == 16 || RANK == 32, "one or two 16-column blocks of t");
  constexpr int TBK = 16;                // tokens and output channels of the block
  constexpr int RB = RANK / 16;
  // dynamic LDS: partial acc [LW][16][16] | partial t [LW][16][RANK] | t bf16 [16][RANK] | 1/lambda [K]
  // and 128 floats that a second span past K reads (its values are discarded)
  extern __shared__ __attribute__((aligned(16))) float lds[];
  constexpr int BN = TBK * NB;            // output channels of the workgroup
  float* red_acc = lds;
  float* red_t = red_acc + LW * TBK * BN;
  uint16_t* t_l = reinterpret_cast<uint16_t*>(red_t + LW * TBK * RANK);
  float* inv_l = red_t + LW * TBK * RANK + TBK * RANK / 2;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ncb = (N + BN - 1) / BN;
  const int n0 = (blockIdx.x % ncb) * BN;
  const int m0 = (blockIdx.x / ncb) * TBK;
  const int rows = min(TBK, M - m0);
  const bool write_act = xq_out != nullptr && blockIdx.x % ncb == 0;
  const int G = K / kGroup;
  const int KB = K / 2;
  const int gpw = (G + LW - 1) / LW;
  const int g_lo = min(G, wave * gpw), g_hi = min(G, g_lo + gpw);

  const int frow = lane & 15;            // token (A, t) or output channel (B)
  const int grp = lane >> 4;             // 32-channel block of the step
  const int half = grp >> 1;             // span of the step
  // D of a 16x16 block: lane l holds column l%16 and rows 4*(l/16) + i

  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<uint32_t>(rows) * K * 2u);
  const buf_rsrc w_rsrc = make_rsrc(wq + static_cast<int64_t>(n0) * KB, static_cast<uint32_t>(min(BN, N - n0)) * KB);
  const buf_rsrc ws_rsrc = make_rsrc(ws, static_cast<uint32_t>(G) * N * 4u);
  const buf_rsrc l1_rsrc = make_rsrc(L1t, static_cast<uint32_t>(RANK) * K * 2u);
  const uint32_t x_off = static_cast<uint32_t>(frow * K + 32 * grp) * 2u;
  const uint32_t w_off = static_cast<uint32_t>(frow * KB + 16 * grp);
  const uint32_t sw_off = static_cast<uint32_t>(n0 + frow) * 4u;
  // t MFMA j of a step (v_mfma_f32_16x16x32_bf16): lane l supplies channels
  // 32*(l/16) + 8 j .. +7 as its k-slots, so B lane l (t column l%16 of block
  // rb) takes L1t[16 rb + l%16][the same channels]
  const uint32_t l1_off = static_cast<uint32_t>(frow * K + 32 * grp) * 2u;

  struct Fetch {
    uint4 x[4];                    // 32 bf16 of x
    uint4 w[NB];                   // 32 packed weight codes of column n0 + 16 b + lane%16
    float sw[NB][2];               // weight scales of those columns, both spans
    v8s l1[RB][4];
  };
  // the step of spans g, g+1 (g+1 only when below g_hi)
  auto fetch = [&](int g, Fetch& f) __attribute__((always_inline)) {
    const uint32_t go = static_cast<uint32_t>(g) * kGroup * 2u;
#pragma unroll
    for (int q = 0; q < 4; ++q) f.x[q] = buf_load16(x_rsrc, x_off + go + 16u * q);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f.w[nb] = buf_load16(w_rsrc, w_off + static_cast<uint32_t>(nb * TBK * KB) + static_cast<uint32_t>(g) * 32u);
#pragma unroll
      for (int h = 0; h < 2; ++h)
        f.sw[nb][h] = buf_load4f(ws_rsrc, sw_off + static_cast<uint32_t>(nb * TBK) * 4u + static_cast<uint32_t>(g + h) * N * 4u);
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        f.l1[rb][j] = __builtin_bit_cast(
            v8s, buf_load16(l1_rsrc, l1_off + static_cast<uint32_t>(16 * rb) * K * 2u + go + 16u * j));
  };

  v4f acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = v4f{0.f, 0.f, 0.f, 0.f};
  v4f tacc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) tacc[rb] = v4f{0.f, 0.f, 0.f, 0.f};
  auto work = [&](int g, const Fetch& f) __attribute__((always_inline)) {
    const bool two = g + 1 < g_hi;
    // x~ = x * (1/lambda) for the lane's 32 channels (1/lambda from LDS)
    const float4* ip = reinterpret_cast<const float4*>(inv_l + g * kGroup + 32 * grp);
    float v[32];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t xw[4] = {f.x[q].x, f.x[q].y, f.x[q].z, f.x[q].w};
      const float4 i0 = ip[2 * q];
      const float4 i1 = ip[2 * q + 1];
      const float iv[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[8 * q + 2 * j] = __uint_as_float(xw[j] << 16) * iv[2 * j];
        v[8 * q + 2 * j + 1] = __uint_as_float(xw[j] & 0xFFFF0000u) * iv[2 * j + 1];
      }
    }
    // a second span past the wave's range (its channels belong to the next
    // wave or lie past K) is zero, so that it adds nothing to t
    if (half == 1 && !two) {
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = 0.0f;
    }
    // the span's scale (Eq. 2): absmax of the token's 64 channels (lanes l, l^16)
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
    amax = max_xor16(amax);
    const float s = q4_scale(amax);
    const float inv = q4_inv(s);
    float xs32[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) xs32[i] = v[i] * inv;
    const v6u d = codes_fp6_32(xs32);
    v8i af;          // words 6-7 are not read with FP6 operands and stay unset
#pragma unroll
    for (int k = 0; k < 6; ++k) af[k] = static_cast<int>(d[k]);
    if (write_act && frow < rows && (half == 0 || two)) {
      const uint2 b0 = fp6_code_block(d[0], d[1], d[2]);
      const uint2 b1 = fp6_code_block(d[3], d[4], d[5]);
      *reinterpret_cast<uint4*>(xq_out + static_cast<int64_t>(m0 + frow) * KB + g * 32 + 16 * grp) =
          make_uint4(b0.x, b0.y, b1.x, b1.y);
      if ((grp & 1) == 0) xs_out[static_cast<int64_t>(g + half) * M + m0 + frow] = s;
    }
    // the spans' exact integer partials, then acc += P * xs * ws, span g first
    float sxs[2][4];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) sxs[h][i] = __shfl(s, 4 * grp + i + 32 * h);   // token 4*(l/16)+i, span h
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const v8i bf = codes_to_fp6(f.w[nb]);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (h == 1 && !two) break;
        const int sc = half == h ? kE8M0Code : 0;
        const v4f p = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf, v4f{}, kFmtFp6, kFmtFp6, 0, sc, 0, sc);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[nb][i] = __builtin_fmaf(p[i], sxs[h][i] * f.sw[nb][h], acc[nb][i]);
      }
    }
    // t partial: A = bf16(x~) of 8 channels per MFMA, B = the matching L1t slice
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v8bf a;
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = static_cast<__bf16>(v[8 * j + i]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        tacc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(v8bf, f.l1[rb][j]), tacc[rb], 0, 0, 0);
    }
  };

  // epilogue operands: the 32x32 MFMA's B (L2t rows of 32 columns of the
  // block, columns past BN zero) and the bias bits (converted only at the end)
  constexpr int KSTEPS = RANK / 16;
  constexpr int EB = (BN + 31) / 32;     // 32-column epilogue blocks
  const int ecol = lane & 31, ehalf = lane >> 5;
  const buf_rsrc l2_rsrc = make_rsrc(L2t + static_cast<int64_t>(n0) * RANK,
                                     static_cast<uint32_t>(min(BN, N - n0)) * RANK * 2u);
  const buf_rsrc b_rsrc = make_rsrc(bias, bias != nullptr ? static_cast<uint32_t>(N) * 2u : 0u);
  v8s lv[EB][KSTEPS];
  uint32_t bbits[EB];
#pragma unroll
  for (int eb = 0; eb < EB; ++eb) {
    const int c = 32 * eb + ecol;
    const bool ok = c < BN && n0 + c < N;
#pragma unroll
    for (int k = 0; k < KSTEPS; ++k)
      lv[eb][k] = c < BN ? __builtin_bit_cast(v8s, buf_load16(l2_rsrc, static_cast<uint32_t>(c * RANK + k * 16 + ehalf * 8) * 2u))
                         : v8s{0, 0, 0, 0, 0, 0, 0, 0};
    bbits[eb] = __builtin_amdgcn_raw_buffer_load_b16(b_rsrc, static_cast<uint32_t>(ok ? n0 + c : N) * 2u, 0, 0);
  }

  // the wave's slice of 1/lambda to LDS, then the first steps; all of it is
  // waited for before the first step is used
  if (g_lo < g_hi) {
    const buf_rsrc i_rsrc = make_rsrc(inv_smooth, static_cast<uint32_t>(K) * 4u);
    const int nfl = (g_hi - g_lo) * kGroup;
    for (int c = 0; c < nfl; c += 256)
      if (c + 4 * lane < nfl)
        buf_load16_lds(i_rsrc, static_cast<uint32_t>(g_lo * kGroup + c + 4 * lane) * 4u, inv_l + g_lo * kGroup + c);
  }
  // a fetch is 4 requests of x, then kLater (weights, their scales, L1t);
  // the 1/lambda copies were issued before it and requests complete in issue
  // order, so waiting until only the later requests are outstanding lets the
  // quantization of the first step overlap the weights' arrival
  constexpr int kLater = 3 * NB + 4 * RB;
  if constexpr (NB == 4) {
    // one step per wave (K <= 1024, chosen by the launcher): no prefetch buffer
    if (g_lo < g_hi) {
      Fetch fa;
      fetch(g_lo, fa);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLater) : "memory");
      work(g_lo, fa);
    }
  } else if (g_lo < g_hi) {
    Fetch fa, fb;
    fetch(g_lo, fa);
    int g = g_lo;
    if (g + 2 < g_hi) {
      fetch(g + 2, fb);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLater + 4 + kLater) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLater) : "memory");
    }
    for (; g + 2 < g_hi; g += 4) {
      work(g, fa);
      if (g + 4 < g_hi) fetch(g + 4, fa);
      work(g + 2, fb);
      if (g + 6 < g_hi) fetch(g + 6, fb);
    }
    if (g < g_hi) work(g, fa);
  }

  // partial blocks -> LDS: acc as [wave][token][column], t as [wave][token][column]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) red_acc[(wave * TBK + 4 * grp + i) * BN + nb * TBK + frow] = acc[nb][i];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) red_t[(wave * TBK + 4 * grp + i) * RANK + 16 * rb + frow] = tacc[rb][i];
  }
  __syncthreads();
  // t = bf16(sum over the waves in order), one element per thread
  for (int e = tid; e < TBK * RANK; e += 64 * LW) {
    const int tok = e / RANK, j = e % RANK;
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < LW; ++w) sum += red_t[(w * TBK + tok) * RANK + j];
    const uint16_t b = static_cast<uint16_t>(f32_to_bf16_rne(sum));
    t_l[tok * RANK + j] = b;
    if (write_act && tok < rows) t_out[static_cast<int64_t>(m0 + tok) * RANK + j] = b;
  }
  // this wave's result register of the 32x32 epilogue blocks: v = wave (rows
  // below 16), token 8(v/4) + 4(l/32) + v%4, column 32 eb + l%32
  const int v0 = wave;
  const int tok = 8 * (v0 >> 2) + 4 * ehalf + (v0 & 3);
  float c2[EB];
#pragma unroll
  for (int eb = 0; eb < EB; ++eb) {
    const int c = 32 * eb + ecol;
    c2[eb] = 0.0f;
#pragma unroll
    for (int w = 0; w < LW; ++w) c2[eb] += c < BN ? red_acc[(w * TBK + tok) * BN + c] : 0.0f;
  }
  __syncthreads();                      // t_l complete
  const int arow = lane & 31;           // A operand: token l%32 (rows 16-31 zero)
#pragma unroll
  for (int eb = 0; eb < EB; ++eb) {
    v16f c;
#pragma unroll
    for (int v = 0; v < 16; ++v) c[v] = v == v0 ? c2[eb] : 0.0f;
#pragma unroll
    for (int k = 0; k < KSTEPS; ++k) {
      v8s tv = v8s{0, 0, 0, 0, 0, 0, 0, 0};
      if (arow < TBK) tv = *reinterpret_cast<const v8s*>(t_l + arow * RANK + k * 16 + ehalf * 8);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, tv), __builtin_bit_cast(v8bf, lv[eb][k]), c,
                                                  0, 0, 0);
    }
    float yv = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (v == v0) yv = c[v];
    const int col = 32 * eb + ecol;
    if (tok < rows && col < BN && n0 + col < N)
      y[static_cast<int64_t>(m0 + tok) * N + n0 + col] =
          static_cast<uint16_t>(f32_to_bf16_rne(yv + bf16_to_f32(bbits[eb])));
  }
}

hipError_t launch_asp_layer_small(int M, int N, int K, int r, const uint16_t* x, const float* inv_smooth,
                                  const uint16_t* L1t, const uint8_t* wq, const float* ws, const uint16_t* L2t,
                                  const uint16_t* bias, uint16_t* y, uint8_t* xq, float* xs, uint16_t* t,
                                  hipStream_t stream) {
  const int units = ((M + 15) / 16) * ((N + 15) / 16);
  int nb = 1;
  const int maxnb = K <= 1024 ? 4 : 2;
  while (nb < maxnb && units > 256 * nb) nb *= 2;
  const bool tiny = M <= 16 || units <= 256 * nb;
  const dim3 grid(tiny ? ((M + 15) / 16) * ((N + 16 * nb - 1) / (16 * nb)) : ((M + LB - 1) / LB) * ((N + LB - 1) / LB)),
      block(64 * LW);
  const size_t lds = tiny ? static_cast<size_t>(LW) * 16 * (16 * nb + r) * 4 + 16 * r * 2 + static_cast<size_t>(K + 128) * 4
                          : static_cast<size_t>(2) * LW * 16 * 64 * 4 + LB * r * 2 + static_cast<size_t>(K) * 4;
  auto go = [&](auto kernel) {
    if (lds > 64 * 1024) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kernel, grid, block, lds, stream, x, inv_smooth, L1t, wq, ws, L2t, bias, y, xq, xs, t, M, N,
                       K);
    return hipGetLastError();
  };
  auto pick = [&](auto k1, auto k2, auto k4, auto ksmall) {
    if (!tiny) return go(ksmall);
    return nb == 1 ? go(k1) : (nb == 2 ? go(k2) : go(k4));
  };
  switch (r) {
    case 16: return pick(asp_layer_tiny_kernel<16, 1>, asp_layer_tiny_kernel<16, 2>, asp_layer_tiny_kernel<16, 4>, asp_layer_small_kernel<16>);
    case 32: return pick(asp_layer_tiny_kernel<32, 1>, asp_layer_tiny_kernel<32, 2>, asp_layer_tiny_kernel<32, 4>, asp_layer_small_kernel<32>);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace qwam
