// Activation kernels with the block Hadamard rotation of Eq. 3:
//     x~ = H diag(lambda)^-1 x,
// H block-diagonal with Hadamard blocks of size B (the largest power of two
// dividing K, at most 1024, App. B.1), applied online with the fast
// Walsh-Hadamard transform (the weights were rotated offline).  The transform
// runs in float32, one rounding per butterfly, stages on element bit 0, 1, ..
// in that order, then one multiply by fl32(1/sqrt(B)).
//
// A block spans several groups, so a workgroup (16 tokens) works in tiles of
// T channels (a multiple of B and of 64 dividing K, at most 1024):
//   rotate:   pass p of a tile is 1024 consecutive elements of the [16][T]
//             tile; lane l holds 16 consecutive channels of one token, so
//             butterfly stages 0-3 run in registers and stages 4 .. log2(B)-1
//             between lanes l and l ^ 2^(s-4) (DPP, ds_swizzle and the
//             permlane swaps of gfx950).  The rotated tile goes to LDS
//             (rows padded by 4 floats against bank conflicts).
//   quantize: each wave reads its groups of the tile back in the lane layout
//             of qwam_act.h and runs the plain kernel's per-group steps (or,
//             deflated, the two phases of the deflated kernel, rotating the
//             tiles again in phase 2).
#include <cmath>
#include <type_traits>

#include "qwam_act.h"
#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int kTilePad = 4;   // floats of padding per LDS tile row

// Fast Walsh-Hadamard transform of a block of 2^logB elements held 16 per lane
// (lane bit b <-> element bit 4 + b): v becomes v H_B, unnormalized.
__device__ __forceinline__ void fwht16(float (&v)[16], int lane, int logB) {
#pragma unroll
  for (int h = 1; h < 16; h <<= 1)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (!(i & h)) {
        const float a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
  // Stages between lanes l and l ^ m.  The partner's value p comes by DPP
  // (m = 1, 2: quad permutes; m = 8: rotation by 8 inside a row of 16), by
  // ds_swizzle (m = 4) or by v_permlane16/32_swap (m = 16, 32), instead of a
  // ds_bpermute per element.  The lane of the pair without bit m gets a + b,
  // the other a - b, one rounding each: fma(., +-1, .) computes exactly that.
  for (int s = 4; s < logB; ++s) {
    const int m = 1 << (s - 4);
    const float sgn = (lane & m) != 0 ? -1.0f : 1.0f;   // -1: this lane holds the element with bit s set
    // the lower lane: v + p = a + b; the upper: p - v = a - b
    auto near = [&](auto xchg) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = __builtin_fmaf(v[i], sgn, __int_as_float(xchg(__float_as_int(v[i]))));
    };
    // swap results: [0] = own value in the lower half of each pair of rows
    // (m = 16) or in lanes 0-31 (m = 32), the partner's in the other; [1]
    // the reverse.  The lower lane computes [0] + [1] = a + b, the upper
    // [0] - [1] = a - b.
    auto far = [&](auto swap) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const auto r = swap(__float_as_uint(v[i]));
        v[i] = __builtin_fmaf(__uint_as_float(r[1]), sgn, __uint_as_float(r[0]));
      }
    };
    switch (m) {
      case 1: near([](int u) { return __builtin_amdgcn_update_dpp(0, u, 0xB1, 0xF, 0xF, false); }); break;  // quad_perm [1,0,3,2]
      case 2: near([](int u) { return __builtin_amdgcn_update_dpp(0, u, 0x4E, 0xF, 0xF, false); }); break;  // quad_perm [2,3,0,1]
      case 4: near([](int u) { return __builtin_amdgcn_ds_swizzle(u, (4 << 10) | 0x1F); }); break;          // xor 4
      case 8: near([](int u) { return __builtin_amdgcn_update_dpp(0, u, 0x128, 0xF, 0xF, false); }); break; // row_ror:8
      case 16: far([](unsigned u) { return __builtin_amdgcn_permlane16_swap(u, u, false, false); }); break;
      default: far([](unsigned u) { return __builtin_amdgcn_permlane32_swap(u, u, false, false); }); break;
    }
  }
}

}  // namespace

// Registers of one rotation pass: 16 bf16 of x and the matching 1/lambda.
struct RotFetch {
  uint4 xa, xb;
  float4 inv[4];
};

// Rotation passes (= groups) of a tile per wave: a tile of at most 1024
// channels has at most 16, spread over act_waves<RANK>() waves.
template <int RANK>
constexpr int per_wave() { return 16 / act_waves<RANK>(); }

// Barrier for LDS hand-offs between the waves: waits for this wave's LDS
// operations only, so prefetched global loads stay in flight across it.
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int RANK, bool DEFLATE>
__global__ __launch_bounds__(64 * act_waves<RANK>()) void quantize_act_rotated_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth,
    const uint16_t* __restrict__ L1f, const uint16_t* __restrict__ L1, uint8_t* __restrict__ xq, float* __restrict__ xs,
    uint16_t* __restrict__ t, int M, int K, int logB, int T, float hscale, int g32, int red_off) {
  constexpr int RB = RANK / 16;
  constexpr int kMaxPerWave = per_wave<RANK>();
  using Acc = std::conditional_t<DEFLATE, double, float>;
  // dynamic LDS: two tiles [16][T + pad] float (tile tb in buffer tb % 2) |
  // partial t [nwaves][16][RANK] Acc at float offset red_off (after the tiles,
  // or, when both do not fit, over the buffer the last tile does not use) |
  // (DEFLATE) -t [16][RANK] float after both
  extern __shared__ double lds_raw[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nwaves = blockDim.x >> 6;
  const int row = lane & 15;
  const int chunk = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int rows = min(16, M - m0);
  const int TS = T + kTilePad;
  const int ntiles = K / T;
  const int npass = T / kGroup;          // 1024-element passes per tile = groups per tile

  float* tiles = reinterpret_cast<float*>(lds_raw);
  Acc* red = reinterpret_cast<Acc*>(tiles + red_off);
  float* tneg = reinterpret_cast<float*>(red + nwaves * 16 * RANK);
  if (red_off < 2 * 16 * TS) tneg = tiles + 2 * 16 * TS;   // red over a tile buffer

  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m0) * K, static_cast<uint32_t>(rows) * K * 2u);
  const buf_rsrc q_rsrc = make_rsrc(xq + static_cast<int64_t>(m0) * (K / 2), static_cast<uint32_t>(rows) * (K / 2));
  const uint32_t q_off = static_cast<uint32_t>(row * (K / 2) + chunk * 8);

  // pass k of this wave in a tile covers elements (wave + k nwaves) * 1024 + 16 lane .. +15
  auto fetch_tile = [&](int tb, RotFetch (&rf)[kMaxPerWave]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kMaxPerWave; ++k) {
      const int p = wave + k * nwaves;
      if (p < npass) {
        const int e = p * 1024 + 16 * lane;
        const int ch = tb * T + e % T;
        const uint32_t xo = static_cast<uint32_t>((e / T) * K + ch) * 2u;
        rf[k].xa = buf_load16(x_rsrc, xo);
        rf[k].xb = buf_load16(x_rsrc, xo + 16u);
        const float4* ip = reinterpret_cast<const float4*>(inv_smooth + ch);
#pragma unroll
        for (int q = 0; q < 4; ++q) rf[k].inv[q] = ip[q];
      }
    }
  };
  // smooth, transform and scale the fetched passes into the LDS tile (tokens past M are zero)
  auto rotate_tile = [&](const RotFetch (&rf)[kMaxPerWave], float* tile) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kMaxPerWave; ++k) {
      const int p = wave + k * nwaves;
      if (p < npass) {
        const int e = p * 1024 + 16 * lane;
        float v[16];
        smooth16_regs(rf[k].xa, rf[k].xb, rf[k].inv, v);
        fwht16(v, lane, logB);
        float4* dst = reinterpret_cast<float4*>(tile + (e / T) * TS + e % T);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          dst[q] = make_float4(v[4 * q] * hscale, v[4 * q + 1] * hscale, v[4 * q + 2] * hscale, v[4 * q + 3] * hscale);
      }
    }
  };
  auto read_group = [&](const float* tile, int gl, float (&v)[16]) __attribute__((always_inline)) {
    const float4* src = reinterpret_cast<const float4*>(tile + row * TS + gl * kGroup + chunk * 16);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 f = src[q];
      v[4 * q] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
    }
  };
  auto store_codes = [&](int g, const float (&v)[16]) __attribute__((always_inline)) {
    quantize_pack_store(v, q_rsrc, q_off + static_cast<uint32_t>(g) * (kGroup / 2),
                        xs_slot(xs, g, M, m0, row, rows, chunk, g32), g32);
  };

  std::conditional_t<DEFLATE, v4d, v4f> acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = {};

  // pass over the tiles: t partials (and, without deflation, the codes).  The
  // next tile's x and 1/lambda are requested as soon as this tile's are in LDS.
  // Tile tb goes to buffer tb % 2, so one barrier per tile suffices: a wave
  // writes buffer tb % 2 only after the barrier of tile tb - 1, which every
  // wave reaches after its reads of tile tb - 2 from that buffer.
  RotFetch rf[kMaxPerWave];
  fetch_tile(0, rf);
  for (int tb = 0; tb < ntiles; ++tb) {
    float* tile = tiles + (tb & 1) * 16 * TS;
    rotate_tile(rf, tile);
    if (tb + 1 < ntiles) fetch_tile(tb + 1, rf);
    v8s l1[kMaxPerWave][RB][2];
#pragma unroll
    for (int k = 0; k < kMaxPerWave; ++k) {
      const int gl = wave + k * nwaves;
      if (gl < npass) load_l1_fragments<RB>(L1f, tb * npass + gl, lane, l1[k]);
    }
    lds_sync();
#pragma unroll
    for (int k = 0; k < kMaxPerWave; ++k) {
      const int gl = wave + k * nwaves;
      if (gl < npass) {
        float v[16];
        read_group(tile, gl, v);
        if constexpr (DEFLATE) {
          t_step_f64<RB>(v, l1[k], acc);
        } else {
          store_codes(tb * npass + gl, v);
          t_step_bf16<RB>(v, l1[k], acc);
        }
      }
    }
  }
  // the second pass takes the last tile first, still in LDS from the first
  // pass, then tiles 0 .. ntiles - 2 again; tile 0's x is requested here
  if constexpr (DEFLATE)
    if (ntiles > 1) fetch_tile(0, rf);
  lds_sync();                                   // the partials may overwrite a tile buffer
  store_t_partials<RB>(red, wave, lane, acc);
  lds_sync();
  reduce_t<RANK>(red, nwaves, rows, t + static_cast<int64_t>(m0) * RANK, DEFLATE ? tneg : nullptr);

  if constexpr (DEFLATE) {
    lds_sync();
    // second pass: deflate and quantize.  Step 0 reads the last tile where
    // the first pass left it (buffer Lb; the partial t tiles, if they were
    // placed over a tile, went to the other buffer); step i >= 1 rotates tile
    // i - 1 again into buffer (Lb + i) % 2, which every wave last read at
    // step i - 2, before the previous barrier.
    const int a_ch = deflate_channel(lane);
    const float* tn_row = tneg + row * RANK;
    const int Lb = (ntiles - 1) & 1;
    for (int i = 0; i < ntiles; ++i) {
      const int tb = i == 0 ? ntiles - 1 : i - 1;
      float* tile = tiles + ((Lb + i) & 1) * 16 * TS;
      if (i > 0) {
        rotate_tile(rf, tile);
        if (i < ntiles - 1) fetch_tile(i, rf);
      }
      uint32_t l1w[kMaxPerWave][RANK / 2];
#pragma unroll
      for (int k = 0; k < kMaxPerWave; ++k) {
        const int gl = wave + k * nwaves;
        if (gl < npass) load_l1_row<RANK>(L1, (tb * npass + gl) * kGroup + a_ch, l1w[k]);
      }
      lds_sync();
#pragma unroll
      for (int k = 0; k < kMaxPerWave; ++k) {
        const int gl = wave + k * nwaves;
        if (gl < npass) {
          float v[16];
          read_group(tile, gl, v);
          deflate_step<RANK>(v, l1w[k], tn_row);
          store_codes(tb * npass + gl, v);
        }
      }
    }
  }
}

// Few tokens (M <= kFewTokens, K <= KMAX): one 256-thread workgroup per
// token, so that a call of a few tokens spreads over as many CUs as tokens
// instead of running on one.  The same arithmetic as above, laid out for one
// token:
//   rotate:   wave w < ceil(K / 1024) transforms channels 1024 w + 16 lane ..
//             +15 in registers (fwht16) into an LDS row of K floats, and
//             bf16(x~) as doubles into a second row;
//   t:        thread i sums column j = i % r over its range of CH = KMAX r /
//             256 consecutive channels in double, from its L1t row segment
//             (requested at the start); the 256 / r range sums of a column
//             are then added in range order and rounded once to bf16 (the
//             sum is exact up to double rounding, as in the oracle's float64
//             sum);
//   deflate:  thread i takes channels i, i + 256, .. (CPT = KMAX / 256) and
//             removes the r directions from them, j ascending, with its L1
//             rows: cur <- fma(L1[c][j], -t_j, cur) (an exact product, one
//             rounding: the oracle's step);
//   quantize: the rotation waves read their 16 channels per lane back and
//             quantize per group (lanes l, l^1 share a group of 32; l .. l^3
//             one of 64), one code block per lane.
constexpr int kFewTokens = 64;

template <int RANK, int KMAX, bool DEFLATE>
__global__ __launch_bounds__(256) void quantize_act_rotated_few_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ inv_smooth, const uint16_t* __restrict__ L1t,
    const uint16_t* __restrict__ L1, uint8_t* __restrict__ xq, float* __restrict__ xs, uint16_t* __restrict__ t,
    int M, int K, int logB, float hscale, int group) {
  constexpr int Q = 256 / RANK;                 // channel ranges per column of t
  constexpr int CH = KMAX / Q;                  // channels per range
  constexpr int CPT = KMAX / 256;               // channels per thread in the deflation
  // LDS: bf16(x~) row [K] double | range sums [Q][RANK] double | x~ row [K] float | -t [RANK] float
  extern __shared__ double lds_raw[];
  double* xd = lds_raw;
  double* sums = xd + K;
  float* xt = reinterpret_cast<float*>(sums + Q * RANK);
  float* tn = xt + K;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m = blockIdx.x;
  const int npass = (K + 1023) / 1024;
  const int e = wave * 1024 + 16 * lane;        // first channel of this lane's rotation slice
  const bool rot_wave = wave < npass;
  const bool rot_lane = rot_wave && e < K;
  const int tj = tid % RANK;                    // column of t
  const int c0 = (tid / RANK) * CH;             // first channel of the range

  // requests: the lane's x and 1/lambda (rotation waves), the thread's L1t
  // segment and (deflated) its L1 rows, all issued unconditionally as buffer
  // loads (bytes past each array read as zero), so that the rotation waits
  // for its own two requests only and not for the L1t and L1 ones behind them
  const buf_rsrc x_rsrc = make_rsrc(x + static_cast<int64_t>(m) * K, static_cast<uint32_t>(K) * 2u);
  const buf_rsrc inv_rsrc = make_rsrc(inv_smooth, static_cast<uint32_t>(K) * 4u);
  const buf_rsrc lt_rsrc = make_rsrc(L1t, static_cast<uint32_t>(RANK * K) * 2u);
  RotFetch rf;
  rf.xa = buf_load16(x_rsrc, static_cast<uint32_t>(e) * 2u);
  rf.xb = buf_load16(x_rsrc, static_cast<uint32_t>(e) * 2u + 16u);
#pragma unroll
  for (int q = 0; q < 4; ++q)
    rf.inv[q] = __builtin_bit_cast(float4, buf_load16(inv_rsrc, static_cast<uint32_t>(e) * 4u + 16u * q));
  uint4 lt[CH / 8];
#pragma unroll
  for (int k = 0; k < CH / 8; ++k) {
    // a segment past K would read the next row: zero it (its terms are skipped too)
    const uint4 w = buf_load16(lt_rsrc, static_cast<uint32_t>(tj * K + c0 + 8 * k) * 2u);
    lt[k] = c0 + 8 * k < K ? w : make_uint4(0, 0, 0, 0);
  }
  uint32_t l1w[DEFLATE ? CPT : 1][RANK / 2];
  if constexpr (DEFLATE) {
    const buf_rsrc l1_rsrc = make_rsrc(L1, static_cast<uint32_t>(K * RANK) * 2u);
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
#pragma unroll
      for (int q = 0; q < RANK / 8; ++q) {
        const uint4 w = buf_load16(l1_rsrc, static_cast<uint32_t>((tid + 256 * i) * RANK + 8 * q) * 2u);
        l1w[i][4 * q] = w.x;
        l1w[i][4 * q + 1] = w.y;
        l1w[i][4 * q + 2] = w.z;
        l1w[i][4 * q + 3] = w.w;
      }
    }
  }

  // rotate into the LDS rows (lanes past K stay out of every block: B divides K);
  // the other waves rotate zeros and store nothing (a branch around the
  // rotation would let the compiler move the x and 1/lambda requests into it,
  // behind the L1t and L1 ones, and the rotation would wait for all of them)
  {
    float v[16];
    smooth16_regs(rf.xa, rf.xb, rf.inv, v);
    fwht16(v, lane, logB);
    if (rot_lane) {
      float4* dst = reinterpret_cast<float4*>(xt + e);
      double2* dd = reinterpret_cast<double2*>(xd + e);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 f = make_float4(v[4 * q] * hscale, v[4 * q + 1] * hscale, v[4 * q + 2] * hscale,
                                     v[4 * q + 3] * hscale);
        dst[q] = f;
        dd[2 * q] = make_double2(bf16_to_f32(f32_to_bf16_rne(f.x)), bf16_to_f32(f32_to_bf16_rne(f.y)));
        dd[2 * q + 1] = make_double2(bf16_to_f32(f32_to_bf16_rne(f.z)), bf16_to_f32(f32_to_bf16_rne(f.w)));
      }
    }
  }
  __syncthreads();

  // column tj of t over the thread's channel range, in double
  {
    // four interleaved partial sums (a quarter of the dependent chain each):
    // the products are exact in double and each sum is within ~1e-14 of the
    // exact one, so the order does not reach the single rounding to bf16
    double s[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int k = 0; k < CH / 8; ++k) {
      if (c0 + 8 * k < K) {
        const uint32_t w[4] = {lt[k].x, lt[k].y, lt[k].z, lt[k].w};
        const double2* xp = reinterpret_cast<const double2*>(xd + c0 + 8 * k);
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const double2 a = xp[h];
          s[h] = __builtin_fma(a.x, static_cast<double>(__uint_as_float(w[h] << 16)), s[h]);
          s[h] = __builtin_fma(a.y, static_cast<double>(__uint_as_float(w[h] & 0xFFFF0000u)), s[h]);
        }
      }
    }
    sums[(tid / RANK) * RANK + tj] = (s[0] + s[1]) + (s[2] + s[3]);
  }
  __syncthreads();
  if (tid < RANK) {
    double s = 0.0;
    for (int q = 0; q < Q; ++q) s += sums[q * RANK + tid];
    const uint32_t b = f64_to_bf16_rne(s);
    t[static_cast<int64_t>(m) * RANK + tid] = static_cast<uint16_t>(b);
    tn[tid] = -bf16_to_f32(b);
  }

  if constexpr (DEFLATE) {
    __syncthreads();
    // -t and the thread's channels into registers first (the stores into xt
    // would otherwise make every read of tn wait for them); each channel
    // still takes its r updates one after another, j ascending
    float tr[RANK], v[CPT];
#pragma unroll
    for (int j = 0; j < RANK; ++j) tr[j] = tn[j];
#pragma unroll
    for (int i = 0; i < CPT; ++i) v[i] = tid + 256 * i < K ? xt[tid + 256 * i] : 0.0f;
#pragma unroll
    for (int j = 0; j < RANK; j += 2) {
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const uint32_t w = l1w[i][j / 2];
        v[i] = __builtin_fmaf(__uint_as_float(w << 16), tr[j], v[i]);
        v[i] = __builtin_fmaf(__uint_as_float(w & 0xFFFF0000u), tr[j + 1], v[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      if (tid + 256 * i < K) xt[tid + 256 * i] = v[i];
    __syncthreads();
  }

  // quantize the lane's 16 channels; one code block per lane
  if (rot_wave) {
    float v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q] = 0.0f;
    if (rot_lane) {
      const float4* src = reinterpret_cast<const float4*>(xt + e);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 f = src[q];
        v[4 * q] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
      }
    }
    float amax = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; ++q) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[q]));
    // lanes of one group: l, l^1 (32 channels), and l^2, l^3 (64)
    amax = __builtin_fmaxf(amax, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(amax), 0xB1, 0xF, 0xF, false)));
    if (group == kGroup)
      amax = __builtin_fmaxf(amax, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(amax), 0x4E, 0xF, 0xF, false)));
    const float sc = q4_scale(amax);
    const float inv = q4_inv(sc);
    float xs16[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) xs16[q] = v[q] * inv;
    uint32_t d0, d1, d2;
    codes_fp6_16(xs16, d0, d1, d2);
    if (rot_lane) {
      *reinterpret_cast<uint2*>(xq + static_cast<int64_t>(m) * (K / 2) + e / 2) = fp6_code_block(d0, d1, d2);
      if (e % group == 0) xs[static_cast<int64_t>(e / group) * M + m] = sc;
    }
  }
}

// Tile width: the largest multiple of max(B, 64) that divides K and is at
// most 1024.
static int rotate_tile_width(int K, int B) {
  const int base = B > kGroup ? B : kGroup;
  for (int c = 1024 / base; c > 1; --c)
    if ((K / base) % c == 0) return base * c;
  return base;
}

hipError_t launch_quantize_act_rotated(int M, int K, int r, int group, int B, bool deflate, const uint16_t* x,
                                       const float* inv_smooth, const uint16_t* L1t, const uint16_t* L1f,
                                       const uint16_t* L1, uint8_t* xq, float* xs, uint16_t* t,
                                       hipStream_t stream) {
  int logB = 0;
  while ((1 << logB) < B) ++logB;
  if ((1 << logB) != B || B < 16 || B > 1024 || K % B != 0) return hipErrorInvalidValue;
  const int T = rotate_tile_width(K, B);
  // a tile has at most 16 passes / groups: per_wave<r>() per wave
  if (T / kGroup > 16) return hipErrorInvalidValue;
  const float hscale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(B)));
  // few tokens: one workgroup per token (r = 16 up to K = 2048, r = 32 up to K = 1024)
  if (M <= kFewTokens && (r == 16 || r == 32) && K * r <= 256 * 128) {
    auto few = [&](auto kernel) {
      const size_t lds = static_cast<size_t>(K + 256) * sizeof(double) + static_cast<size_t>(K + r) * sizeof(float);
      hipLaunchKernelGGL(kernel, dim3(M), dim3(256), lds, stream, x, inv_smooth, L1t, L1, xq, xs, t, M, K, logB,
                         hscale, group);
      return hipGetLastError();
    };
    const int kmax = K <= 256 ? 256 : K <= 512 ? 512 : K <= 1024 ? 1024 : 2048;
#define QWAM_FEW(R, KM)                                                                             \
  if (r == R && kmax == KM)                                                                         \
    return deflate ? few(quantize_act_rotated_few_kernel<R, KM, true>)                              \
                   : few(quantize_act_rotated_few_kernel<R, KM, false>);
    QWAM_FEW(16, 256) QWAM_FEW(16, 512) QWAM_FEW(16, 1024) QWAM_FEW(16, 2048)
    QWAM_FEW(32, 256) QWAM_FEW(32, 512) QWAM_FEW(32, 1024)
#undef QWAM_FEW
  }
  auto go = [&](auto kernel, int nwaves, size_t acc_bytes) {
    // two tiles, then the partial t tiles, or those over a tile buffer when
    // all of it would not fit in LDS (and they fit in a tile)
    const size_t tile_bytes = static_cast<size_t>(16) * (T + kTilePad) * sizeof(float);
    const size_t red_bytes = static_cast<size_t>(nwaves) * 16 * r * acc_bytes;
    const size_t tneg_bytes = deflate ? 16 * r * sizeof(float) : 0;
    const bool over = 2 * tile_bytes + red_bytes + tneg_bytes > 160 * 1024 && red_bytes <= tile_bytes;
    // over a tile: the buffer the last tile does not use (the deflated
    // variant's second pass reads that tile again)
    const int last_buf = (K / T - 1) & 1;
    const int red_off = static_cast<int>((over ? 1 - last_buf : 2) * tile_bytes / sizeof(float));
    const size_t lds = 2 * tile_bytes + (over ? 0 : red_bytes) + tneg_bytes;
    if (lds > 160 * 1024) return hipErrorInvalidValue;
    if (lds > 64 * 1024) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kernel, dim3((M + 15) / 16), dim3(64 * nwaves), lds, stream, x, inv_smooth, L1f, L1, xq, xs, t,
                       M, K, logB, T, hscale, group == 32 ? 1 : 0, red_off);
    return hipGetLastError();
  };
#define QWAM_ROT_CASE(R)                                                                            \
  case R:                                                                                           \
    return deflate ? go(quantize_act_rotated_kernel<R, true>, act_waves<R>(), sizeof(double))       \
                   : go(quantize_act_rotated_kernel<R, false>, act_waves<R>(), sizeof(float));
  switch (r) {
    QWAM_ROT_CASE(16)
    QWAM_ROT_CASE(32)
    QWAM_ROT_CASE(48)
    QWAM_ROT_CASE(64)
    default:
      return hipErrorInvalidValue;
  }
#undef QWAM_ROT_CASE
}

}  // namespace qwam
