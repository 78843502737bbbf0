// The protected subspace from the AOG accumulator (Sec. 4.2, Eq. 7; the
// procedure of the probe estimator): after the last probe batch the estimate
// is G^ = A / (N P), and in the quantizer's coordinates
//     G~ = H diag(lambda) G^ diag(lambda) H
// (H the orthonormal block Hadamard matrix of the rotation, or the identity).
// V is the top-r eigenvectors of G~, its eigenvalues the action mass of the
// layer's directions (Prop. of App. A.3: the top-r eigenspace minimises the
// quadratic error tr G~ - tr V^T G~ V).
//
// Method: blocked subspace iteration with a final Rayleigh-Ritz step, block
// p = 64 >= r + 16, all on the GPU:
//   * G~ is never formed: each product G~ V is the thin chain
//       X = diag(lambda) H V          (row transform of the block, float32)
//       W = A X                       (split-K GEMM on the FP32 matrix cores)
//       Y = s H diag(lambda) W        (fixed-order sum of the K splits, row transform)
//     A is d x d and read once per product (HBM-bound); the block is p x d
//     and stays in L2;
//   * orthonormalisation by CholeskyQR: Gram matrix in float64 (per-chunk
//     partials, then a fixed-order sum in a kernel of its own), Cholesky and
//     triangular inverse by blocks of 16 rows in one workgroup, then
//     V = W R^-1 (tiled, float64 sums); one pass per iteration, two (i.e.
//     CholeskyQR2) on the block that enters Rayleigh-Ritz;
//   * Rayleigh-Ritz: T = V^T G~ V (p x p, float64), parallel cyclic Jacobi in
//     one workgroup (disjoint rotation pairs by the circle method), Ritz
//     vectors V Q sorted by eigenvalue, descending; the largest-magnitude entry
//     of each is made positive (the convention of the oracle's eigenvectors).
// The start block comes from splitmix64 (Steele, Lea and Flood, 2014) over the
// element index, mapped to [-1, 1).  Every reduction runs in a fixed order, so
// runs are bit-identical.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qwam_device.h"
#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int P = kEigBlock;     // block width (64)
constexpr int NT = 256;
constexpr int GCH = 64;          // columns per Gram partial
constexpr int AT = 32;           // columns (rows of V) per workgroup of the basis update and Ritz step
constexpr int JT = 512;          // threads of the Jacobi workgroup

typedef float v16f __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

// Vt[j][n] uniform in [-1, 1): the top 24 bits of splitmix64(seed + j * d + n)
__global__ __launch_bounds__(NT) void eig_init_kernel(float* __restrict__ Vt, int d, uint64_t seed) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * NT + threadIdx.x;
  if (i >= static_cast<int64_t>(P) * d) return;
  const uint64_t z = splitmix64(seed + static_cast<uint64_t>(i));
  Vt[i] = static_cast<float>(static_cast<int64_t>(z >> 40) - (int64_t(1) << 23)) * 0x1p-23f;
}

// Largest segment length L (a multiple of the Hadamard block B, at most 1024,
// dividing d) handled by one workgroup of the row transforms
int row_segment(int d, int B) {
  int L = B > 1 ? B : 64;
  while (L * 2 <= 1024 && d % (L * 2) == 0) L *= 2;
  return L;
}

// One segment of L entries of one block row per workgroup (grid: d / L
// segments x P rows), in LDS:
//   PRE : out = diag(lam) H in
//   POST: out = scale * H diag(lam) (sum over `nparts` parts of in, in order)
// H: fast Walsh-Hadamard transform of every block of B entries (B = 0: none),
// normalised by 1 / sqrt(B); L is a multiple of B, so every block lies in one
// segment.
template <bool POST>
__global__ __launch_bounds__(NT) void eig_row_kernel(const float* __restrict__ in, int nparts, int64_t part_stride,
                                                     float* __restrict__ out, const float* __restrict__ lam, int B,
                                                     float scale, int d, int L) {
  extern __shared__ float seg[];
  const int c0 = blockIdx.x * L;
  const int64_t base = static_cast<int64_t>(blockIdx.y) * d + c0;
  const int tid = threadIdx.x;
  for (int i4 = tid; i4 < L / 4; i4 += NT) {
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int s = 0; s < nparts; ++s) {
      const float4 p = *reinterpret_cast<const float4*>(in + s * part_stride + base + 4 * i4);
      v.x += p.x;
      v.y += p.y;
      v.z += p.z;
      v.w += p.w;
    }
    if (POST && lam != nullptr) {
      const float4 l = *reinterpret_cast<const float4*>(lam + c0 + 4 * i4);
      v.x *= l.x;
      v.y *= l.y;
      v.z *= l.z;
      v.w *= l.w;
    }
    *reinterpret_cast<float4*>(seg + 4 * i4) = v;
  }
  __syncthreads();
  float norm = 1.0f;
  if (B > 1) {
    for (int h = 1; h < B; h <<= 1) {
      for (int q = tid; q < L / 2; q += NT) {
        const int i = ((q & ~(h - 1)) << 1) | (q & (h - 1));
        const float a = seg[i], b = seg[i + h];
        seg[i] = a + b;
        seg[i + h] = a - b;
      }
      __syncthreads();
    }
    norm = 1.0f / __builtin_sqrtf(static_cast<float>(B));
  }
  for (int i4 = tid; i4 < L / 4; i4 += NT) {
    float4 v = *reinterpret_cast<const float4*>(seg + 4 * i4);
    v.x *= norm;
    v.y *= norm;
    v.z *= norm;
    v.w *= norm;
    if (!POST && lam != nullptr) {
      const float4 l = *reinterpret_cast<const float4*>(lam + c0 + 4 * i4);
      v.x *= l.x;
      v.y *= l.y;
      v.z *= l.z;
      v.w *= l.w;
    }
    if (POST) {
      v.x *= scale;
      v.y *= scale;
      v.z *= scale;
      v.w *= scale;
    }
    *reinterpret_cast<float4*>(out + base + 4 * i4) = v;
  }
}

// part[s][j][n] = sum over k in split s of Xt[j][k] A[n][k]  (A symmetric, so
// this is (A X)[n][j]).  Workgroup: 64 columns n x the 64 block rows j, one
// K split; wave (wm, wn) owns the 32 x 32 block (rows 32 wm.., columns
// 32 wn..) on v_mfma_f32_32x32x2_f32.
//   * Steps of GK = 64 channels: the 64 x 64 tiles of A and Xt are copied
//     straight into LDS (buffer_load ... lds, 16 bytes per lane, one copy
//     instruction filling 4 rows of 256 bytes, i.e. whole cache lines).  Row r
//     keeps its 16-byte chunk c at slot c ^ (r & 15), so the fragment reads
//     (rows r .. r + 15, one chunk) hit distinct banks.  Two stages: the copy
//     of step t + 1 runs during the MFMAs of step t.
//   * Within a step of 8 channels, lane l supplies row / column l % 32 and
//     lane half h channels 4h .. 4h + 3 to four MFMAs (the same channel order
//     on both operands).  Even and odd 8-channel steps go to two accumulators
//     (so consecutive MFMAs of a wave do not wait on each other), added at the
//     end.
constexpr int GK = 64;

__global__ __launch_bounds__(NT) void eig_gemm_kernel(const float* __restrict__ Xt, const float* __restrict__ A,
                                                      float* __restrict__ part, int d, int kchunk) {
  __shared__ __attribute__((aligned(16))) float la0[64 * GK], lx0[64 * GK];
  __shared__ __attribute__((aligned(16))) float la1[64 * GK], lx1[64 * GK];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * 64;
  const int s = blockIdx.y;
  const int k0 = s * kchunk;
  const int nsteps = kchunk / GK;
  const uint32_t rowb = static_cast<uint32_t>(d) * 4u;
  const buf_rsrc a_rsrc = make_rsrc(A + static_cast<int64_t>(n0) * d, 64u * rowb);
  const buf_rsrc x_rsrc = make_rsrc(Xt, 64u * rowb);
  // copy i of this wave: rows 4 (4 wave + i) + lane / 16, slot lane % 16
  uint32_t c_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * (4 * wave + i) + (lane >> 4);
    const int c = (lane & 15) ^ (r & 15);
    c_off[i] = static_cast<uint32_t>(r) * rowb + static_cast<uint32_t>(k0 + 4 * c) * 4u;
  }
  auto issue = [&](int t, float* la, float* lx) __attribute__((always_inline)) {
    const uint32_t ko = static_cast<uint32_t>(t) * GK * 4u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      buf_load16_lds(a_rsrc, c_off[i] + ko, la + (4 * wave + i) * 4 * GK);
      buf_load16_lds(x_rsrc, c_off[i] + ko, lx + (4 * wave + i) * 4 * GK);
    }
  };
  const int ra = wn * 32 + (lane & 31), rx = wm * 32 + (lane & 31);
  const int h = lane >> 5;
  v16f acc0 = {}, acc1 = {};
  auto compute = [&](const float* la, const float* lx) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < GK / 8; ++t) {
      const int c = 2 * t + h;
      const float4 a = *reinterpret_cast<const float4*>(la + ra * GK + 4 * (c ^ (ra & 15)));
      const float4 x = *reinterpret_cast<const float4*>(lx + rx * GK + 4 * (c ^ (rx & 15)));
      v16f& acc = (t & 1) ? acc1 : acc0;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.x, a.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.y, a.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.z, a.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.w, a.w, acc, 0, 0, 0);
    }
  };
  issue(0, la0, lx0);
  for (int t = 0; t < nsteps; t += 2) {
    wait_vmcnt<0>();             // this thread's copies of step t have landed
    lds_barrier();               // ... and every thread's; step t - 1's stage is free
    if (t + 1 < nsteps) issue(t + 1, la1, lx1);
    compute(la0, lx0);
    if (t + 1 < nsteps) {
      wait_vmcnt<0>();
      lds_barrier();
      if (t + 2 < nsteps) issue(t + 2, la0, lx0);
      compute(la1, lx1);
    }
  }
  // result layout: lane l holds column l % 32, rows 8 (v / 4) + 4 (l / 32) + v % 4
  float* out = part + static_cast<int64_t>(s) * P * d;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int j = wm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    out[static_cast<int64_t>(j) * d + n0 + wn * 32 + (lane & 31)] = acc0[v] + acc1[v];
  }
}

// gpart[c][a][b] = sum over the GCH columns n of chunk c of U[a][n] W[b][n],
// float64, n ascending.  Thread (ta, tb) = (tid / 16, tid % 16) owns the 16
// entries a = ta + 16 p, b = tb + 16 q; the chunk passes through LDS in two
// halves of 32 columns, converted to float64 (row stride 34 doubles: the 16
// rows b of one read fall in distinct banks).
__global__ __launch_bounds__(NT) void eig_gram_kernel(const float* __restrict__ Ut, const float* __restrict__ Wt,
                                                      double* __restrict__ gpart, int d) {
  constexpr int HW = 32, RS = HW + 2;
  __shared__ __attribute__((aligned(16))) double us[P][RS], ws[P][RS];
  const int c = blockIdx.x, tid = threadIdx.x;
  const int ta = tid >> 4, tb = tid & 15;
  double acc[4][4];
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[p][q] = 0.0;
  for (int h = 0; h < GCH; h += HW) {
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int e4 = tid + NT * v;            // 512 float4 per array
      const int a = e4 >> 3, c4 = e4 & 7;
      const int64_t g = static_cast<int64_t>(a) * d + c * GCH + h + 4 * c4;
      const float4 u = *reinterpret_cast<const float4*>(Ut + g);
      const float4 w = *reinterpret_cast<const float4*>(Wt + g);
      *reinterpret_cast<double2*>(&us[a][4 * c4]) = make_double2(u.x, u.y);
      *reinterpret_cast<double2*>(&us[a][4 * c4 + 2]) = make_double2(u.z, u.w);
      *reinterpret_cast<double2*>(&ws[a][4 * c4]) = make_double2(w.x, w.y);
      *reinterpret_cast<double2*>(&ws[a][4 * c4 + 2]) = make_double2(w.z, w.w);
    }
    __syncthreads();
#pragma unroll 4
    for (int n = 0; n < HW; n += 2) {
      double2 u[4], w[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) u[p] = *reinterpret_cast<const double2*>(&us[ta + 16 * p][n]);
#pragma unroll
      for (int q = 0; q < 4; ++q) w[q] = *reinterpret_cast<const double2*>(&ws[tb + 16 * q][n]);
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[p][q] = __builtin_fma(u[p].x, w[q].x, acc[p][q]);
          acc[p][q] = __builtin_fma(u[p].y, w[q].y, acc[p][q]);
        }
    }
    __syncthreads();
  }
  double* out = gpart + static_cast<int64_t>(c) * P * P;
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) out[(ta + 16 * p) * P + tb + 16 * q] = acc[p][q];
}

// C[e] = sum of the nch Gram partials of entry e, in chunk order: four
// threads sum consecutive quarters of the chunks, the quarters are added in
// order.  Grid: P * P / 64 workgroups of 64 entries.
__global__ __launch_bounds__(NT) void eig_gsum_kernel(const double* __restrict__ gpart, int nch,
                                                      double* __restrict__ C) {
  __shared__ double red[4][64];
  const int t = threadIdx.x & 63, qtr = threadIdx.x >> 6;
  const int e = blockIdx.x * 64 + t;
  const int c0 = (nch * qtr) / 4, c1 = (nch * (qtr + 1)) / 4;
  double v = 0.0;
#pragma unroll 8
  for (int c = c0; c < c1; ++c) v += gpart[static_cast<int64_t>(c) * P * P + e];
  red[qtr][t] = v;
  __syncthreads();
  if (qtr == 0) C[e] = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
}

// 1/sqrt(x) for x > 0: the hardware estimate refined by two Newton steps
// y <- y + y (1 - x y^2) / 2 (quadratic convergence from its ~2^-22 relative
// error, so the result is within an ulp or two); no division on the chain
__device__ __forceinline__ double rsqrt_f64(double x) {
  double y = __builtin_amdgcn_rsq(x);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const double e = __builtin_fma(-x * y, y, 1.0);
    y = __builtin_fma(0.5 * y, e, y);
  }
  return y;
}

// 1/x for finite x != 0 (|x| below ~1e300): the hardware estimate refined by
// two Newton steps y <- y + y (1 - x y)
__device__ __forceinline__ double rcp_f64(double x) {
  double y = __builtin_amdgcn_rcp(x);
#pragma unroll
  for (int i = 0; i < 2; ++i) y = __builtin_fma(y, __builtin_fma(-x, y, 1.0), y);
  return y;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(u)), l));
  const uint32_t hi =
      static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(u >> 32)), l));
  return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

// C = R^T R (Cholesky, R upper) and Rinv = R^-1 (upper, its lower part exact
// zeros) to global memory, in one workgroup of four waves.  Lane j holds
// column j; wave q holds rows 16 q .. 16 q + 15 of it in registers (blocks of
// 16 rows).  Only the upper triangle of C is read.
//   * Factorisation, right-looking by blocks: the wave that owns diagonal
//     block b factors its 16 rows alone (step k: the pivot from lane k, lane
//     j forms R[k][j], the row goes to LDS and the wave updates its remaining
//     rows of the block); one workgroup barrier; then every wave below the
//     block subtracts the block's rank-16 product from its rows.
//   * A pivot below 1e-13 of the largest diagonal entry (a block of lower
//     rank) is raised to that floor, so the inverse stays finite; the next
//     iterations refill such a direction.
//   * Inverse, R z = e_j for column j, by blocks from the last: the owner wave
//     solves its 16 rows (column-oriented within the block), its rows of z go
//     to LDS, one barrier, and every wave above the block subtracts the
//     block's contribution from its rows.
// Inside a block the row of R reaches the wave's other lanes by cross-lane
// reads (no LDS round trip on the chain of pivots).
constexpr int CB = 16;          // rows per block (and per wave)

__global__ __launch_bounds__(NT) void eig_chol_kernel(const double* __restrict__ C, double* __restrict__ Rinv) {
  __shared__ __attribute__((aligned(16))) double rl[P][P + 2];    // rows of R
  __shared__ __attribute__((aligned(16))) double rc[P][P + 2];    // columns of R: rc[j][k] = R[k][j]
  __shared__ __attribute__((aligned(16))) double zl[P][P + 2];    // rows of R^-1 as they are solved
  __shared__ double dinv[P];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r0 = CB * wave;
  double c[CB];
#pragma unroll
  for (int i = 0; i < CB; ++i) c[i] = C[(r0 + i) * P + lane];
  double m = C[lane * (P + 1)];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double t = __shfl_xor(m, o);
    m = t > m ? t : m;
  }
  const double fl = m > 0.0 ? 1e-13 * m : 1e-300;

#pragma unroll
  for (int b = 0; b < P / CB; ++b) {
    if (wave == b) {
#pragma unroll
      for (int kk = 0; kk < CB; ++kk) {
        const int k = CB * b + kk;
        const double ckk = readlane_f64(c[kk], k);
        const double piv = ckk > fl ? ckk : fl;
        const double inv = rsqrt_f64(piv);              // 1 / R[k][k]
        const double rkk = piv * inv;                   // R[k][k]
        const double rk = lane > k ? c[kk] * inv : (lane == k ? rkk : 0.0);
        c[kk] = rk;
        rl[k][lane] = rk;
        rc[lane][k] = rk;
        if (lane == 0) dinv[k] = inv;
        // R[k][i] of the block's later rows i from lane i (the next pivot's
        // row first)
#pragma unroll
        for (int ii = kk + 1; ii < CB; ++ii) c[ii] = __builtin_fma(-readlane_f64(rk, CB * b + ii), rk, c[ii]);
      }
    }
    __syncthreads();
    if (wave > b) {
#pragma unroll
      for (int kk = 0; kk < CB; ++kk) {
        const int k = CB * b + kk;
        const double rkj = rl[k][lane];
#pragma unroll
        for (int ii = 0; ii < CB; ++ii) c[ii] = __builtin_fma(-rl[k][r0 + ii], rkj, c[ii]);
      }
    }
  }

  double z[CB];
#pragma unroll
  for (int i = 0; i < CB; ++i) z[i] = (r0 + i == lane) ? 1.0 : 0.0;
#pragma unroll
  for (int b = P / CB - 1; b >= 0; --b) {
    if (wave == b) {
#pragma unroll
      for (int ii = CB - 1; ii >= 0; --ii) {
        const int i = CB * b + ii;
        z[ii] *= dinv[i];
        zl[i][lane] = z[ii];
#pragma unroll
        for (int kk = 0; kk < ii; ++kk) z[kk] = __builtin_fma(-rc[i][CB * b + kk], z[ii], z[kk]);
      }
    }
    __syncthreads();
    if (wave < b) {
#pragma unroll
      for (int ii = 0; ii < CB; ++ii) {
        const int i = CB * b + ii;
        const double zi = zl[i][lane];
#pragma unroll
        for (int kk = 0; kk < CB; ++kk) z[kk] = __builtin_fma(-rc[i][r0 + kk], zi, z[kk]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < CB; ++i) Rinv[(r0 + i) * P + lane] = z[i];
}

// Vt[i][n] = sum over k of Rinv[k][i] Wt[k][n] (V = W R^-1; Rinv is zero below
// its diagonal), k ascending, float64, for the AT columns n of the workgroup.
// Thread (ti, tn) = (tid / 16, tid % 16) owns rows 4 ti .. 4 ti + 3 and columns
// 2 tn, 2 tn + 1.
__global__ __launch_bounds__(NT) void eig_apply_kernel(const float* __restrict__ Wt, const double* __restrict__ Rinv,
                                                       float* __restrict__ Vt, int d) {
  __shared__ __attribute__((aligned(16))) double rs[P][P];
  __shared__ __attribute__((aligned(16))) double wsd[P][AT + 2];
  const int tid = threadIdx.x;
  const int n0 = blockIdx.x * AT;
  for (int e = tid; e < P * P / 2; e += NT)
    *reinterpret_cast<double2*>(&rs[0][2 * e]) = reinterpret_cast<const double2*>(Rinv)[e];
  for (int e = tid; e < P * AT / 4; e += NT) {
    const int k = e / (AT / 4), c4 = e % (AT / 4);
    const float4 w = *reinterpret_cast<const float4*>(Wt + static_cast<int64_t>(k) * d + n0 + 4 * c4);
    *reinterpret_cast<double2*>(&wsd[k][4 * c4]) = make_double2(w.x, w.y);
    *reinterpret_cast<double2*>(&wsd[k][4 * c4 + 2]) = make_double2(w.z, w.w);
  }
  __syncthreads();
  const int ti = tid >> 4, tn = tid & 15;
  double acc[4][2];
#pragma unroll
  for (int p = 0; p < 4; ++p) acc[p][0] = acc[p][1] = 0.0;
#pragma unroll 8
  for (int k = 0; k < P; ++k) {
    const double2 r01 = *reinterpret_cast<const double2*>(&rs[k][4 * ti]);
    const double2 r23 = *reinterpret_cast<const double2*>(&rs[k][4 * ti + 2]);
    const double2 w = *reinterpret_cast<const double2*>(&wsd[k][2 * tn]);
    const double r[4] = {r01.x, r01.y, r23.x, r23.y};
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      acc[p][0] = __builtin_fma(r[p], w.x, acc[p][0]);
      acc[p][1] = __builtin_fma(r[p], w.y, acc[p][1]);
    }
  }
#pragma unroll
  for (int p = 0; p < 4; ++p)
    *reinterpret_cast<float2*>(Vt + static_cast<int64_t>(4 * ti + p) * d + n0 + 2 * tn) =
        make_float2(static_cast<float>(acc[p][0]), static_cast<float>(acc[p][1]));
}

// One workgroup: T = the summed V^T (G~ V), symmetrised; cyclic Jacobi with
// the 32 disjoint pairs of each round of the circle method (index 0 fixed,
// 1 .. 63 rotating), a sweep being 63 rounds; the rotation of each pair zeroes
// T[a][b] (Golub and Van Loan's symmetric 2 x 2 Schur step).  The pairs of a
// round are disjoint and cover every index, so T <- J^T T J splits into the
// 32 x 32 independent 2 x 2 blocks (rows of pair k, columns of pair m), each
// updated in one pass (rows, then columns), and Q <- Q J into 64 x 32
// independent row pairs.  Stops when the off-diagonal mass is below 1e-26 of
// the diagonal's, or after 30 sweeps.  Out: theta (eigenvalues, descending),
// Q (its columns the eigenvectors of T in that order), both float64.
__global__ __launch_bounds__(JT) void eig_jacobi_kernel(const double* __restrict__ C, double* __restrict__ Qout,
                                                        double* __restrict__ theta) {
  __shared__ double t[P][P + 1], q[P][P + 1];
  __shared__ double2 rot[P / 2];
  __shared__ int2 prs[P / 2];
  __shared__ double red[2][JT];
  __shared__ int order[P];
  __shared__ int done;
  const int tid = threadIdx.x;
  for (int e = tid; e < P * P; e += JT) {
    const int a = e / P, b = e % P;
    t[a][b] = a == b ? C[e] : 0.5 * (C[a * P + b] + C[b * P + a]);
    q[a][b] = a == b ? 1.0 : 0.0;
  }
  __syncthreads();
  const int bk = tid >> 4, bm0 = tid & 15;     // T blocks (bk, bm0 + 16 j)
  const int qm = tid & 31, qi0 = tid >> 5;     // Q rows qi0 + 16 u of pair qm
  for (int sweep = 0; sweep < 30; ++sweep) {
    double off = 0.0, dia = 0.0;
    for (int e = tid; e < P * P; e += JT) {
      const double v = t[e / P][e % P];
      if (e / P == e % P) dia += v * v; else off += v * v;
    }
    red[0][tid] = off;
    red[1][tid] = dia;
    __syncthreads();
    for (int w = JT / 2; w > 0; w >>= 1) {
      if (tid < w) {
        red[0][tid] += red[0][tid + w];
        red[1][tid] += red[1][tid + w];
      }
      __syncthreads();
    }
    if (tid == 0) done = !(red[0][0] > 1e-26 * red[1][0]);
    __syncthreads();
    if (done) break;
    for (int round = 0; round < P - 1; ++round) {
      if (tid < P / 2) {
        const int k = tid;
        const int pa = (k == 0) ? 0 : ((k - 1 + round) % (P - 1)) + 1;
        const int pb = ((P - 1 - k - 1 + round) % (P - 1)) + 1;
        const int a = pa < pb ? pa : pb, b = pa < pb ? pb : pa;
        double c = 1.0, s = 0.0;
        const double apq = t[a][b];
        if (apq != 0.0) {
          // tau = (T_bb - T_aa) / (2 T_ab); tt = sign(tau) / (|tau| + sqrt(1 + tau^2)),
          // the smaller root of tt^2 + 2 tau tt - 1 = 0; c = 1 / sqrt(1 + tt^2).
          // Reciprocals and square roots by refined hardware estimates; a
          // |tau| beyond 1e100 (tau^2 would overflow) takes tt = 1 / (2 tau)
          const double diff = t[b][b] - t[a][a];
          const double aa = __builtin_fabs(apq);
          double tt;
          if (__builtin_fabs(diff) > 1e100 * aa) {
            tt = 0.5 * apq / diff;
          } else {
            const double tau = diff * rcp_f64(2.0 * apq);
            const double q = 1.0 + tau * tau;
            const double root = q * rsqrt_f64(q);
            tt = (tau >= 0.0 ? 1.0 : -1.0) * rcp_f64(__builtin_fabs(tau) + root);
          }
          c = rsqrt_f64(1.0 + tt * tt);
          s = tt * c;
        }
        prs[k] = make_int2(a, b);
        rot[k] = make_double2(c, s);
      }
      __syncthreads();
      {
        const int2 ab = prs[bk];
        const double2 cs = rot[bk];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int bm = bm0 + 16 * j;
          const int2 ef = prs[bm];
          const double2 cs2 = rot[bm];
          const double xae = t[ab.x][ef.x], xaf = t[ab.x][ef.y], xbe = t[ab.y][ef.x], xbf = t[ab.y][ef.y];
          const double yae = cs.x * xae - cs.y * xbe, yaf = cs.x * xaf - cs.y * xbf;
          const double ybe = cs.y * xae + cs.x * xbe, ybf = cs.y * xaf + cs.x * xbf;
          t[ab.x][ef.x] = cs2.x * yae - cs2.y * yaf;
          t[ab.x][ef.y] = cs2.y * yae + cs2.x * yaf;
          t[ab.y][ef.x] = cs2.x * ybe - cs2.y * ybf;
          t[ab.y][ef.y] = cs2.y * ybe + cs2.x * ybf;
        }
        const int2 gh = prs[qm];
        const double2 cq = rot[qm];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = qi0 + 16 * u;
          const double qa = q[i][gh.x], qb = q[i][gh.y];
          q[i][gh.x] = cq.x * qa - cq.y * qb;
          q[i][gh.y] = cq.y * qa + cq.x * qb;
        }
      }
      __syncthreads();
    }
  }
  // order by eigenvalue, descending (ties: lower index first)
  if (tid < P) {
    const double v = t[tid][tid];
    int pos = 0;
    for (int j = 0; j < P; ++j) {
      const double w = t[j][j];
      if (w > v || (w == v && j < tid)) ++pos;
    }
    order[pos] = tid;
  }
  __syncthreads();
  if (tid < P) theta[tid] = t[order[tid]][order[tid]];
  for (int e = tid; e < P * P; e += JT) {
    const int i = e / P, col = e % P;
    Qout[i * P + col] = q[i][order[col]];
  }
}

// V[n][i] = sum over j of Vt[j][n] Q[j][i] for i < r (Ritz vectors, float64
// sums, j ascending) over the AT rows n of the workgroup; then per column the
// entry of largest magnitude among those rows (the first row on ties): its
// signed value and its row.  Thread (tn, ti0) = (tid % 32, tid / 32) owns
// row n0 + tn, columns ti0 + 8 u.
__global__ __launch_bounds__(NT) void eig_ritz_kernel(const float* __restrict__ Vt, const double* __restrict__ Q,
                                                      float* __restrict__ V, float* __restrict__ cmax,
                                                      int* __restrict__ cidx, int d, int r) {
  __shared__ double qs[P][kEigMaxRank];
  __shared__ double vs[P][AT + 1];
  __shared__ float out[AT][kEigMaxRank + 1];
  const int tid = threadIdx.x;
  const int n0 = blockIdx.x * AT;
  for (int e = tid; e < P * r; e += NT) qs[e / r][e % r] = Q[(e / r) * P + (e % r)];
  for (int e = tid; e < P * AT; e += NT) {
    const int k = e / AT, c = e % AT;
    vs[k][c] = Vt[static_cast<int64_t>(k) * d + n0 + c];
  }
  __syncthreads();
  const int tn = tid & 31, ti0 = tid >> 5;
  constexpr int U = kEigMaxRank / 8;
  double acc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) acc[u] = 0.0;
  for (int k = 0; k < P; ++k) {
    const double v = vs[k][tn];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (ti0 + 8 * u < r) acc[u] = __builtin_fma(v, qs[k][ti0 + 8 * u], acc[u]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (ti0 + 8 * u < r) out[tn][ti0 + 8 * u] = static_cast<float>(acc[u]);
  __syncthreads();
  for (int e = tid; e < AT * r; e += NT) V[static_cast<int64_t>(n0) * r + e] = out[e / r][e % r];
  if (tid < r) {
    float best = -1.0f, bval = 0.0f;
    int bidx = 0;
    for (int c = 0; c < AT; ++c) {
      const float f = out[c][tid];
      if (__builtin_fabsf(f) > best) {
        best = __builtin_fabsf(f);
        bval = f;
        bidx = n0 + c;
      }
    }
    cmax[blockIdx.x * r + tid] = bval;
    cidx[blockIdx.x * r + tid] = bidx;
  }
}

// Each workgroup finds, for every column, the entry of largest magnitude (the
// first row on ties) among the per-workgroup maxima, and flips its own AT rows
// of the column if that entry is negative (only the maxima written by the
// previous launch are read, never another workgroup's rows); workgroup 0
// writes the r eigenvalues.  The scan: thread (part, column) takes every
// (NT / r)-th block maximum, the parts are merged in LDS.
__device__ __forceinline__ bool better_max(float am, int mi, float best, int bidx) {
  return am > best || (am == best && mi < bidx);
}

__global__ __launch_bounds__(NT) void eig_sign_kernel(float* __restrict__ V, const float* __restrict__ cmax,
                                                      const int* __restrict__ cidx, int nblk,
                                                      const double* __restrict__ theta, float* __restrict__ evals,
                                                      int r) {
  __shared__ float sgn[kEigMaxRank];
  __shared__ float pbest[NT], pval[NT];
  __shared__ int pidx[NT];
  const int tid = threadIdx.x;
  const int parts = NT / r;
  const int i = tid % r, part = tid / r;
  float best = -1.0f, bval = 0.0f;
  int bidx = 0x7fffffff;
  if (part < parts) {
    for (int b = part; b < nblk; b += parts) {
      const float m = cmax[b * r + i];
      const int mi = cidx[b * r + i];
      if (better_max(__builtin_fabsf(m), mi, best, bidx)) {
        best = __builtin_fabsf(m);
        bval = m;
        bidx = mi;
      }
    }
  }
  pbest[tid] = best;
  pval[tid] = bval;
  pidx[tid] = bidx;
  __syncthreads();
  if (tid < r) {
    for (int q = 1; q < parts; ++q) {
      const int o = q * r + tid;
      if (better_max(pbest[o], pidx[o], best, bidx)) {
        best = pbest[o];
        bval = pval[o];
        bidx = pidx[o];
      }
    }
    sgn[tid] = bval < 0.0f ? -1.0f : 1.0f;
    if (blockIdx.x == 0) evals[tid] = static_cast<float>(theta[tid]);
  }
  __syncthreads();
  float* tile = V + static_cast<int64_t>(blockIdx.x) * AT * r;
  for (int e = tid; e < AT * r; e += NT) tile[e] *= sgn[e % r];
}

int gemm_splits(int d) {
  int s = d / 512;
  s = s < 1 ? 1 : (s > 8 ? 8 : s);
  while (s > 1 && (d % s != 0 || (d / s) % 64 != 0)) --s;
  return s;
}

struct EigWs {
  float *Vt, *Wt, *Xt, *part;
  double *gpart, *C, *Rinv, *Q, *theta;
  float* cmax;
  int* cidx;
};

int64_t align256(int64_t b) { return (b + 255) & ~int64_t(255); }

int64_t layout(int d, int r, char* base, EigWs* w) {
  const int S = gemm_splits(d);
  const int64_t blk = static_cast<int64_t>(P) * d * 4;
  const int nblk = d / AT;
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  char* vt = take(blk);
  char* wt = take(blk);
  char* xt = take(blk);
  char* part = take(blk * S);
  char* gp = take(static_cast<int64_t>(d / GCH) * P * P * 8);
  char* cs = take(P * P * 8);
  char* ri = take(P * P * 8);
  char* q = take(P * P * 8);
  char* th = take(P * 8);
  char* cm = take(static_cast<int64_t>(nblk) * r * 4);
  char* ci = take(static_cast<int64_t>(nblk) * r * 4);
  if (w) {
    w->Vt = reinterpret_cast<float*>(vt);
    w->Wt = reinterpret_cast<float*>(wt);
    w->Xt = reinterpret_cast<float*>(xt);
    w->part = reinterpret_cast<float*>(part);
    w->gpart = reinterpret_cast<double*>(gp);
    w->C = reinterpret_cast<double*>(cs);
    w->Rinv = reinterpret_cast<double*>(ri);
    w->Q = reinterpret_cast<double*>(q);
    w->theta = reinterpret_cast<double*>(th);
    w->cmax = reinterpret_cast<float*>(cm);
    w->cidx = reinterpret_cast<int*>(ci);
  }
  return off;
}

}  // namespace

int64_t eig_workspace_bytes(int d, int r) { return layout(d, r, nullptr, nullptr); }

hipError_t launch_aog_eig(int d, int r, int iters, const float* A, float scale, const float* lam, int B,
                          float* V, float* evals, void* workspace, hipStream_t st) {
  EigWs w;
  layout(d, r, static_cast<char*>(workspace), &w);
  const int S = gemm_splits(d);
  const int nch = d / GCH;
  const int nblk = d / AT;
  const int L = row_segment(d, B);
  const size_t seg_lds = static_cast<size_t>(L) * sizeof(float);
  const bool pre = (lam != nullptr) || B > 1;

  // block -> block: G~ applied to the rows of `in` (p x d), into `out`
  auto apply_op = [&](const float* in, float* out) {
    const float* x = in;
    if (pre) {
      hipLaunchKernelGGL(eig_row_kernel<false>, dim3(d / L, P), dim3(NT), seg_lds, st, in, 1, int64_t(0), w.Xt,
                         lam, B, 1.0f, d, L);
      x = w.Xt;
    }
    hipLaunchKernelGGL(eig_gemm_kernel, dim3(d / 64, S), dim3(NT), 0, st, x, A, w.part, d, d / S);
    hipLaunchKernelGGL(eig_row_kernel<true>, dim3(d / L, P), dim3(NT), seg_lds, st, w.part, S,
                       static_cast<int64_t>(P) * d, out, lam, B, scale, d, L);
  };
  // C = U W^T (float64) from the block rows of U and W
  auto gram = [&](const float* u, const float* wv) {
    hipLaunchKernelGGL(eig_gram_kernel, dim3(nch), dim3(NT), 0, st, u, wv, w.gpart, d);
    hipLaunchKernelGGL(eig_gsum_kernel, dim3(P * P / 64), dim3(NT), 0, st, w.gpart, nch, w.C);
  };
  // rows of `src` orthonormalised into `dst` (one CholeskyQR pass)
  auto orth = [&](const float* src, float* dst) {
    gram(src, src);
    hipLaunchKernelGGL(eig_chol_kernel, dim3(1), dim3(NT), 0, st, w.C, w.Rinv);
    hipLaunchKernelGGL(eig_apply_kernel, dim3(nblk), dim3(NT), 0, st, src, w.Rinv, dst, d);
  };

  hipLaunchKernelGGL(eig_init_kernel, dim3((P * d + NT - 1) / NT), dim3(NT), 0, st, w.Vt, d,
                     static_cast<uint64_t>(0x51ED2701ull));
  // one CholeskyQR pass per iteration (the next product only needs a
  // well-conditioned block); the block that enters Rayleigh-Ritz gets the
  // second pass of CholeskyQR2
  orth(w.Vt, w.Wt);
  for (int it = 0; it < iters; ++it) {
    apply_op(w.Wt, w.Vt);
    orth(w.Vt, w.Wt);
  }
  orth(w.Wt, w.Vt);
  // Rayleigh-Ritz on the final block
  apply_op(w.Vt, w.Wt);
  gram(w.Vt, w.Wt);
  hipLaunchKernelGGL(eig_jacobi_kernel, dim3(1), dim3(JT), 0, st, w.C, w.Q, w.theta);
  hipLaunchKernelGGL(eig_ritz_kernel, dim3(nblk), dim3(NT), 0, st, w.Vt, w.Q, V, w.cmax, w.cidx, d, r);
  hipLaunchKernelGGL(eig_sign_kernel, dim3(nblk), dim3(NT), 0, st, V, w.cmax, w.cidx, nblk, w.theta, evals, r);
  return hipGetLastError();
}

}  // namespace qwam
