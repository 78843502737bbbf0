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
//   * orthonormalisation by CholeskyQR2: Gram matrix in float64 (fixed-order
//     sum of per-chunk partials), Cholesky and triangular inverse in one
//     workgroup, then V = W R^-1;
//   * Rayleigh-Ritz: T = V^T G~ V (p x p, float64), parallel cyclic Jacobi in
//     one workgroup (disjoint rotation pairs by the circle method), Ritz
//     vectors V Q sorted by eigenvalue, descending; the largest-magnitude entry
//     of each is made positive (the convention of the oracle's eigenvectors).
// The start block comes from splitmix64 (Steele, Lea and Flood, 2014) over the
// element index, mapped to [-1, 1).  Every reduction runs in a fixed order, so
// runs are bit-identical.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qwam_internal.h"

namespace qwam {

namespace {

constexpr int P = kEigBlock;     // block width (64)
constexpr int NT = 256;
constexpr int GCH = 64;          // columns per Gram partial

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

// One row (a block vector) per workgroup, in LDS:
//   PRE : out = diag(lam) H in
//   POST: out = scale * H diag(lam) (sum over `nparts` parts of in, in order)
// H: fast Walsh-Hadamard transform of every block of B entries (B = 0: none),
// normalised by 1 / sqrt(B).
template <bool POST>
__global__ __launch_bounds__(NT) void eig_row_kernel(const float* __restrict__ in, int nparts, int64_t part_stride,
                                                     float* __restrict__ out, const float* __restrict__ lam, int B,
                                                     float scale, int d) {
  extern __shared__ float row[];
  const int j = blockIdx.x;
  const int tid = threadIdx.x;
  for (int i = tid; i < d; i += NT) {
    float v = 0.0f;
    for (int s = 0; s < nparts; ++s) v += in[s * part_stride + static_cast<int64_t>(j) * d + i];
    if (POST && lam != nullptr) v *= lam[i];
    row[i] = v;
  }
  __syncthreads();
  float norm = 1.0f;
  if (B > 1) {
    for (int h = 1; h < B; h <<= 1) {
      for (int q = tid; q < d / 2; q += NT) {
        const int i = (q / h) * 2 * h + (q % h);
        const float a = row[i], b = row[i + h];
        row[i] = a + b;
        row[i + h] = a - b;
      }
      __syncthreads();
    }
    norm = 1.0f / __builtin_sqrtf(static_cast<float>(B));
  }
  for (int i = tid; i < d; i += NT) {
    float v = row[i] * norm;
    if (!POST && lam != nullptr) v *= lam[i];
    if (POST) v *= scale;
    out[static_cast<int64_t>(j) * d + i] = v;
  }
}

// part[s][j][n] = sum over k in split s of Xt[j][k] A[n][k]  (A symmetric, so
// this is (A X)[n][j]).  Workgroup: 64 columns n x the 64 block rows j, one
// K split; wave (wm, wn) owns the 32 x 32 block (rows 32 wm.., columns
// 32 wn..) on v_mfma_f32_32x32x2_f32.  Lane l supplies row / column l % 32;
// within a step of 8 channels, lane half h supplies channels 4h .. 4h+3 to
// the four MFMAs (the same channel order on both operands), so each lane
// reads 16 contiguous bytes of a row of Xt and of A.
__global__ __launch_bounds__(NT) void eig_gemm_kernel(const float* __restrict__ Xt, const float* __restrict__ A,
                                                      float* __restrict__ part, int d, int kchunk) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * 64;
  const int s = blockIdx.y;
  const int jrow = wm * 32 + (lane & 31);
  const int nrow = n0 + wn * 32 + (lane & 31);
  const int64_t k0 = static_cast<int64_t>(s) * kchunk + 4 * (lane >> 5);
  const float4* xp = reinterpret_cast<const float4*>(Xt + static_cast<int64_t>(jrow) * d + k0);
  const float4* ap = reinterpret_cast<const float4*>(A + static_cast<int64_t>(nrow) * d + k0);
  v16f acc = {};
  for (int k = 0; k < kchunk; k += 8) {
    const float4 x = xp[k / 4];
    const float4 a = ap[k / 4];
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.x, a.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.y, a.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.z, a.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x.w, a.w, acc, 0, 0, 0);
  }
  // result layout: lane l holds column l % 32, rows 8 (v / 4) + 4 (l / 32) + v % 4
  float* out = part + static_cast<int64_t>(s) * P * d;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int j = wm * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    out[static_cast<int64_t>(j) * d + n0 + wn * 32 + (lane & 31)] = acc[v];
  }
}

// gpart[c][a][b] = sum over the GCH columns n of chunk c of U[a][n] W[b][n], float64
__global__ __launch_bounds__(NT) void eig_gram_kernel(const float* __restrict__ Ut, const float* __restrict__ Wt,
                                                      double* __restrict__ gpart, int d) {
  __shared__ float us[P][GCH + 1], ws[P][GCH + 1];
  const int c = blockIdx.x, tid = threadIdx.x;
  for (int e = tid; e < P * GCH; e += NT) {
    const int a = e / GCH, n = e % GCH;
    us[a][n] = Ut[static_cast<int64_t>(a) * d + c * GCH + n];
    ws[a][n] = Wt[static_cast<int64_t>(a) * d + c * GCH + n];
  }
  __syncthreads();
  const int a = tid >> 2, b0 = (tid & 3) * 16;
  double acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0;
  for (int n = 0; n < GCH; ++n) {
    const double u = us[a][n];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = __builtin_fma(u, static_cast<double>(ws[b0 + i][n]), acc[i]);
  }
  double* out = gpart + static_cast<int64_t>(c) * P * P + a * P + b0;
#pragma unroll
  for (int i = 0; i < 16; ++i) out[i] = acc[i];
}

// sum of the Gram partials in chunk order, symmetrised, into g[P][P] (LDS)
__device__ void gram_sum(const double* __restrict__ gpart, int nch, double (*g)[P + 1]) {
  const int tid = threadIdx.x;
  for (int e = tid; e < P * P; e += NT) {
    double v = 0.0;
    for (int c = 0; c < nch; ++c) v += gpart[static_cast<int64_t>(c) * P * P + e];
    g[e / P][e % P] = v;
  }
  __syncthreads();
  for (int e = tid; e < P * P; e += NT) {
    const int a = e / P, b = e % P;
    if (a < b) {
      const double v = 0.5 * (g[a][b] + g[b][a]);
      g[a][b] = v;
      g[b][a] = v;
    }
  }
  __syncthreads();
}

// One workgroup: C = sum of the Gram partials; C = R^T R (Cholesky, R upper);
// Rinv = R^-1 (upper) to global memory.  A pivot below 1e-13 of the largest
// diagonal entry (a block of lower rank) is raised to that floor, so the
// inverse stays finite; the next iterations refill such a direction.
__global__ __launch_bounds__(NT) void eig_chol_kernel(const double* __restrict__ gpart, int nch,
                                                      double* __restrict__ Rinv) {
  __shared__ double c[P][P + 1], r[P][P + 1];
  __shared__ double floor_v;
  const int tid = threadIdx.x;
  gram_sum(gpart, nch, c);
  if (tid == 0) {
    double m = 0.0;
    for (int a = 0; a < P; ++a) m = c[a][a] > m ? c[a][a] : m;
    floor_v = m > 0.0 ? 1e-13 * m : 1e-300;
  }
  for (int e = tid; e < P * P; e += NT) r[e / P][e % P] = 0.0;
  __syncthreads();
  for (int k = 0; k < P; ++k) {
    if (tid == 0) {
      const double piv = c[k][k] > floor_v ? c[k][k] : floor_v;
      r[k][k] = __builtin_sqrt(piv);
    }
    __syncthreads();
    for (int j = k + 1 + tid; j < P; j += NT) r[k][j] = c[k][j] / r[k][k];
    __syncthreads();
    for (int e = tid; e < P * P; e += NT) {
      const int i = e / P, j = e % P;
      if (i > k && j >= i) {
        const double v = c[i][j] - r[k][i] * r[k][j];
        c[i][j] = v;
        c[j][i] = v;
      }
    }
    __syncthreads();
  }
  // column col of R^-1 by back substitution (R x = e_col), one thread per
  // column, into c (no longer needed): thread col only touches column col
  if (tid < P) {
    const int col = tid;
    for (int i = P - 1; i >= 0; --i) {
      double v = 0.0;
      if (i <= col) {
        v = (i == col) ? 1.0 : 0.0;
        for (int k = i + 1; k <= col; ++k) v -= r[i][k] * c[k][col];
        v /= r[i][i];
      }
      c[i][col] = v;
    }
  }
  __syncthreads();
  for (int e = tid; e < P * P; e += NT) Rinv[e] = c[e / P][e % P];
}

// Vt[i][n] = sum_{k <= i} Rinv[k][i] W[k][n]  (V = W R^-1), one thread per column n
__global__ __launch_bounds__(NT) void eig_apply_kernel(const float* __restrict__ Wt, const double* __restrict__ Rinv,
                                                       float* __restrict__ Vt, int d) {
  __shared__ double ri[P * P];
  for (int e = threadIdx.x; e < P * P; e += NT) ri[e] = Rinv[e];
  __syncthreads();
  const int n = blockIdx.x * NT + threadIdx.x;
  if (n >= d) return;
  double w[P];
#pragma unroll
  for (int k = 0; k < P; ++k) w[k] = Wt[static_cast<int64_t>(k) * d + n];
#pragma unroll
  for (int i = 0; i < P; ++i) {
    double v = 0.0;
#pragma unroll
    for (int k = 0; k <= i; ++k) v = __builtin_fma(ri[k * P + i], w[k], v);
    Vt[static_cast<int64_t>(i) * d + n] = static_cast<float>(v);
  }
}

// One workgroup: T = sum of the partials of V^T (G~ V), symmetrised; cyclic
// Jacobi with the 32 disjoint pairs of each round of the circle method (index 0
// fixed, 1 .. 63 rotating), a sweep being 63 rounds; the rotation of each pair
// zeroes T[a][b] (Golub and Van Loan's symmetric 2 x 2 Schur step); stops when
// the off-diagonal mass is below 1e-26 of the diagonal's, or after 30 sweeps.
// Out: theta (eigenvalues, descending), Q (its columns the eigenvectors of T in
// that order), both float64.
__global__ __launch_bounds__(NT) void eig_jacobi_kernel(const double* __restrict__ gpart, int nch,
                                                        double* __restrict__ Qout, double* __restrict__ theta) {
  __shared__ double t[P][P + 1], q[P][P + 1];
  __shared__ double rc[P / 2], rs[P / 2];
  __shared__ int ra[P / 2], rb[P / 2];
  __shared__ double red[NT];
  __shared__ int order[P];
  __shared__ int done;
  const int tid = threadIdx.x;
  gram_sum(gpart, nch, t);
  for (int e = tid; e < P * P; e += NT) q[e / P][e % P] = (e / P == e % P) ? 1.0 : 0.0;
  if (tid == 0) done = 0;
  __syncthreads();
  for (int sweep = 0; sweep < 30; ++sweep) {
    // convergence test
    double off = 0.0, dia = 0.0;
    for (int e = tid; e < P * P; e += NT) {
      const double v = t[e / P][e % P];
      if (e / P == e % P) dia += v * v; else off += v * v;
    }
    red[tid] = off;
    __syncthreads();
    for (int w = NT / 2; w > 0; w >>= 1) {
      if (tid < w) red[tid] += red[tid + w];
      __syncthreads();
    }
    const double off_all = red[0];
    __syncthreads();
    red[tid] = dia;
    __syncthreads();
    for (int w = NT / 2; w > 0; w >>= 1) {
      if (tid < w) red[tid] += red[tid + w];
      __syncthreads();
    }
    if (tid == 0) done = !(off_all > 1e-26 * red[0]);
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
          const double tau = (t[b][b] - t[a][a]) / (2.0 * apq);
          const double tt = (tau >= 0.0 ? 1.0 : -1.0) / (__builtin_fabs(tau) + __builtin_sqrt(1.0 + tau * tau));
          c = 1.0 / __builtin_sqrt(1.0 + tt * tt);
          s = tt * c;
        }
        ra[k] = a;
        rb[k] = b;
        rc[k] = c;
        rs[k] = s;
      }
      __syncthreads();
      // rows: T <- J^T T
      for (int e = tid; e < (P / 2) * P; e += NT) {
        const int k = e / P, j = e % P;
        const int a = ra[k], b = rb[k];
        const double c = rc[k], s = rs[k];
        const double ta = t[a][j], tb = t[b][j];
        t[a][j] = c * ta - s * tb;
        t[b][j] = s * ta + c * tb;
      }
      __syncthreads();
      // columns: T <- T J, Q <- Q J
      for (int e = tid; e < (P / 2) * P; e += NT) {
        const int k = e / P, i = e % P;
        const int a = ra[k], b = rb[k];
        const double c = rc[k], s = rs[k];
        const double ta = t[i][a], tb = t[i][b];
        t[i][a] = c * ta - s * tb;
        t[i][b] = s * ta + c * tb;
        const double qa = q[i][a], qb = q[i][b];
        q[i][a] = c * qa - s * qb;
        q[i][b] = s * qa + c * qb;
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
  for (int e = tid; e < P * P; e += NT) {
    const int i = e / P, col = e % P;
    Qout[i * P + col] = q[i][order[col]];
  }
}

// V[n][i] = sum_j Vt[j][n] Q[j][i] for i < r (Ritz vectors, float64 sums), and
// per workgroup and column the entry of largest magnitude (the first row on
// ties): its signed value and its row
__global__ __launch_bounds__(NT) void eig_ritz_kernel(const float* __restrict__ Vt, const double* __restrict__ Q,
                                                      float* __restrict__ V, float* __restrict__ cmax,
                                                      int* __restrict__ cidx, int d, int r) {
  __shared__ double qs[P * kEigMaxRank];
  __shared__ float bm[NT], bv[NT];
  __shared__ int bi[NT];
  for (int e = threadIdx.x; e < P * r; e += NT) qs[e] = Q[(e / r) * P + (e % r)];
  __syncthreads();
  const int n = blockIdx.x * NT + threadIdx.x;
  double w[P];
#pragma unroll
  for (int k = 0; k < P; ++k) w[k] = (n < d) ? Vt[static_cast<int64_t>(k) * d + n] : 0.0f;
  for (int i = 0; i < r; ++i) {
    double v = 0.0;
    for (int k = 0; k < P; ++k) v = __builtin_fma(w[k], qs[k * r + i], v);
    const float f = static_cast<float>(v);
    if (n < d) V[static_cast<int64_t>(n) * r + i] = f;
    bm[threadIdx.x] = (n < d) ? __builtin_fabsf(f) : -1.0f;
    bv[threadIdx.x] = f;
    bi[threadIdx.x] = n;
    __syncthreads();
    for (int s = NT / 2; s > 0; s >>= 1) {
      if (threadIdx.x < s) {
        const float o = bm[threadIdx.x + s];
        const int oi = bi[threadIdx.x + s];
        if (o > bm[threadIdx.x] || (o == bm[threadIdx.x] && oi < bi[threadIdx.x])) {
          bm[threadIdx.x] = o;
          bv[threadIdx.x] = bv[threadIdx.x + s];
          bi[threadIdx.x] = oi;
        }
      }
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      cmax[blockIdx.x * r + i] = bv[0];
      cidx[blockIdx.x * r + i] = bi[0];
    }
    __syncthreads();
  }
}

// Each workgroup finds, for every column, the entry of largest magnitude (the
// first row on ties) among the per-workgroup maxima, and flips its own rows
// of the column if that entry is negative (only the maxima written by the
// previous launch are read, never another workgroup's rows); workgroup 0
// writes the r eigenvalues.
__global__ __launch_bounds__(NT) void eig_sign_kernel(float* __restrict__ V, const float* __restrict__ cmax,
                                                      const int* __restrict__ cidx, int nblk,
                                                      const double* __restrict__ theta, float* __restrict__ evals,
                                                      int d, int r) {
  __shared__ float sgn[kEigMaxRank];
  if (threadIdx.x < r) {
    const int i = threadIdx.x;
    float best = -1.0f, bval = 0.0f;
    int bidx = 0;
    for (int b = 0; b < nblk; ++b) {
      const float m = cmax[b * r + i];
      const int mi = cidx[b * r + i];
      const float am = __builtin_fabsf(m);
      if (am > best || (am == best && mi < bidx)) {
        best = am;
        bval = m;
        bidx = mi;
      }
    }
    sgn[i] = bval < 0.0f ? -1.0f : 1.0f;
    if (blockIdx.x == 0) evals[i] = static_cast<float>(theta[i]);
  }
  __syncthreads();
  const int n = blockIdx.x * NT + threadIdx.x;
  if (n < d)
    for (int i = 0; i < r; ++i) V[static_cast<int64_t>(n) * r + i] *= sgn[i];
}

int gemm_splits(int d) {
  int s = d / 512;
  s = s < 1 ? 1 : (s > 8 ? 8 : s);
  while (s > 1 && (d % s != 0 || (d / s) % 8 != 0)) --s;
  return s;
}

struct EigWs {
  float *Vt, *Wt, *Xt, *part;
  double *gpart, *Rinv, *Q, *theta;
  float* cmax;
  int* cidx;
};

int64_t align256(int64_t b) { return (b + 255) & ~int64_t(255); }

int64_t layout(int d, int r, char* base, EigWs* w) {
  const int S = gemm_splits(d);
  const int64_t blk = static_cast<int64_t>(P) * d * 4;
  const int nblk = (d + NT - 1) / NT;
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
  const int nblk = (d + NT - 1) / NT;
  const size_t row_lds = static_cast<size_t>(d) * sizeof(float);
  const bool pre = (lam != nullptr) || B > 1;

  // block -> block: G~ applied to the rows of `in` (p x d), into `out`
  auto apply_op = [&](const float* in, float* out) {
    const float* x = in;
    if (pre) {
      hipLaunchKernelGGL(eig_row_kernel<false>, dim3(P), dim3(NT), row_lds, st, in, 1, int64_t(0), w.Xt, lam, B,
                         1.0f, d);
      x = w.Xt;
    }
    hipLaunchKernelGGL(eig_gemm_kernel, dim3(d / 64, S), dim3(NT), 0, st, x, A, w.part, d, d / S);
    hipLaunchKernelGGL(eig_row_kernel<true>, dim3(P), dim3(NT), row_lds, st, w.part, S,
                       static_cast<int64_t>(P) * d, out, lam, B, scale, d);
  };
  // rows of `src` orthonormalised into `dst` (one CholeskyQR pass)
  auto orth = [&](const float* src, float* dst) {
    hipLaunchKernelGGL(eig_gram_kernel, dim3(nch), dim3(NT), 0, st, src, src, w.gpart, d);
    hipLaunchKernelGGL(eig_chol_kernel, dim3(1), dim3(NT), 0, st, w.gpart, nch, w.Rinv);
    hipLaunchKernelGGL(eig_apply_kernel, dim3(nblk), dim3(NT), 0, st, src, w.Rinv, dst, d);
  };

  hipLaunchKernelGGL(eig_init_kernel, dim3((P * d + NT - 1) / NT), dim3(NT), 0, st, w.Vt, d,
                     static_cast<uint64_t>(0x51ED2701ull));
  orth(w.Vt, w.Wt);
  orth(w.Wt, w.Vt);
  for (int it = 0; it < iters; ++it) {
    apply_op(w.Vt, w.Wt);
    orth(w.Wt, w.Vt);
    orth(w.Vt, w.Wt);
    float* tmp = w.Vt;   // the orthonormal block is now in Wt
    w.Vt = w.Wt;
    w.Wt = tmp;
  }
  // Rayleigh-Ritz on the final block
  apply_op(w.Vt, w.Wt);
  hipLaunchKernelGGL(eig_gram_kernel, dim3(nch), dim3(NT), 0, st, w.Vt, w.Wt, w.gpart, d);
  hipLaunchKernelGGL(eig_jacobi_kernel, dim3(1), dim3(NT), 0, st, w.gpart, nch, w.Q, w.theta);
  hipLaunchKernelGGL(eig_ritz_kernel, dim3(nblk), dim3(NT), 0, st, w.Vt, w.Q, V, w.cmax, w.cidx, d, r);
  hipLaunchKernelGGL(eig_sign_kernel, dim3(nblk), dim3(NT), 0, st, V, w.cmax, w.cidx, nblk, w.theta, evals, d, r);
  return hipGetLastError();
}

}  // namespace qwam
