/*
 * qwam.h -- C ABI of the Action-Subspace-Protected (ASP) W4A4 linear layer
 * for AMD Instinct MI355X (gfx950).
 *
 * One ASP layer computes (row-vector convention, x is [M][K], y is [M][N])
 *
 *     y = Q4(x / lambda) . Q4(R)^T  +  ((x / lambda) . L1) . L2  (+ bias)
 *
 * following "Q-WAM: 4-Bit Quantization of World Action Models with
 * Action-Subspace Protection":
 *   - Q4 is the symmetric 4-bit group quantizer of Eq. 2 (Sec. 3), one float32
 *     scale per group of 64 consecutive input channels (or of 32, App. B.1's
 *     group size, with group = 32): scale = absmax / 7,
 *     code = clamp(round_half_even(v * (1 / scale)), -8, 7).  Weights are
 *     quantized once offline, activations per token at run time (Sec. 3,
 *     App. B.1).
 *   - lambda is the per-channel smoothing factor of Eq. 3 / App. B.1 (the
 *     activation is divided by it, the weight multiplied by it).
 *   - Optionally (layer field `hadamard` = B, the block size), the block
 *     Hadamard rotation of Eq. 3: x~ = H diag(lambda)^-1 x with H
 *     block-diagonal, orthonormal Hadamard blocks of size B; App. B.1 takes B
 *     = the largest power of two dividing K, at most 1024.  The weights must
 *     have been rotated the same way before packing (R is then the rotated
 *     residual and L1 a basis in rotated coordinates); the activation
 *     kernels rotate x online with the fast Walsh-Hadamard transform in
 *     float32: one rounding per butterfly, stages on channel bit 0, 1, ..,
 *     log2(B)-1 in that order (channel index within the block), then one
 *     multiply by fl32(1/sqrt(B)).
 *   - L1 = bf16(V) and L2 = bf16(V^T W~) are the factors of the 16-bit branch
 *     (V^T W~)^T (V^T x~) of Eq. 9, V being the top-r eigenvectors of the
 *     layer's Gramian (Eq. 7); R = W~ - L1 L2 is the deflated weight W~_perp.
 *   - The deployed layer is two kernels (App. B.1): one smooths, projects and
 *     quantizes the activation (qwam_quantize_act), the other multiplies the
 *     packed 4-bit operands and adds the branch and the bias in its epilogue
 *     (qwam_asp_linear).
 *
 * Conventions for every call
 *   - All array pointers are DEVICE pointers owned by the caller (the library
 *     never allocates and never frees).  The qwam_layer struct itself is a HOST
 *     struct read during the call only.
 *   - bf16 arrays are passed as uint16_t bit patterns.
 *   - Every call is asynchronous: it validates its arguments on the host,
 *     enqueues its kernel(s) on `stream` (a hipStream_t; NULL = the null
 *     stream) and returns.  Results are visible once the stream is
 *     synchronised.  The library never synchronises.
 *   - Every vector-loaded array must be 16-byte aligned (QWAM_ERR_MISALIGNED).
 *   - Arguments are checked before any HIP call is made and device memory is
 *     never dereferenced on the host; a failing check returns its status and
 *     enqueues nothing.  qwam_last_error() then returns a message
 *     (thread-local, valid until the thread's next call).
 *   - No exception or abort crosses the ABI.  Calls are reentrant; distinct
 *     streams may run calls concurrently on disjoint outputs.
 *   - Inputs must be finite (no NaN / Inf); other inputs give unspecified
 *     codes.
 *
 * Layouts (row-major, G = K / group)
 *   x    bf16    [M][K]      activations (row = token)
 *   R    float   [N][K]      residual weight, row = output channel
 *   smooth float [K]         lambda
 *   wq   uint8   [N][K/2]    packed weight codes (code blocks, below)
 *   ws   float   [G][N]      weight scales, group-major
 *   wsp  uint32  [G][N]      each weight scale as bf16 pieces hi | lo << 16 (qwam_layer)
 *   inv_smooth float [K]     fl32(1 / lambda)
 *   xq   uint8   [M][K/2]    packed activation codes (code blocks, below)
 *   xs   float   [G][M]      activation scales, group-major
 *   L1t  bf16    [r][K]      L1 transposed: row j is the j-th protected direction
 *   L1   bf16    [K][r]      L1 itself (row k: channel k of every direction), for the deflation
 *   L1f  bf16    [K*r]       L1 in fragment order (qwam_layer), for the down-projection t
 *   L2t  bf16    [N][r]      L2 transposed: row n holds (V^T W~)[:, n]
 *   t    bf16    [M][r]      t = bf16(sum_k bf16(x~_k) L1[k, j]), float32 accumulation
 *   bias bf16    [N]         optional
 *   y    bf16    [M][N]      output, round to nearest even from float32
 *
 * Code blocks: 4 bits per code.  The codes c[k0 .. k0+15] of 16 consecutive
 * channels of a row (k0 a multiple of 16) form one 8-byte block (bytes
 * k0/2 .. k0/2+7), read as two little-endian 32-bit words W0, W1.  Code j of
 * the block is the 6-bit field F_j = s << 5 | |c|, field j at bits 6j .. 6j+5
 * of the 96-bit stream
 * D0 | D1 << 32 | D2 << 64, whose bits 3-4 of every field are zero.  Those
 * bit positions of D0 and D1 (0x18618618 and 0x86186186) together are
 * exactly the data bits of D2, which is stored there:
 * W0 = D0 | (D2 & 0x18618618), W1 = D1 | (D2 & 0x86186186).  A field holds
 * the rounded scaled value rint(x), x = fl32(v * fl32(1/scale)), in sign and
 * magnitude: s is the IEEE sign bit of rint(x), which is that of x (rint
 * keeps the sign: rint(-0.3) = -0.0; with scale 0, x = v * 0).  So a zero
 * code may carry s = 1; it reads as 0.  Codes lie in [-7, 7]: with the scale
 * absmax / 7 the clamp of Eq. 2 never reaches -8.
 * (D0 = W0 & ~0x18618618, D1 = W1 & ~0x86186186 and
 * D2 = (W0 & 0x18618618) | (W1 & 0x86186186) give back the stream, whose
 * fields are the FP6 e2m3 values code / 8: that is how the GEMM consumes them.)
 *
 * Rotation: hadamard == 0, or a power of two with 16 <= hadamard <= 1024
 * dividing K (QWAM_ERR_INVALID_ARG otherwise).  It affects the activation
 * calls only; qwam_pack_weights and qwam_asp_linear do not read it.
 *
 * Shape limits: group == 64 or 32; K % 64 == 0, 64 <= K <= 65536; N % 16 == 0,
 * 16 <= N <= 1048576; r in {16, 32, 48, 64}; 1 <= M <= 1048576; for
 * qwam_asp_linear also M * K / 64 < 2^29 and N * K / 64 < 2^29
 * (QWAM_ERR_UNSUPPORTED otherwise).
 */
#ifndef QWAM_H
#define QWAM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QWAM_ABI_VERSION 13
#define QWAM_GROUP 64

typedef enum {
    QWAM_OK = 0,
    QWAM_ERR_INVALID_ARG = 1,   /* null pointer, bad shape or group size            */
    QWAM_ERR_UNSUPPORTED = 2,   /* well-formed but outside the supported limits     */
    QWAM_ERR_MISALIGNED = 3,    /* a vector-loaded array is not 16-byte aligned     */
    QWAM_ERR_NO_DEVICE = 4,     /* no HIP device is visible                         */
    QWAM_ERR_HIP = 5            /* the HIP runtime reported an error at launch      */
} qwam_status;

/* One packed ASP layer: a plain struct of caller-owned device pointers. */
typedef struct qwam_layer {
    int32_t K;                  /* input channels (multiple of 64)                  */
    int32_t N;                  /* output channels (multiple of 16)                 */
    int32_t r;                  /* rank of the protected subspace (16/32/48/64)     */
    int32_t group;              /* 64 or 32: channels per scale                       */
    int32_t hadamard;           /* block size B of the rotation, or 0 for none       */
    const uint8_t *wq;          /* [N][K/2]  packed residual codes                   */
    const float *ws;            /* [K/group][N] residual group scales                */
    const float *inv_smooth;    /* [K]       fl32(1/lambda)                          */
    const uint16_t *L1t;        /* [r][K]    bf16                                    */
    const uint16_t *L2t;        /* [N][r]    bf16                                    */
    const uint16_t *bias;       /* [N]       bf16, or NULL for no bias               */
    const uint16_t *L1;         /* [K][r]    bf16, the same factor as L1t row by row; */
                                /* read by qwam_quantize_act_deflated only (may be    */
                                /* NULL for a layer that is never deflated)           */
    const uint32_t *wsp;        /* [K/group][N] each ws as two bf16 pieces,          */
                                /* hi | lo << 16 with hi = bf16(ws) and              */
                                /* lo = bf16(ws - hi), both rounded to nearest even; */
                                /* written by qwam_pack_weights, read by             */
                                /* qwam_asp_linear                                   */
    const uint16_t *L1f;        /* L1 again, bf16, in the activation kernels'        */
                                /* fragment order [K/64][r/16][2][64][8]: entry      */
                                /* (g, b, h, l, e) = L1[64g + 16(l/16) + 8h + e]      */
                                /*                     [16b + l%16];                 */
                                /* read by the activation calls                      */
} qwam_layer;

/*
 * Offline weight pack (weights are quantized once, Sec. 3; the exported codes
 * of App. B.1).  Quantizes each group of `group` (64 or 32) consecutive entries
 * of each row of R with the quantizer of Eq. 2 (scale = fl32(absmax / 7); a group with absmax
 * below 7 * 2^-126 gets scale 0 and codes 0), packs the codes into code blocks
 * and writes
 * inv_smooth[k] = fl32(1 / smooth[k]).  It also writes each scale as the two
 * bf16 pieces the GEMM's scale products take (wsp, see qwam_layer).
 *   R          in   float [N][K]
 *   smooth     in   float [K], every entry finite and nonzero
 *   wq         out  uint8 [N][K/2]
 *   ws         out  float [K/group][N]
 *   wsp        out  uint32 [K/group][N]
 *   inv_smooth out  float [K]
 */
qwam_status qwam_pack_weights(int32_t K, int32_t N, int32_t group,
                              const float *R, const float *smooth,
                              uint8_t *wq, float *ws, uint32_t *wsp,
                              float *inv_smooth, void *stream);

/*
 * Activation side of one layer call (the first kernel of App. B.1): for every
 * token, x~ = fl32(x * inv_smooth) (Eq. 3, the smoothing divide done as a
 * multiply by the packed reciprocal), per-token group quantization of x~
 * (Eq. 2, absmax / 7 per token and group), code-word packing, and the rank-r
 * down-projection t = V^T x~ of Eq. 9 (bf16 inputs, float32 accumulation,
 * bf16 result), in one pass over x.  With L->hadamard != 0, x~ is also
 * rotated (Eq. 3) before it is quantized and projected.
 *   L   in   layer (reads K, r, group, hadamard, inv_smooth, L1t, L1f;
 *            L1t and L1f must both be set)
 *   x   in   bf16 [M][K]
 *   xq  out  uint8 [M][K/2]
 *   xs  out  float [K/group][M]
 *   t   out  bf16 [M][r]
 */
qwam_status qwam_quantize_act(const qwam_layer *L, int32_t M, const uint16_t *x,
                              uint8_t *xq, float *xs, uint16_t *t, void *stream);

/*
 * Activation side with the paper's deflation (Eq. 8 / Eq. 9): as
 * qwam_quantize_act, but the 4-bit path quantizes x~_perp = x~ - L1 t instead
 * of x~, so that the part of the activation the 16-bit branch carries is not
 * quantized twice.  Per token:
 *   x~      = fl32(x * inv_smooth)
 *   t       = bf16(sum_k bf16(x~_k) L1[k, j]) -- here rounded once from a
 *             float64 accumulation, i.e. the bf16 of the exact sum except
 *             within ~1e-13 relative of a rounding boundary
 *   x~_perp = x~, then for j = 0 .. r-1 in order:
 *             x~_perp <- fl32(x~_perp - t_j L1[:, j])   (exact products)
 *   xq, xs  = group quantization (Eq. 2) and code blocks of x~_perp
 * The outputs feed qwam_asp_linear unchanged: y = Q4(x~_perp) Q4(R)^T + t L2.
 * Arguments, layouts, ownership and errors as for qwam_quantize_act; it also
 * reads L->L1 (the deflation takes each channel's row of L1 whole), which
 * must be set and 16-byte aligned (QWAM_ERR_INVALID_ARG / QWAM_ERR_MISALIGNED).
 */
qwam_status qwam_quantize_act_deflated(const qwam_layer *L, int32_t M, const uint16_t *x,
                                       uint8_t *xq, float *xs, uint16_t *t, void *stream);

/*
 * The ASP GEMM (the second kernel of App. B.1): the integer partial sum of
 * every group, P[m, n, g] = sum_{k in g} qx[m, k] qw[n, k] (exact: the codes
 * are FP6 e2m3 operands of the matrix cores, every product and sum an integer
 * below 2^24), scaled by xs[g][m] * ws[g][n] and accumulated over the groups
 * in float32, plus the branch t . L2 and the bias, rounded to bf16:
 *     y[m, n] = bf16( sum_g xs ws P + sum_j t[m, j] L2t[n, j] + bias[n] )
 * The scale product xs * ws of a group is formed from two-piece bf16 splits
 * of each scale (hi = bf16(s), lo = bf16(s - hi)), within about 2^-15 of the
 * float32 product: the weight's from L->wsp, the activation's formed in the
 * kernel; the float32 sum runs in any order (App. B.1 allows the
 * accumulation order to differ).
 *   L   in   packed layer (L->wsp must be set)
 *   xq, xs, t  in  outputs of qwam_quantize_act for the same M
 *   y   out  bf16 [M][N]
 */
qwam_status qwam_asp_linear(const qwam_layer *L, int32_t M, const uint8_t *xq,
                            const float *xs, const uint16_t *t, uint16_t *y,
                            void *stream);

/*
 * The whole layer for few tokens in one call: the activation step of
 * qwam_quantize_act and the GEMM of qwam_asp_linear fused into one launch
 * (App. B.1 deploys them as two kernels; with at most 64 tokens both are
 * latency-bound, so every workgroup quantizes the tokens it needs itself).
 * The codes, scales and t are those qwam_quantize_act produces (t may differ
 * in float32 summation order); y as qwam_asp_linear.
 *   L   in   packed layer: r = 16 or 32, group 64, hadamard 0, K <= 16384
 *   M   in   1 <= M <= 64 (QWAM_ERR_UNSUPPORTED above)
 *   x   in   bf16 [M][K]
 *   y   out  bf16 [M][N]
 *   xq, xs, t  out, optional: all NULL, or all set (as for qwam_quantize_act)
 */
qwam_status qwam_asp_layer(const qwam_layer *L, int32_t M, const uint16_t *x, uint16_t *y,
                           uint8_t *xq, float *xs, uint16_t *t, void *stream);

/*
 * Test access to the exact integer group partials of qwam_asp_linear's
 * integer GEMM (same unpack and matrix-core path).
 *   L   in   packed layer (reads K, N, group, wq)
 *   xq  in   uint8 [M][K/2]
 *   P   out  int32 [M][N][K/group]
 */
qwam_status qwam_debug_group_partials(const qwam_layer *L, int32_t M, const uint8_t *xq,
                                      int32_t *P, void *stream);

/*
 * Accumulation of the Action Observability Gramian estimate (Sec. 4.1 and the
 * procedure of the probe estimator): every probe vector-Jacobian product
 * g = J^T u adds g g^T to a d x d accumulator, and G^ = A / (N P) after the
 * last input.  A batch of n such vectors, stored channel-major, is added at
 * once:
 *     A[i][j] += sum_k gT[i][k] gT[j][k]
 * (products of two bf16 values exact, sums in float32).  Only the tiles on or
 * above the diagonal are computed, and each is also written transposed, so a
 * symmetric A stays exactly symmetric.
 *   d   in      channels of the layer input, d % 16 == 0, 16 <= d <= 16384
 *   n   in      vectors in the batch, n % 64 == 0, n >= 64, d * n < 2^30
 *   gT  in      bf16 [d][n]: row c holds channel c of the n vectors
 *   A   in/out  float [d][d], accumulated in place
 */
qwam_status qwam_aog_accumulate(int32_t d, int32_t n, const uint16_t *gT, float *A, void *stream);

/*
 * The protected subspace from the AOG accumulator (Sec. 4.2, Eq. 7; the
 * procedure of the probe estimator; Prop. of App. A.3): the top-r eigenvectors
 * and eigenvalues of the estimate in the quantizer's coordinates,
 *     G~ = scale * H diag(lam) A diag(lam) H,
 * scale = 1 / (N P) for N inputs and P probes, lam the smoothing factors, H
 * the orthonormal block Hadamard matrix of block `hadamard` (the identity for
 * 0).  By blocked subspace iteration (a block of 64 vectors, `iters` products
 * with G~, each followed by a CholeskyQR orthonormalisation, the last block by
 * CholeskyQR2; Gram sums and Cholesky factors in float64) and a Rayleigh-Ritz
 * step (cyclic Jacobi in float64); products with A on the float32 matrix
 * cores.  The
 * result is deterministic.  Column i of V is the eigenvector of the i-th
 * largest eigenvalue, its largest-magnitude entry made positive.
 *   d       in   channels, d % 64 == 0, 128 <= d <= 16384
 *   r       in   1 <= r <= 48
 *   iters   in   0 .. 1000 products with G~ before the Rayleigh-Ritz step;
 *                the error falls like (lambda_65 / lambda_r)^iters
 *   A       in   float [d][d], symmetric (the accumulator of
 *                qwam_aog_accumulate); read as A^T
 *   scale   in   positive, finite
 *   lam     in   float [d] or NULL (no smoothing)
 *   hadamard in  0, or a power of two in [16, 1024] dividing d
 *   V       out  float [d][r]
 *   evals   out  float [r], descending
 *   workspace    device memory of at least
 *                qwam_aog_protected_basis_workspace(d, r) bytes, 16-byte
 *                aligned, owned by the caller; its contents on entry do not
 *                matter; calls that share it must not overlap
 */
qwam_status qwam_aog_protected_basis(int32_t d, int32_t r, int32_t iters, const float *A, float scale,
                                     const float *lam, int32_t hadamard, float *V, float *evals,
                                     void *workspace, int64_t workspace_bytes, void *stream);

/* Bytes of workspace qwam_aog_protected_basis needs for (d, r); -1 if the
 * shape is not supported. */
int64_t qwam_aog_protected_basis_workspace(int32_t d, int32_t r);

/* Message describing the calling thread's last non-OK status ("" if none). */
const char *qwam_last_error(void);

/* Static name of a status code. */
const char *qwam_status_string(qwam_status s);

/* QWAM_ABI_VERSION of the loaded library. */
int32_t qwam_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QWAM_H */
