// Host-side launchers of the ASP kernels (internal to libqwam).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qwam {

hipError_t launch_pack_weights(int K, int N, int group, const float* R, const float* smooth, uint8_t* wq,
                               float* ws, uint32_t* wsp, float* inv_smooth, hipStream_t stream);

// L1f: the fragment-ordered copy of L1 (qwam_layer) that the activation
// kernels' down-projection reads
hipError_t launch_quantize_act(int M, int K, int r, int group, const uint16_t* x, const float* inv_smooth,
                               const uint16_t* L1f, uint8_t* xq, float* xs, uint16_t* t,
                               hipStream_t stream);

// the 4-bit path quantizes the deflated activation x~ - L1 t (Eq. 8 / Eq. 9);
// L1 is [K][r] bf16 (the deflation's rows), L1t the same factor as [r][K]
hipError_t launch_quantize_act_deflated(int M, int K, int r, int group, const uint16_t* x,
                                        const float* inv_smooth, const uint16_t* L1f, const uint16_t* L1,
                                        uint8_t* xq, float* xs, uint16_t* t, hipStream_t stream);

// the same two activation kernels with the block Hadamard rotation of Eq. 3
// (block B, a power of two with 16 <= B <= 1024 dividing K)
hipError_t launch_quantize_act_rotated(int M, int K, int r, int group, int B, bool deflate, const uint16_t* x,
                                       const float* inv_smooth, const uint16_t* L1t, const uint16_t* L1f,
                                       const uint16_t* L1, uint8_t* xq, float* xs, uint16_t* t,
                                       hipStream_t stream);

hipError_t launch_asp_gemm(int M, int N, int K, int r, int group, const uint8_t* xq, const float* xs,
                           const uint16_t* t, const uint8_t* wq, const float* ws, const uint32_t* wsp,
                           const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                           hipStream_t stream);

hipError_t launch_group_partials(int M, int N, int K, int group, const uint8_t* xq, const uint8_t* wq,
                                 int32_t* P, hipStream_t stream);

// AOG accumulation: A [d][d] += gT gT^T, gT bf16 [d][n], n % 64 == 0
hipError_t launch_aog_accumulate(int d, int n, const uint16_t* gT, float* A, hipStream_t stream);

// top-r eigenvectors of G~ = scale H diag(lam) A diag(lam) H by subspace
// iteration with a block of kEigBlock vectors; r <= kEigMaxRank, d % 64 == 0
constexpr int kEigBlock = 64;
constexpr int kEigMaxRank = 48;
int64_t eig_workspace_bytes(int d, int r);
hipError_t launch_aog_eig(int d, int r, int iters, const float* A, float scale, const float* lam, int B, float* V,
                          float* evals, void* workspace, hipStream_t stream);

// the few-token GEMM (one wave per 32 x 32 block), used for M <= kSmallM
constexpr int kSmallM = 64;

hipError_t launch_asp_gemm_small(int M, int N, int K, int r, int group, const uint8_t* xq, const float* xs,
                                 const uint16_t* t, const uint8_t* wq, const float* ws,
                                 const uint16_t* L2t, const uint16_t* bias, uint16_t* y,
                                 hipStream_t stream);

// the whole layer for M <= kSmallM in one launch (r = 16 or 32, group 64, no
// rotation); xq / xs / t are optional outputs (all null or none)
hipError_t launch_asp_layer_small(int M, int N, int K, int r, const uint16_t* x, const float* inv_smooth,
                                  const uint16_t* L1t, const uint8_t* wq, const float* ws, const uint16_t* L2t,
                                  const uint16_t* bias, uint16_t* y, uint8_t* xq, float* xs, uint16_t* t,
                                  hipStream_t stream);

hipError_t launch_group_partials_small(int M, int N, int K, int group, const uint8_t* xq, const uint8_t* wq,
                                       int32_t* P, hipStream_t stream);

}  // namespace qwam
