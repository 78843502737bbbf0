// Measurement probes: what the chip itself sustains, so that every roofline
// fraction the benchmark reports can be read against a measured ceiling as
// well as against the vendor's figure.  None of this is part of the layer.
//
//   * matrix-core loops: each wave keeps four independent accumulators and
//     issues one MFMA after another (no dependent pair back to back), for the
//     matrix-core formats the layer uses or is compared with;
//   * a VALU loop of independent float32 fused multiply-adds (one lane result
//     per instruction; packed float32 instructions are never generated);
//   * a streaming copy (16 bytes per lane per access, grid-stride);
//   * an empty kernel, for the launch floor.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qwam_probe.h"

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v32f __attribute__((ext_vector_type(32)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;

thread_local char g_err[256] = "";

// operand words from the thread index: varied but never NaN / Inf patterns
// for the formats below (every FP6 / FP8 field and every bf16 is finite)
__device__ __forceinline__ int seed_word(int salt) {
  const unsigned t = threadIdx.x * 2654435761u + static_cast<unsigned>(salt) * 40503u;
  return static_cast<int>(t & 0x3C3C3C3Cu);    // clears the top two bits of every byte
}

template <int KIND>
__global__ __launch_bounds__(kThreads) void mfma_loop_kernel(int iters, float* out) {
  float sink = 0.0f;
  if constexpr (KIND == QWAM_PROBE_MFMA_FP6 || KIND == QWAM_PROBE_MFMA_FP8 || KIND == QWAM_PROBE_MFMA_FP4) {
    constexpr int fmt = KIND == QWAM_PROBE_MFMA_FP6 ? 2 : KIND == QWAM_PROBE_MFMA_FP4 ? 4 : 0;
    v8i a, b;
    for (int i = 0; i < 8; ++i) { a[i] = seed_word(i); b[i] = seed_word(i + 8); }
    v16f c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c0, fmt, fmt, 0, 127, 0, 127);
      c1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c1, fmt, fmt, 0, 127, 0, 127);
      c2 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c2, fmt, fmt, 0, 127, 0, 127);
      c3 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c3, fmt, fmt, 0, 127, 0, 127);
    }
    for (int v = 0; v < 16; ++v) sink += c0[v] + c1[v] + c2[v] + c3[v];
  } else if constexpr (KIND == QWAM_PROBE_MFMA_I8) {
    v4i a, b;
    for (int i = 0; i < 4; ++i) { a[i] = seed_word(i); b[i] = seed_word(i + 4); }
    v16i c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c3, 0, 0, 0);
    }
    for (int v = 0; v < 16; ++v) sink += static_cast<float>(c0[v] + c1[v] + c2[v] + c3[v]);
  } else if constexpr (KIND == QWAM_PROBE_MFMA_BF16) {
    v8bf a, b;
    for (int i = 0; i < 8; ++i) {
      a[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x + i) & 7) * 0.125f);
      b[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x * 3 + i) & 7) * 0.125f);
    }
    v16f c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
    for (int v = 0; v < 16; ++v) sink += c0[v] + c1[v] + c2[v] + c3[v];
  } else {   // QWAM_PROBE_MFMA_BF16_2B: the two-block K = 4 form
    v4s a, b;
    for (int i = 0; i < 4; ++i) {
      a[i] = static_cast<short>(0x3F80 + ((threadIdx.x + i) & 7));
      b[i] = static_cast<short>(0x3F80 + ((threadIdx.x * 5 + i) & 7));
    }
    v32f c0 = {}, c1 = {};
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x4bf16_1k(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x4bf16_1k(a, b, c1, 0, 0, 0);
      c0 = __builtin_amdgcn_mfma_f32_32x32x4bf16_1k(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x4bf16_1k(a, b, c1, 0, 0, 0);
    }
    for (int v = 0; v < 32; ++v) sink += c0[v] + c1[v];
  }
  out[blockIdx.x * kThreads + threadIdx.x] = sink;
}

// 16 independent float32 FMA chains per lane, 16 FMAs per chain and iteration
__global__ __launch_bounds__(kThreads) void valu_fma_loop_kernel(int iters, float* out) {
  float a[16];
  const float m = 0.999f + static_cast<float>(threadIdx.x & 7) * 1e-5f;
  const float c = 1e-3f * static_cast<float>(blockIdx.x & 3);
#pragma unroll
  for (int i = 0; i < 16; ++i) a[i] = static_cast<float>(i + threadIdx.x);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int i = 0; i < 16; ++i) a[i] = __builtin_fmaf(a[i], m, c);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += a[i];
  out[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                        int64_t n16) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n16; i += stride)
    dst[i] = src[i];
}

__global__ void empty_kernel() {}

qwam_status fail(qwam_status s, const char* msg) {
  snprintf(g_err, sizeof(g_err), "%s", msg);
  return s;
}

qwam_status launched(hipError_t e) {
  if (e != hipSuccess) return fail(QWAM_ERR_HIP, hipGetErrorString(e));
  g_err[0] = '\0';
  return QWAM_OK;
}

}  // namespace

extern "C" {

qwam_status qwam_probe_mfma(int32_t kind, int32_t workgroups, int32_t iters, float* out, void* stream) {
  if (workgroups < 1 || workgroups > 65536 || iters < 1 || iters > (1 << 24))
    return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_mfma: workgroups in [1, 65536], iters in [1, 2^24]");
  if (out == nullptr) return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_mfma: out is NULL");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 g(workgroups), b(kThreads);
  switch (kind) {
    case QWAM_PROBE_MFMA_FP6: hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_FP6>, g, b, 0, s, iters, out); break;
    case QWAM_PROBE_MFMA_FP8: hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_FP8>, g, b, 0, s, iters, out); break;
    case QWAM_PROBE_MFMA_FP4: hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_FP4>, g, b, 0, s, iters, out); break;
    case QWAM_PROBE_MFMA_I8: hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_I8>, g, b, 0, s, iters, out); break;
    case QWAM_PROBE_MFMA_BF16: hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_BF16>, g, b, 0, s, iters, out); break;
    case QWAM_PROBE_MFMA_BF16_2B:
      hipLaunchKernelGGL(mfma_loop_kernel<QWAM_PROBE_MFMA_BF16_2B>, g, b, 0, s, iters, out);
      break;
    default: return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_mfma: unknown kind");
  }
  return launched(hipGetLastError());
}

qwam_status qwam_probe_valu_fma(int32_t workgroups, int32_t iters, float* out, void* stream) {
  if (workgroups < 1 || workgroups > 65536 || iters < 1 || iters > (1 << 24))
    return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_valu_fma: workgroups in [1, 65536], iters in [1, 2^24]");
  if (out == nullptr) return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_valu_fma: out is NULL");
  hipLaunchKernelGGL(valu_fma_loop_kernel, dim3(workgroups), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     iters, out);
  return launched(hipGetLastError());
}

qwam_status qwam_probe_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream) {
  if (src == nullptr || dst == nullptr) return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_copy: NULL buffer");
  if (bytes <= 0 || bytes % 16 != 0) return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_copy: bytes must be a positive multiple of 16");
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u)
    return fail(QWAM_ERR_MISALIGNED, "qwam_probe_copy: buffers must be 16-byte aligned");
  if (workgroups < 1 || workgroups > 65536) return fail(QWAM_ERR_INVALID_ARG, "qwam_probe_copy: workgroups in [1, 65536]");
  hipLaunchKernelGGL(copy_kernel, dim3(workgroups), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), bytes / 16);
  return launched(hipGetLastError());
}

qwam_status qwam_probe_empty(void* stream) {
  hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream));
  return launched(hipGetLastError());
}

const char* qwam_probe_last_error(void) { return g_err; }

}  // extern "C"
